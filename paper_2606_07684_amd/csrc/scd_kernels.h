// Internal declarations shared by the host API and the HIP kernels of the SCD codec.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace scd {

// Most jobs one launch carries in its kernel arguments (jobs beyond it go to further launches).
constexpr int kMaxJobs = 32;

enum JobFlags : int32_t {
  kRopeOut = 1,   // rotate output column pairs (i, i + d_h/2) of every head by the row's position
  kDeropeIn = 2,  // inverse-rotate input column pairs of A before the contraction
};

// One dense product C[M, n] = prologue(A)[M, k] * B[n, k]^T (+ bias[n]) followed by the epilogue
// the flags select.  A, B and C are row-major and contiguous.
struct GemmJob {
  const void* a;
  const void* b;
  void* c;
  const void* bias;   // [n] added before RoPE, or null
  const void* mu_in;  // [k] subtracted from A after deRoPE, or null
  int32_t n;
  int32_t k;
  int32_t flags;
  int32_t tile_begin;  // first tile index of this job within the launch
};

struct GemmParams {
  GemmJob jobs[kMaxJobs];
  int32_t n_jobs;
  int32_t total_tiles;
  int64_t m;            // rows of A and C (shared by every job of the launch)
  int32_t g;            // rows per token (row r belongs to token r / g)
  int32_t head_dim;
  int32_t n_seqs;
  int32_t pad_;
  const int32_t* cu_seqlens;  // [n_seqs + 1] or null (one request)
  const int32_t* pos0;        // [n_seqs] or null
  const float2* rope;         // [max_pos][head_dim / 2] (cos, sin)
  int64_t max_pos;
};

// Tile shape of the generic launcher (rows x columns of C per workgroup).
constexpr int kGenericBM = 128;
constexpr int kGenericBN = 128;

// Launchers (return the hipError_t of the launch).
hipError_t launch_gemm_bf16(const GemmParams& p, hipStream_t stream);
hipError_t launch_gemm_f32(const GemmParams& p, hipStream_t stream);
hipError_t launch_rope_table(float2* table, int64_t max_pos, int head_dim, double theta,
                             hipStream_t stream);
hipError_t launch_positions(int32_t* out, int64_t n_tokens, int32_t n_seqs,
                            const int32_t* cu_seqlens, const int32_t* pos0, hipStream_t stream);

}  // namespace scd
