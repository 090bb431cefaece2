// Internal declarations shared by the host API and the HIP kernels of the SCD codec.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace scd {

// Most jobs one launch carries in its kernel arguments (jobs beyond it go to further launches).
// 64 jobs keep the argument block near 3 KiB.
constexpr int kMaxJobs = 64;

enum JobFlags : int32_t {
  kRopeOut = 1,   // rotate output column pairs (i, i + d_h/2) of every head by the row's position
  kDeropeIn = 2,  // inverse-rotate input column pairs of A before the contraction
  kVecOut = 4,    // vec[n] is added to every output row before RoPE (decoder offset, bias)
  kVecIn = 8,     // vec[k] is subtracted from every row of A after deRoPE (encoder offset)
  kSiluOut = 16,  // SiLU x / (1 + e^-x) on every output after vec (aligner hidden layer)
};

// One dense product C[M, n] = prologue(A)[M, k] * B[n, k]^T (+ bias[n]) followed by the epilogue
// the flags select.  A, B and C are row-major and contiguous.
struct GemmJob {
  const void* a;
  const void* b;
  void* c;
  const void* vec;    // [n] (kVecOut) or [k] (kVecIn); null when neither flag is set
  int32_t n;
  int32_t k;
  int32_t flags;
  int32_t tile_begin;  // first tile index of this job within the launch
};
static_assert(sizeof(GemmJob) == 48, "job descriptor size");

struct GemmParams {
  GemmJob jobs[kMaxJobs];
  int32_t n_jobs;
  int32_t total_tiles;
  int64_t m;            // rows of A and C (shared by every job of the launch)
  int32_t g;            // rows per token (row r belongs to token r / g)
  int32_t head_dim;
  int32_t n_seqs;
  int32_t reserved;
  const int32_t* cu_seqlens;  // [n_seqs + 1] or null (one request)
  const int32_t* pos0;        // [n_seqs] or null
  const float2* rope;         // [max_pos][head_dim / 2] (cos, sin)
  int64_t max_pos;
};
static_assert(sizeof(GemmParams) <= 4096, "kernel argument block");

// Tile shape of the generic launcher (rows x columns of C per workgroup).
constexpr int kGenericBM = 128;
constexpr int kGenericBN = 128;

// The codec step a launch performs; each step is its own kernel symbol so profiles attribute time
// per step.
enum class Op : int { kReuseDecode = 0, kPatchKV = 1, kEncodeKV = 2, kEncodeH = 3, kPatchAlign = 4 };

// Launchers (return the hipError_t of the launch).
hipError_t launch_gemm(Op op, bool bf16, const GemmParams& p, hipStream_t stream);

// Patch on the bf16 path: 256 x 256 tiles (tokens x channels), d_model % 64 == 0, head_dim 64 or
// 128, D % 128 == 0.
constexpr int kPatchBM = 256;
constexpr int kPatchBN = 256;
hipError_t launch_patch_bf16(const GemmParams& p, hipStream_t stream);
// The aligner's two products on the same kernel (its own symbol): C = act(A B^T + vec), with
// act = SiLU on jobs flagged kSiluOut; no RoPE.
hipError_t launch_align_bf16(const GemmParams& p, hipStream_t stream);

// Fold of the aligner's output layer into a projection (one-time, weights only):
// wf = wp w2 [n, hidden] and c = wp b2 + bp [n], fp32 accumulation, one rounding.
struct FoldJob {
  const void* wp;  // [n, d_model]  consumer projection W_K or W_V
  const void* w2;  // [d_model, hidden]  aligner output layer
  const void* b2;  // [d_model] or null
  const void* bp;  // [n] or null (projection bias)
  void* wf;        // [n, hidden] out
  void* c;         // [n] out
};
struct FoldParams {
  FoldJob jobs[kMaxJobs];
  int32_t n_jobs;
  int32_t n;        // D
  int32_t d_model;  // multiple of 32
  int32_t hidden;   // multiple of 16
};
static_assert(sizeof(FoldParams) <= 4096, "kernel argument block");
hipError_t launch_patch_fold(bool bf16, const FoldParams& p, hipStream_t stream);

// Reuse decode on the bf16 path: workgroups own a channel chunk of 128 * nhg and a share of the
// launch's row tiles (decode_tile_rows(nhg) rows each); basis_width % (128 * nhg) == 0, one rank
// (% 32 == 0, <= 256) and one branch per launch, head_dim 64 or 128.
int decode_channel_groups(int rank, int basis_width);
int decode_tile_rows(int nhg, int rank);  // rows per tile of the kernel instance
// align: run the aligner's first product (jobs flagged kSiluOut, rank <= 128, no RoPE) under its
// own kernel symbol.
hipError_t launch_decode_bf16(int nhg, const GemmParams& p, hipStream_t stream, bool align = false);

// Largest batch (requests) the bf16 decode kernel stages in LDS.
constexpr int kMaxLdsSeqs = 256;
// Rows every RoPE table holds at least (positions 0..15 are read as in-tile offsets).
constexpr int kRopeMinRows = 16;

// Encode on the bf16 path: a unit is 128 rows x all code columns; k % 128 == 0, n <= 256,
// head_dim 64 or 128 when a job de-rotates.
constexpr int kEncodeRows = 128;
hipError_t launch_encode_bf16(const GemmParams& p, hipStream_t stream);
// ---- Offline Reuse fit (joint Gram of de-rotated producer/consumer rows, then a small fp64
// solve).  The Gram of X = [A B] (N rows of 2w columns) is accumulated per 128 x 128 upper tile and
// per slice of rows into a workspace of partial tiles, then summed over slices in a fixed order.
constexpr int kFitTile = 128;   // Gram tile edge
constexpr int kFitRowStep = 64; // rows per k-step of the Gram kernels; slices are multiples of it

struct FitGramJob {
  const void* a;   // producer cache [T, D] = rows [N, w]
  const void* b;   // consumer cache
  float* gram;     // [2w, 2w] out
  float* colsum;   // [2w] out
};

struct FitGramParams {
  FitGramJob jobs[kMaxJobs];
  int32_t n_jobs;
  int32_t w;           // basis width; the joint rows have 2w columns
  int64_t n_rows;      // N = T * g
  int32_t g;           // rows per token
  int32_t head_dim;
  int32_t derope;      // keys: inverse-rotate both caches' rows first
  int32_t n_slices;
  int64_t slice_rows;  // multiple of kFitRowStep
  int32_t n_seqs;
  int32_t reserved;
  const int32_t* cu_seqlens;
  const int32_t* pos0;
  const float2* rope;
  int64_t max_pos;
  float* partial;      // [n_jobs][n_slices][n_upper][kFitTile^2 + kFitTile]
};
static_assert(sizeof(FitGramParams) <= 4096, "kernel argument block");

struct FitSolveJob {
  const float* gram;    // [2w, 2w]
  const float* colsum;  // [2w]
  void* w_enc;          // [r, w] out (model dtype)
  void* w_dec;          // [w, r] out
  void* mu_enc;         // [w] out, or null (no centring)
  void* mu_dec;         // [w] out, or null
  int32_t rank;
  int32_t reserved;
};

struct FitSolveParams {
  FitSolveJob jobs[kMaxJobs];
  int32_t n_jobs;
  int32_t w;
  int64_t n_rows;
  double lambda;
  int32_t center;
  int32_t bf16;
  double* work;  // n_jobs x fit_solve_layer_doubles(w) fp64
};
static_assert(sizeof(FitSolveParams) <= 4096, "kernel argument block");

// Largest basis width the solve takes (w = D = 1024 for a model with 8 KV heads of 128).
constexpr int kFitMaxSolveWidth = 1024;
// fp64 workspace of the solve per layer: four 2w x 2w matrices and 8 vectors of 2w.
__host__ __device__ constexpr int64_t fit_solve_layer_doubles(int w) {
  return 4 * (2 * static_cast<int64_t>(w)) * (2 * w) + 8 * (2 * static_cast<int64_t>(w));
}

int64_t fit_upper_tiles(int w);  // upper 128 x 128 tiles of the 2w x 2w Gram
// bf16 with 2w = 256: one workgroup per (job, slice) computes the whole Gram
bool fit_full_gram(bool bf16, int w);
// workgroups of a Gram launch per row slice
int64_t fit_units_per_slice(bool bf16, int w, int n_jobs);
hipError_t launch_fit_gram(bool bf16, const FitGramParams& p, hipStream_t stream);
hipError_t launch_fit_solve(const FitSolveParams& p, hipStream_t stream);

// Size of the device-resident scratch array of the allocation-free solve (one per GPU).
constexpr size_t kFitScratchBytes = size_t{64} << 20;
// Device address of the calling thread's current device's scratch array, looked up once per
// device (hipGetSymbolAddress) and cached.
hipError_t fit_scratch(double** ptr);

hipError_t launch_rope_table(float2* table, int64_t max_pos, int head_dim, double theta,
                             hipStream_t stream);
hipError_t launch_positions(int32_t* out, int64_t n_tokens, int32_t n_seqs,
                            const int32_t* cu_seqlens, const int32_t* pos0, hipStream_t stream);

}  // namespace scd
