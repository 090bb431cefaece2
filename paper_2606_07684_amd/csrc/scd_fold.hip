// Fold of the Patch aligner's output layer into the consumer's key/value projections.
//
// Section 4.4.2: the aligner (Eq. aligner) ends in an affine layer, H_hat = act W2^T + b2, and
// Eq. kv_from_patch feeds H_hat straight into the consumer's projections W_K / W_V, with no
// nonlinearity in between.  So, for P = K or V,
//   H_hat W_P^T + b_P = act (W_P W2)^T + (W_P b2 + b_P),
// and the consumer can regenerate a Patch layer's K/V from the aligner's hidden activations with
// one product of inner dimension h instead of two (h then d_model).  The folded weights depend on
// the weights only, so they are formed once per model pair:
//   w_fold = W_P W2   [D, h],      c = W_P b2 + b_P   [D],
// accumulated in fp32 and rounded once to the model's dtype.
//
// This is a one-time preparation step, not part of a request's path: a plain LDS-tiled fp32 VALU
// product (64 x 64 output tiles, 32-wide contraction steps) that reads both operands in their
// stored layouts (W_P [D, d] row-major, W2 [d, h] row-major) without a transposed copy.
#include "scd_kernels.h"

namespace scd {
namespace {

constexpr int kFT = 64;        // output tile edge (rows of W_P x columns of W2)
constexpr int kFK = 32;        // contraction step
constexpr int kFThreads = 256;
constexpr int kFPad = kFT + 4; // LDS row: 16-byte aligned, offset by 4 banks per row

template <bool BF16>
__device__ inline float load1(const void* base, int64_t i) {
  if constexpr (BF16)
    return __uint_as_float(static_cast<uint32_t>(static_cast<const uint16_t*>(base)[i]) << 16);
  else
    return static_cast<const float*>(base)[i];
}

// Eight consecutive elements starting at element i (i a multiple of 8, base 16-byte aligned).
template <bool BF16>
__device__ inline void load8(const void* base, int64_t i, float* f) {
  if constexpr (BF16) {
    const uint4 v = *reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(base) + i);
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      f[2 * e] = __uint_as_float(w[e] << 16);
      f[2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u);
    }
  } else {
    const float4* s = reinterpret_cast<const float4*>(static_cast<const float*>(base) + i);
    const float4 a = s[0], b = s[1];
    f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w;
    f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
  }
}

__device__ inline uint32_t bf16_bits(float f) {
  return static_cast<uint32_t>(__builtin_bit_cast(uint16_t, static_cast<__bf16>(f)));
}

// One 64 x 64 tile of w_fold = W_P W2 per workgroup; each thread owns a 4 x 4 block.
template <bool BF16>
__global__ __launch_bounds__(kFThreads) void patch_fold_kernel(const FoldParams p) {
  __shared__ __attribute__((aligned(16))) float As[kFK][kFPad];  // [k][row of W_P]
  __shared__ __attribute__((aligned(16))) float Bs[kFK][kFPad];  // [k][column of W2]
  const int D = p.n, d = p.d_model, h = p.hidden;
  const int tiles_j = (h + kFT - 1) / kFT;
  const int per_job = ((D + kFT - 1) / kFT) * tiles_j;
  const int job = blockIdx.x / per_job, t = blockIdx.x % per_job;
  const int n0 = (t / tiles_j) * kFT, j0 = (t % tiles_j) * kFT;
  const FoldJob& jb = p.jobs[job];
  const int tid = threadIdx.x, tx = tid % 16, ty = tid / 16;
  // loader slots: a row of W_P and 8 of its columns; a row of W2 and 8 of its columns
  const int an = tid / 4, ak = (tid % 4) * 8;
  const int bk = tid / 8, bj = (tid % 8) * 8;

  float acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;

  for (int k0 = 0; k0 < d; k0 += kFK) {
    float a[8], b[8];
    if (n0 + an < D) load8<BF16>(jb.wp, static_cast<int64_t>(n0 + an) * d + k0 + ak, a);
    else
#pragma unroll
      for (int e = 0; e < 8; ++e) a[e] = 0.f;
    if (j0 + bj < h) load8<BF16>(jb.w2, static_cast<int64_t>(k0 + bk) * h + j0 + bj, b);
    else
#pragma unroll
      for (int e = 0; e < 8; ++e) b[e] = 0.f;
    __syncthreads();  // the previous step's reads are done
#pragma unroll
    for (int e = 0; e < 8; ++e) As[ak + e][an] = a[e];
#pragma unroll
    for (int e = 0; e < 8; ++e) Bs[bk][bj + e] = b[e];
    __syncthreads();
#pragma unroll 8
    for (int kk = 0; kk < kFK; ++kk) {
      const float4 av = *reinterpret_cast<const float4*>(&As[kk][ty * 4]);
      const float4 bv = *reinterpret_cast<const float4*>(&Bs[kk][tx * 4]);
      const float ar[4] = {av.x, av.y, av.z, av.w}, br[4] = {bv.x, bv.y, bv.z, bv.w};
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(ar[i], br[j], acc[i][j]);
    }
  }

  // h % 16 == 0, so a thread's four columns are all inside or all outside the matrix.
  const int j = j0 + tx * 4;
  if (j >= h) return;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int n = n0 + ty * 4 + i;
    if (n >= D) continue;
    const int64_t o = static_cast<int64_t>(n) * h + j;
    if constexpr (BF16) {
      uint2 v;
      v.x = bf16_bits(acc[i][0]) | (bf16_bits(acc[i][1]) << 16);
      v.y = bf16_bits(acc[i][2]) | (bf16_bits(acc[i][3]) << 16);
      *reinterpret_cast<uint2*>(static_cast<uint16_t*>(jb.wf) + o) = v;
    } else {
      *reinterpret_cast<float4*>(static_cast<float*>(jb.wf) + o) =
          make_float4(acc[i][0], acc[i][1], acc[i][2], acc[i][3]);
    }
  }
}

// c = W_P b2 + b_P: one wave per output channel, fp32 partial sums reduced across the wave.
template <bool BF16>
__global__ __launch_bounds__(256) void patch_fold_bias_kernel(const FoldParams p) {
  const FoldJob& jb = p.jobs[blockIdx.y];
  const int lane = threadIdx.x & 63;
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (n >= p.n) return;  // uniform per wave
  float s = 0.f;
  if (jb.b2 != nullptr)
    for (int i = lane; i < p.d_model; i += 64)
      s = fmaf(load1<BF16>(jb.wp, static_cast<int64_t>(n) * p.d_model + i), load1<BF16>(jb.b2, i), s);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
  if (lane != 0) return;
  if (jb.bp != nullptr) s += load1<BF16>(jb.bp, n);
  if constexpr (BF16) static_cast<uint16_t*>(jb.c)[n] = static_cast<uint16_t>(bf16_bits(s));
  else static_cast<float*>(jb.c)[n] = s;
}

}  // namespace

hipError_t launch_patch_fold(bool bf16, const FoldParams& p, hipStream_t stream) {
  if (p.n_jobs <= 0) return hipSuccess;
  const int64_t tiles = static_cast<int64_t>((p.n + kFT - 1) / kFT) * ((p.hidden + kFT - 1) / kFT);
  const dim3 grid(static_cast<unsigned>(tiles * p.n_jobs));
  const dim3 bgrid(static_cast<unsigned>((p.n + 3) / 4), static_cast<unsigned>(p.n_jobs));
  if (bf16) {
    hipLaunchKernelGGL(patch_fold_kernel<true>, grid, dim3(kFThreads), 0, stream, p);
    hipLaunchKernelGGL(patch_fold_bias_kernel<true>, bgrid, dim3(256), 0, stream, p);
  } else {
    hipLaunchKernelGGL(patch_fold_kernel<false>, grid, dim3(kFThreads), 0, stream, p);
    hipLaunchKernelGGL(patch_fold_bias_kernel<false>, bgrid, dim3(256), 0, stream, p);
  }
  return hipGetLastError();
}

}  // namespace scd
