// Patch KV regeneration (Section 4.4.2, Eq. kv_from_patch) as a bf16 MFMA GEMM for gfx950:
//   K = RoPE(H_hat W_K^T + b_K),  V = H_hat W_V^T + b_V   written straight into the KV cache.
//
// One workgroup computes a 256 (channels n) x 256 (tokens t) tile of C^T = W * H_hat^T with four
// waves, each owning 128 channels x 128 tokens as 4 x 4 blocks of v_mfma_f32_32x32x16_bf16.
// The weight tile is the MFMA A operand, so an accumulator register holds one token's channels;
// weight rows are stored into LDS in a permuted order that gives each lane 16 consecutive channels
// of one token.  A wave's 128 channels are whole heads, so every RoPE pair (i, i + d_h/2) meets in
// one lane and the epilogue needs no LDS: bias, rotation and bf16 rounding happen in registers and
// each lane stores two 16-byte vectors per block.  K advances 64 at a time through double-buffered
// LDS (2 x 2 x 256 x 72 bf16 = 144 KiB, rows padded by 16 bytes so MFMA reads are conflict-free);
// the next stage's global loads are in flight while the current stage is multiplied.
#include "scd_kernels.h"

namespace scd {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kBM = 256;   // tokens per tile
constexpr int kBN = 256;   // channels per tile
constexpr int kBK = 64;    // contraction step
constexpr int kLDK = kBK + 8;  // padded LDS row (bf16 elements)
constexpr int kThreads = 256;
constexpr int kNumXcd = 8;

template <int V> struct IntC { static constexpr int value = V; };

__device__ inline int xcd_remap(int bid, int nb) {
  const int q = nb / kNumXcd, rem = nb % kNumXcd;
  const int x = bid % kNumXcd, i = bid / kNumXcd;
  return (x < rem ? x * (q + 1) : rem * (q + 1) + (x - rem) * q) + i;
}

__device__ inline int token_position(const GemmParams& p, int64_t t) {
  int b = 0;
  int64_t local = t;
  if (p.cu_seqlens != nullptr) {
    int lo = 0, hi = p.n_seqs - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (p.cu_seqlens[mid] <= t) lo = mid; else hi = mid - 1;
    }
    b = lo;
    local = t - p.cu_seqlens[b];
  }
  int64_t pos = local + (p.pos0 != nullptr ? p.pos0[b] : 0);
  pos = pos < 0 ? 0 : (pos >= p.max_pos ? p.max_pos - 1 : pos);
  return static_cast<int>(pos);
}

// LDS row that holds weight row `n` of a 32-row block: the MFMA reads rows in natural order and
// row i of the block must be channel 16*((i>>2)&1) + 4*(i>>3) + (i&3), so that accumulator
// element r of lane l is channel 16*(l/32) + r.
__device__ inline int lds_row_of_channel(int n) {
  const int o = n & 31;
  return (n & ~31) | (8 * ((o >> 2) & 3) + 4 * (o >> 4) + (o & 3));
}

__device__ inline float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ inline uint32_t pack_bf16x2(float a, float b) {
  const uint32_t lo = __builtin_bit_cast(uint16_t, static_cast<__bf16>(a));
  const uint32_t hi = __builtin_bit_cast(uint16_t, static_cast<__bf16>(b));
  return lo | (hi << 16);
}

__global__ __launch_bounds__(kThreads, 1) void patch_kv_bf16_kernel(GemmParams p) {
  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * 2 * kBM * kLDK];
  uint16_t* Ws = smem;                    // [2][kBN][kLDK]
  uint16_t* Hs = smem + 2 * kBN * kLDK;   // [2][kBM][kLDK]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wn = wave >> 1, wt = wave & 1;

  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  int j = 0;
  while (j + 1 < p.n_jobs && bid >= p.jobs[j + 1].tile_begin) ++j;
  const GemmJob job = p.jobs[j];
  const int local = bid - job.tile_begin;
  const int N = job.n, K = job.k;
  const int64_t M = p.m;
  const int ntn = (N + kBN - 1) / kBN;
  const int64_t t0 = static_cast<int64_t>(local / ntn) * kBM;
  const int n0 = (local % ntn) * kBN;
  const uint16_t* W = static_cast<const uint16_t*>(job.b);
  const uint16_t* Hh = static_cast<const uint16_t*>(job.a);
  const int nk = K / kBK;

  // Global -> register staging: 8 16-byte chunks per tile row; 2048 chunks per operand tile.
  uint4 rw[8], rh[8];
  auto gload = [&](int kc) {
    const int kb = kc * kBK;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int q = tid + kThreads * i;
      const int row = q >> 3, c = q & 7;
      const int n = n0 + row;
      rw[i] = n < N ? *reinterpret_cast<const uint4*>(W + static_cast<int64_t>(n) * K + kb + 8 * c)
                    : make_uint4(0, 0, 0, 0);
      const int64_t t = t0 + row;
      rh[i] = t < M ? *reinterpret_cast<const uint4*>(Hh + t * K + kb + 8 * c)
                    : make_uint4(0, 0, 0, 0);
    }
  };
  auto sstore = [&](int buf) {
    uint16_t* wb = Ws + buf * kBN * kLDK;
    uint16_t* hb = Hs + buf * kBM * kLDK;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int q = tid + kThreads * i;
      const int row = q >> 3, c = q & 7;
      *reinterpret_cast<uint4*>(wb + lds_row_of_channel(row) * kLDK + 8 * c) = rw[i];
      *reinterpret_cast<uint4*>(hb + row * kLDK + 8 * c) = rh[i];
    }
  };

  f32x16 acc[4][4];
#pragma unroll
  for (int s = 0; s < 4; ++s)
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[s][u][e] = 0.f;

  const int lr = lane & 31, lk = (lane >> 5) * 8;
  auto compute = [&](int buf) {
    const uint16_t* wb = Ws + buf * kBN * kLDK + (wn * 128 + lr) * kLDK + lk;
    const uint16_t* hb = Hs + buf * kBM * kLDK + (wt * 128 + lr) * kLDK + lk;
#pragma unroll
    for (int ks = 0; ks < kBK / 16; ++ks) {
      bf16x8 af[4], bfr[4];
#pragma unroll
      for (int s = 0; s < 4; ++s)
        af[s] = *reinterpret_cast<const bf16x8*>(wb + s * 32 * kLDK + ks * 16);
#pragma unroll
      for (int u = 0; u < 4; ++u)
        bfr[u] = *reinterpret_cast<const bf16x8*>(hb + u * 32 * kLDK + ks * 16);
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int u = 0; u < 4; ++u)
          acc[s][u] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[s], bfr[u], acc[s][u], 0, 0, 0);
    }
  };

  gload(0);
  sstore(0);
  __syncthreads();
  for (int kc = 0; kc < nk; ++kc) {
    const int cur = kc & 1;
    if (kc + 1 < nk) gload(kc + 1);
    compute(cur);
    if (kc + 1 < nk) sstore(cur ^ 1);
    __syncthreads();
  }

  // Epilogue.  Lane l holds, for block (s, u), token t0 + wt*128 + 32u + l%32 and channels
  // n0 + wn*128 + 32s + 16*(l/32) + r, r = 0..15.
  const bool rope = (job.flags & kRopeOut) != 0;
  const bool add_vec = (job.flags & kVecOut) != 0 && job.vec != nullptr;
  const uint16_t* bias = static_cast<const uint16_t*>(job.vec);
  uint16_t* C = static_cast<uint16_t*>(job.c);
  const int dh = p.head_dim, half = dh >> 1;
  // Pairs of blocks that hold (i, i + d_h/2): (0,2),(1,3) for d_h = 128; (0,1),(2,3) for 64.
  const int pstride = half >> 5;  // 2 or 1
  const int nw = n0 + wn * 128;
  const int hl = 16 * (lane >> 5);

  auto load16 = [&](int nb, float* v) {
    if (add_vec && nb < N) {
      const uint4* src = reinterpret_cast<const uint4*>(bias + nb);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const uint4 x = src[h];
        v[8 * h + 0] = bf16_lo(x.x); v[8 * h + 1] = bf16_hi(x.x);
        v[8 * h + 2] = bf16_lo(x.y); v[8 * h + 3] = bf16_hi(x.y);
        v[8 * h + 4] = bf16_lo(x.z); v[8 * h + 5] = bf16_hi(x.z);
        v[8 * h + 6] = bf16_lo(x.w); v[8 * h + 7] = bf16_hi(x.w);
      }
    } else {
#pragma unroll
      for (int e = 0; e < 16; ++e) v[e] = 0.f;
    }
  };
  auto store16 = [&](int64_t t, int nb, const float* y) {
    if (nb >= N) return;
    uint4 o0, o1;
    o0.x = pack_bf16x2(y[0], y[1]);   o0.y = pack_bf16x2(y[2], y[3]);
    o0.z = pack_bf16x2(y[4], y[5]);   o0.w = pack_bf16x2(y[6], y[7]);
    o1.x = pack_bf16x2(y[8], y[9]);   o1.y = pack_bf16x2(y[10], y[11]);
    o1.z = pack_bf16x2(y[12], y[13]); o1.w = pack_bf16x2(y[14], y[15]);
    uint4* dst = reinterpret_cast<uint4*>(C + t * N + nb);
    dst[0] = o0;
    dst[1] = o1;
  };

  // One pair of blocks (S, S + PS) holds channels (i, i + d_h/2); S and PS are compile-time so the
  // accumulators stay in registers.
  auto finish_pair = [&](auto s_c, auto ps_c, int u, int64_t t, const float2* cs_row) {
    constexpr int S = decltype(s_c)::value;
    constexpr int SP = S + decltype(ps_c)::value;
    const int nb = nw + 32 * S + hl, nbp = nw + 32 * SP + hl;
    float a[16], b[16];
    load16(nb, a);
    load16(nbp, b);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      a[r] += acc[S][u][r];
      b[r] += acc[SP][u][r];
    }
    if (rope) {
      const int i0 = (32 * S + hl) & (half - 1);  // pair index of channel r = 0
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float2 c = cs_row[i0 + r];
        const float x = a[r], y = b[r];
        a[r] = x * c.x - y * c.y;
        b[r] = y * c.x + x * c.y;
      }
    }
    store16(t, nb, a);
    store16(t, nbp, b);
  };

#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int64_t t = t0 + wt * 128 + 32 * u + (lane & 31);
    if (t >= M) continue;
    const float2* cs_row =
        rope ? p.rope + static_cast<int64_t>(token_position(p, t)) * half : nullptr;
    if (pstride == 2) {
      finish_pair(IntC<0>{}, IntC<2>{}, u, t, cs_row);
      finish_pair(IntC<1>{}, IntC<2>{}, u, t, cs_row);
    } else {
      finish_pair(IntC<0>{}, IntC<1>{}, u, t, cs_row);
      finish_pair(IntC<2>{}, IntC<1>{}, u, t, cs_row);
    }
  }
}

}  // namespace

hipError_t launch_patch_bf16(const GemmParams& p, hipStream_t stream) {
  if (p.total_tiles <= 0) return hipSuccess;
  hipLaunchKernelGGL(patch_kv_bf16_kernel, dim3(p.total_tiles), dim3(kThreads), 0, stream, p);
  return hipGetLastError();
}

}  // namespace scd
