// Generic MFMA kernel of the SCD codec: C[M, n] = prologue(A)[M, k] * B[n, k]^T, epilogue.
//
// One launch runs a table of jobs that share M.  Every Reuse-decode branch (Eq. decode_kv),
// every Patch branch (Eq. kv_from_patch) and every encode branch (Eq. encode_z_kv and the Patch
// code of Section 4.4.1) is one such product:
//   decode  A = codes [T*g, r]      B = W_dec [w, r]     epilogue + mu, RoPE on keys
//   patch   A = H_hat [T, d_model]  B = W_K|W_V [D, d]   epilogue + bias, RoPE on keys
//   encode  A = K|V  [T*g, w]       B = W_enc [r, w]     prologue deRoPE on keys, - mu
//
// Workgroup: 256 threads (2 x 2 waves), a 128 x 128 tile of C, K consumed 32 at a time through
// double-buffered LDS.  bf16 uses v_mfma_f32_16x16x32_bf16, fp32 uses v_mfma_f32_16x16x4_f32,
// both accumulating in fp32.  Each 32-wide K chunk is two 16-wide pieces; when A needs deRoPE
// the second piece is the first one's RoPE partner (columns i and i + d_h/2 of one head), so a
// thread holds both members of every pair it rotates.  Both operands use the same piece order,
// so the contraction is unchanged.  The epilogue goes through LDS so that RoPE pairs meet in one
// thread and every global store is a 16-byte vector.
#include <type_traits>

#include "scd_kernels.h"

namespace scd {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kNumXcd = 8;

// Workgroups are dispatched round-robin over the XCDs.  Renumber them so each XCD receives a
// contiguous range of tiles: neighbouring tiles (which share A rows) then share one L2.
__device__ inline int xcd_remap(int bid, int nb) {
  const int q = nb / kNumXcd, rem = nb % kNumXcd;
  const int x = bid % kNumXcd, i = bid / kNumXcd;
  return (x < rem ? x * (q + 1) : rem * (q + 1) + (x - rem) * q) + i;
}

// Position of code row `row` (token row / g) within its own request.
__device__ inline int64_t row_position(const GemmParams& p, int64_t row) {
  if (row >= p.m) return 0;
  int64_t t = row / p.g;
  int b = 0;
  if (p.cu_seqlens != nullptr) {
    int lo = 0, hi = p.n_seqs - 1;  // largest b with cu[b] <= t
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (p.cu_seqlens[mid] <= t) lo = mid; else hi = mid - 1;
    }
    b = lo;
    t -= p.cu_seqlens[b];
  }
  return t + (p.pos0 != nullptr ? p.pos0[b] : 0);
}

__device__ inline int64_t table_row(const GemmParams& p, int64_t pos) {
  return pos < 0 ? 0 : (pos >= p.max_pos ? p.max_pos - 1 : pos);
}

template <bool BF16> struct Elem;
template <> struct Elem<true> {
  using T = uint16_t;
  static constexpr int kVecs = 1;  // 16-byte vectors per 8 elements
  __device__ static inline void unpack(const uint4* v, float* f) {
    const uint32_t w[4] = {v[0].x, v[0].y, v[0].z, v[0].w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[2 * i] = __uint_as_float(w[i] << 16);
      f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  }
  __device__ static inline uint32_t bits(float f) {
    return static_cast<uint32_t>(__builtin_bit_cast(uint16_t, static_cast<__bf16>(f)));
  }
  __device__ static inline void pack(const float* f, uint4* v) {
    v[0].x = bits(f[0]) | (bits(f[1]) << 16);
    v[0].y = bits(f[2]) | (bits(f[3]) << 16);
    v[0].z = bits(f[4]) | (bits(f[5]) << 16);
    v[0].w = bits(f[6]) | (bits(f[7]) << 16);
  }
  __device__ static inline float load1(const void* p, int64_t i) {
    return __uint_as_float(static_cast<uint32_t>(static_cast<const uint16_t*>(p)[i]) << 16);
  }
};
template <> struct Elem<false> {
  using T = float;
  static constexpr int kVecs = 2;
  __device__ static inline void unpack(const uint4* v, float* f) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      f[4 * i] = __uint_as_float(v[i].x);
      f[4 * i + 1] = __uint_as_float(v[i].y);
      f[4 * i + 2] = __uint_as_float(v[i].z);
      f[4 * i + 3] = __uint_as_float(v[i].w);
    }
  }
  __device__ static inline void pack(const float* f, uint4* v) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      v[i].x = __float_as_uint(f[4 * i]);
      v[i].y = __float_as_uint(f[4 * i + 1]);
      v[i].z = __float_as_uint(f[4 * i + 2]);
      v[i].w = __float_as_uint(f[4 * i + 3]);
    }
  }
  __device__ static inline float load1(const void* p, int64_t i) {
    return static_cast<const float*>(p)[i];
  }
};

// Tag types that name each step's kernel.
struct ReuseDecode {};
struct PatchKV {};
struct EncodeKV {};
struct EncodeH {};
struct PatchAlign {};

template <typename OP, bool BF16, int BM, int BN, int WM, int WN>
__global__ __launch_bounds__(WM * WN * 64) void gemm_nt_kernel(GemmParams p) {
  using EL = Elem<BF16>;
  using T = typename EL::T;
  constexpr int BK = 32;
  constexpr int NT = WM * WN * 64;
  constexpr int NV = EL::kVecs;
  constexpr int LDK = BK + 16 / static_cast<int>(sizeof(T));  // LDS row, padded by 16 bytes
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int FM = WTM / 16, FN = WTN / 16;
  constexpr int LDC = BN + 4;
  constexpr int TPA = (BM * 2) / NT, TPB = (BN * 2) / NT;
  static_assert(TPA * NT == BM * 2 && TPB * NT == BN * 2, "loader split");
  constexpr size_t kAB = 2u * (BM + BN) * LDK * sizeof(T);
  constexpr size_t kC = static_cast<size_t>(BM) * LDC * sizeof(float);
  constexpr size_t kSmem = kAB > kC ? kAB : kC;

  __shared__ __attribute__((aligned(16))) unsigned char smem[kSmem];
  __shared__ int s_pos[BM];
  T* As = reinterpret_cast<T*>(smem);
  T* Bs = As + 2 * BM * LDK;
  float* Cs = reinterpret_cast<float*>(smem);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;

  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  int j = 0;
  while (j + 1 < p.n_jobs && bid >= p.jobs[j + 1].tile_begin) ++j;
  const GemmJob job = p.jobs[j];
  const int local = bid - job.tile_begin;
  const int ntn = (job.n + BN - 1) / BN;
  const int64_t m0 = static_cast<int64_t>(local / ntn) * BM;
  const int n0 = (local % ntn) * BN;
  const bool derope = (job.flags & kDeropeIn) != 0;
  const bool rope_out = (job.flags & kRopeOut) != 0;
  const bool vec_in = (job.flags & kVecIn) != 0 && job.vec != nullptr;
  const bool vec_out = (job.flags & kVecOut) != 0 && job.vec != nullptr;
  const bool silu_out = (job.flags & kSiluOut) != 0;
  const int dh = p.head_dim, half = dh / 2;
  const int K = job.k, N = job.n;
  const int64_t M = p.m;
  const int nk = (K + BK - 1) / BK;
  const int heads_in_row = K / dh;
  const T* A = static_cast<const T*>(job.a);
  const T* B = static_cast<const T*>(job.b);

  if (derope || rope_out) {
    for (int r = tid; r < BM; r += NT) s_pos[r] = static_cast<int>(row_position(p, m0 + r));
  }
  __syncthreads();

  auto bases = [&](int kc, int& b0, int& b1) {
    if (derope) {
      const int o = kc / heads_in_row, h = kc % heads_in_row;
      b0 = h * dh + o * 16;
      b1 = b0 + half;
    } else {
      b0 = kc * BK;
      b1 = b0 + 16;
    }
  };

  uint4 ra[TPA][2][NV], rb[TPB][2][NV];
  const uint4 zero = make_uint4(0, 0, 0, 0);

  auto gload = [&](int kc) {
    int b0, b1;
    bases(kc, b0, b1);
#pragma unroll
    for (int t = 0; t < TPA; ++t) {
      const int task = tid + t * NT, row = task >> 1, q = task & 1;
      const int64_t gr = m0 + row;
#pragma unroll
      for (int pc = 0; pc < 2; ++pc) {
        const int col = (pc ? b1 : b0) + 8 * q;
        const bool ok = gr < M && col < K;
        // out-of-range pieces read an in-bounds address and are replaced by zero
        const uint4* src = reinterpret_cast<const uint4*>(A + (ok ? gr * K + col : 0));
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          const uint4 x = src[v];
          ra[t][pc][v] = ok ? x : zero;
        }
      }
    }
#pragma unroll
    for (int t = 0; t < TPB; ++t) {
      const int task = tid + t * NT, row = task >> 1, q = task & 1;
      const int gn = n0 + row;
#pragma unroll
      for (int pc = 0; pc < 2; ++pc) {
        const int col = (pc ? b1 : b0) + 8 * q;
        const bool ok = gn < N && col < K;
        const uint4* src =
            reinterpret_cast<const uint4*>(B + (ok ? static_cast<int64_t>(gn) * K + col : 0));
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          const uint4 x = src[v];
          rb[t][pc][v] = ok ? x : zero;
        }
      }
    }
  };

  auto sstore = [&](int kc, int buf) {
    int b0, b1;
    bases(kc, b0, b1);
#pragma unroll
    for (int t = 0; t < TPA; ++t) {
      const int task = tid + t * NT, row = task >> 1, q = task & 1;
      uint4* d0 = reinterpret_cast<uint4*>(As + (buf * BM + row) * LDK + 8 * q);
      uint4* d1 = reinterpret_cast<uint4*>(As + (buf * BM + row) * LDK + 16 + 8 * q);
      if (derope || vec_in) {
        float u[8], v[8];
        EL::unpack(ra[t][0], u);
        EL::unpack(ra[t][1], v);
        if (derope) {
          const int i0 = (b0 % dh) + 8 * q;
          const float2* cs = p.rope + table_row(p, s_pos[row]) * half + i0;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float2 c = cs[e];
            const float uu = u[e], vv = v[e];
            u[e] = uu * c.x + vv * c.y;
            v[e] = vv * c.x - uu * c.y;
          }
        }
        if (vec_in) {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int c0 = b0 + 8 * q + e, c1 = b1 + 8 * q + e;
            if (c0 < K) u[e] -= EL::load1(job.vec, c0);
            if (c1 < K) v[e] -= EL::load1(job.vec, c1);
          }
        }
        uint4 o0[NV], o1[NV];
        EL::pack(u, o0);
        EL::pack(v, o1);
#pragma unroll
        for (int w = 0; w < NV; ++w) { d0[w] = o0[w]; d1[w] = o1[w]; }
      } else {
#pragma unroll
        for (int w = 0; w < NV; ++w) { d0[w] = ra[t][0][w]; d1[w] = ra[t][1][w]; }
      }
    }
#pragma unroll
    for (int t = 0; t < TPB; ++t) {
      const int task = tid + t * NT, row = task >> 1, q = task & 1;
      uint4* d0 = reinterpret_cast<uint4*>(Bs + (buf * BN + row) * LDK + 8 * q);
      uint4* d1 = reinterpret_cast<uint4*>(Bs + (buf * BN + row) * LDK + 16 + 8 * q);
#pragma unroll
      for (int w = 0; w < NV; ++w) { d0[w] = rb[t][0][w]; d1[w] = rb[t][1][w]; }
    }
  };

  f32x4 acc[FM][FN];
#pragma unroll
  for (int a = 0; a < FM; ++a)
#pragma unroll
    for (int b = 0; b < FN; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int lr = lane & 15, lk = (lane >> 4) * 8;
  auto compute = [&](int buf) {
    const T* Ab = As + buf * BM * LDK;
    const T* Bb = Bs + buf * BN * LDK;
    if constexpr (BF16) {
      bf16x8 af[FM], bfr[FN];
#pragma unroll
      for (int a = 0; a < FM; ++a)
        af[a] = *reinterpret_cast<const bf16x8*>(Ab + (wm * WTM + a * 16 + lr) * LDK + lk);
#pragma unroll
      for (int b = 0; b < FN; ++b)
        bfr[b] = *reinterpret_cast<const bf16x8*>(Bb + (wn * WTN + b * 16 + lr) * LDK + lk);
#pragma unroll
      for (int a = 0; a < FM; ++a)
#pragma unroll
        for (int b = 0; b < FN; ++b)
          acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[a], bfr[b], acc[a][b], 0, 0, 0);
    } else {
      float af[FM][8], bfr[FN][8];
#pragma unroll
      for (int a = 0; a < FM; ++a) {
        const float4* s = reinterpret_cast<const float4*>(Ab + (wm * WTM + a * 16 + lr) * LDK + lk);
        const float4 x0 = s[0], x1 = s[1];
        af[a][0] = x0.x; af[a][1] = x0.y; af[a][2] = x0.z; af[a][3] = x0.w;
        af[a][4] = x1.x; af[a][5] = x1.y; af[a][6] = x1.z; af[a][7] = x1.w;
      }
#pragma unroll
      for (int b = 0; b < FN; ++b) {
        const float4* s = reinterpret_cast<const float4*>(Bb + (wn * WTN + b * 16 + lr) * LDK + lk);
        const float4 x0 = s[0], x1 = s[1];
        bfr[b][0] = x0.x; bfr[b][1] = x0.y; bfr[b][2] = x0.z; bfr[b][3] = x0.w;
        bfr[b][4] = x1.x; bfr[b][5] = x1.y; bfr[b][6] = x1.z; bfr[b][7] = x1.w;
      }
#pragma unroll
      for (int e = 0; e < 8; ++e)
#pragma unroll
        for (int a = 0; a < FM; ++a)
#pragma unroll
          for (int b = 0; b < FN; ++b)
            acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[a][e], bfr[b][e], acc[a][b], 0, 0, 0);
    }
  };

  if (nk > 0) {
    gload(0);
    sstore(0, 0);
    __syncthreads();
    for (int kc = 0; kc < nk; ++kc) {
      const int cur = kc & 1;
      if (kc + 1 < nk) gload(kc + 1);
      compute(cur);
      if (kc + 1 < nk) sstore(kc + 1, cur ^ 1);
      __syncthreads();
    }
  }

  // Accumulators -> LDS (fp32).  MFMA output: lane holds column lane%16, rows 4*(lane/16)+e.
#pragma unroll
  for (int a = 0; a < FM; ++a)
#pragma unroll
    for (int b = 0; b < FN; ++b)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int row = wm * WTM + a * 16 + 4 * (lane >> 4) + e;
        const int col = wn * WTN + b * 16 + (lane & 15);
        Cs[row * LDC + col] = acc[a][b][e];
      }
  __syncthreads();

  T* C = static_cast<T*>(job.c);
  if (rope_out) {
    const int gph = dh / 16;          // 8-wide groups in half a head
    constexpr int GPR = BN / 16;      // pair groups per tile row
    for (int task = tid; task < BM * GPR; task += NT) {
      const int row = task / GPR, cg = task % GPR;
      const int o = (cg % gph) * 8;
      const int c0 = (cg / gph) * dh + o, c1 = c0 + half;
      const int64_t gm = m0 + row;
      const int gc0 = n0 + c0, gc1 = n0 + c1;
      if (gm >= M || gc0 >= N) continue;
      float u[8], v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) { u[e] = Cs[row * LDC + c0 + e]; v[e] = Cs[row * LDC + c1 + e]; }
      if (vec_out) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          u[e] += EL::load1(job.vec, gc0 + e);
          v[e] += EL::load1(job.vec, gc1 + e);
        }
      }
      const float2* cs = p.rope + table_row(p, s_pos[row]) * half + o;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float2 c = cs[e];
        const float uu = u[e], vv = v[e];
        u[e] = uu * c.x - vv * c.y;
        v[e] = vv * c.x + uu * c.y;
      }
      uint4 o0[NV], o1[NV];
      EL::pack(u, o0);
      EL::pack(v, o1);
      uint4* d0 = reinterpret_cast<uint4*>(C + gm * N + gc0);
      uint4* d1 = reinterpret_cast<uint4*>(C + gm * N + gc1);
#pragma unroll
      for (int w = 0; w < NV; ++w) { d0[w] = o0[w]; d1[w] = o1[w]; }
    }
  } else {
    constexpr int GPR = BN / 8;
    for (int task = tid; task < BM * GPR; task += NT) {
      const int row = task / GPR, c0 = (task % GPR) * 8;
      const int64_t gm = m0 + row;
      const int gc0 = n0 + c0;
      if (gm >= M || gc0 >= N) continue;
      float u[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) u[e] = Cs[row * LDC + c0 + e];
      if (vec_out) {
#pragma unroll
        for (int e = 0; e < 8; ++e) u[e] += EL::load1(job.vec, gc0 + e);
      }
      if (silu_out) {
#pragma unroll
        for (int e = 0; e < 8; ++e) u[e] = u[e] / (1.f + expf(-u[e]));
      }
      uint4 o0[NV];
      EL::pack(u, o0);
      uint4* d0 = reinterpret_cast<uint4*>(C + gm * N + gc0);
#pragma unroll
      for (int w = 0; w < NV; ++w) d0[w] = o0[w];
    }
  }
}

__global__ void rope_table_kernel(float2* table, int64_t n, int half, int head_dim,
                                  double theta) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (idx >= n) return;
  const int64_t pos = idx / half;
  const int i = static_cast<int>(idx % half);
  const double omega = pow(theta, -2.0 * static_cast<double>(i) / static_cast<double>(head_dim));
  const double a = static_cast<double>(pos) * omega;
  double s, c;
  sincos(a, &s, &c);
  table[idx] = make_float2(static_cast<float>(c), static_cast<float>(s));
}

__global__ void positions_kernel(int32_t* out, int64_t n_tokens, int32_t n_seqs,
                                 const int32_t* cu, const int32_t* pos0) {
  const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t >= n_tokens) return;
  int b = 0;
  int64_t local = t;
  if (cu != nullptr) {
    int lo = 0, hi = n_seqs - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (cu[mid] <= t) lo = mid; else hi = mid - 1;
    }
    b = lo;
    local = t - cu[b];
  }
  out[t] = static_cast<int32_t>(local + (pos0 != nullptr ? pos0[b] : 0));
}

}  // namespace

template <typename OP, bool BF16>
hipError_t launch_one(const GemmParams& p, hipStream_t stream) {
  hipLaunchKernelGGL((gemm_nt_kernel<OP, BF16, kGenericBM, kGenericBN, 2, 2>),
                     dim3(p.total_tiles), dim3(256), 0, stream, p);
  return hipGetLastError();
}

template <typename OP>
hipError_t launch_op(bool bf16, const GemmParams& p, hipStream_t stream) {
  return bf16 ? launch_one<OP, true>(p, stream) : launch_one<OP, false>(p, stream);
}

hipError_t launch_gemm(Op op, bool bf16, const GemmParams& p, hipStream_t stream) {
  if (p.total_tiles <= 0) return hipSuccess;
  switch (op) {
    case Op::kReuseDecode: return launch_op<ReuseDecode>(bf16, p, stream);
    case Op::kPatchKV: return launch_op<PatchKV>(bf16, p, stream);
    case Op::kEncodeKV: return launch_op<EncodeKV>(bf16, p, stream);
    case Op::kEncodeH: return launch_op<EncodeH>(bf16, p, stream);
    case Op::kPatchAlign: return launch_op<PatchAlign>(bf16, p, stream);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_rope_table(float2* table, int64_t max_pos, int head_dim, double theta,
                             hipStream_t stream) {
  const int half = head_dim / 2;
  const int64_t n = max_pos * half;
  if (n <= 0) return hipSuccess;
  const int64_t blocks = (n + 255) / 256;
  hipLaunchKernelGGL(rope_table_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream,
                     table, n, half, head_dim, theta);
  return hipGetLastError();
}

hipError_t launch_positions(int32_t* out, int64_t n_tokens, int32_t n_seqs,
                            const int32_t* cu_seqlens, const int32_t* pos0, hipStream_t stream) {
  if (n_tokens <= 0) return hipSuccess;
  const int64_t blocks = (n_tokens + 255) / 256;
  hipLaunchKernelGGL(positions_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream,
                     out, n_tokens, n_seqs, cu_seqlens, pos0);
  return hipGetLastError();
}

}  // namespace scd
