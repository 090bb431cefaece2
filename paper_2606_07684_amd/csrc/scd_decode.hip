// Reuse decode (Section 4.3.2, Eq. decode_kv) on the bf16 path for gfx950:
//   K = RoPE(unrows(Z_K W_dec,K^T + mu_K)),  V = unrows(Z_V W_dec,V^T + mu_V)
// written straight into the consumer's KV cache.  The step is bound by HBM writes (every
// reconstructed element is written once; codes and bases are r/w of that traffic).
//
// A workgroup owns CN = 128 * NWC channels of one layer-branch and a group of kTilesPerGroup token
// tiles.  It stages its basis chunk (CN rows of W_dec, permuted as in the Patch kernel so each MFMA
// accumulator lane holds 16 consecutive channels of one token) and the offset chunk in LDS once,
// then every wave computes 128 channels x 32 tokens per tile with v_mfma_f32_32x32x16_bf16: the
// basis is the A operand, the codes (loaded straight from HBM into registers one 32-wide chunk
// ahead) the B operand.  Offset, RoPE and bf16 rounding happen in registers and each lane writes
// 16-byte vectors with non-temporal stores.  The workgroups of one token group (one per channel
// chunk) are launched next to each other, so they run on one XCD and its L2 serves the code
// tile to all of them.
#include "scd_kernels.h"

namespace scd {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kNumXcd = 8;
constexpr int kThreads = 256;

template <int V> struct IntC { static constexpr int value = V; };

__device__ inline int xcd_remap(int bid, int nb) {
  const int q = nb / kNumXcd, rem = nb % kNumXcd;
  const int x = bid % kNumXcd, i = bid / kNumXcd;
  return (x < rem ? x * (q + 1) : rem * (q + 1) + (x - rem) * q) + i;
}

// Position (table row) of code row `row` (token row / g) within its own request.
__device__ inline int row_position(const GemmParams& p, int64_t row) {
  const int64_t t = row / p.g;
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

template <int NWC>
__global__ __launch_bounds__(kThreads) void reuse_decode_bf16_kernel(GemmParams p) {
  constexpr int CN = 128 * NWC;             // channels per workgroup
  constexpr int NWT = 4 / NWC;              // waves along tokens
  constexpr int TT = 32 * NWT;              // tokens per tile
  extern __shared__ __attribute__((aligned(16))) uint16_t lds[];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wc = wave % NWC, wt = wave / NWC;

  // unit -> (job, token group, channel chunk); channel chunk fastest
  const int unit = xcd_remap(blockIdx.x, gridDim.x);
  int j = 0;
  while (j + 1 < p.n_jobs && unit >= p.jobs[j + 1].tile_begin) ++j;
  const GemmJob job = p.jobs[j];
  const int N = job.n, K = job.k;
  const int n_nc = N / CN;
  const int local = unit - job.tile_begin;
  const int nc = local % n_nc, tg = local / n_nc;
  const int64_t M = p.m;
  const int n0 = nc * CN;
  const int ldk = K + 8;  // LDS row stride of the basis chunk (elements)
  uint16_t* Fs = lds;                 // [CN][ldk]
  uint16_t* mus = lds + CN * ldk;     // [CN]
  const uint16_t* F = static_cast<const uint16_t*>(job.b);
  const uint16_t* Z = static_cast<const uint16_t*>(job.a);
  const uint16_t* mu = static_cast<const uint16_t*>(job.vec);
  const bool add_mu = (job.flags & kVecOut) != 0 && mu != nullptr;
  const bool rope = (job.flags & kRopeOut) != 0;

  // Stage the basis chunk (rows n0 .. n0+CN) and the offset chunk.
  {
    const int cpr = K / 8;  // 16-byte chunks per row
    for (int q = tid; q < CN * cpr; q += kThreads) {
      const int row = q / cpr, c = q % cpr;
      const uint4 v = *reinterpret_cast<const uint4*>(F + static_cast<int64_t>(n0 + row) * K + 8 * c);
      *reinterpret_cast<uint4*>(Fs + lds_row_of_channel(row) * ldk + 8 * c) = v;
    }
    for (int q = tid; q < CN / 8; q += kThreads) {
      const uint4 v = add_mu ? *reinterpret_cast<const uint4*>(mu + n0 + 8 * q)
                             : make_uint4(0, 0, 0, 0);
      *reinterpret_cast<uint4*>(mus + 8 * q) = v;
    }
  }
  __syncthreads();

  const int dh = p.head_dim, half = dh >> 1;
  const int pstride = half >> 5;  // blocks between RoPE partners: 2 (d_h 128) or 1 (d_h 64)
  const int hl = 16 * (lane >> 5);
  const int lk = 8 * (lane >> 5);
  const int nkc = K / 32;
  const uint16_t* fw = Fs + (wc * 128 + (lane & 31)) * ldk + lk;
  uint16_t* C = static_cast<uint16_t*>(job.c);
  const int64_t row_first = static_cast<int64_t>(tg) * kTilesPerGroup * TT;

  for (int tile = 0; tile < kTilesPerGroup; ++tile) {
    const int64_t row0 = row_first + static_cast<int64_t>(tile) * TT;
    if (row0 >= M) break;
    const int64_t row = row0 + wt * 32 + (lane & 31);
    const bool valid = row < M;
    const uint16_t* zrow = Z + (valid ? row : 0) * K + lk;

    f32x16 acc[4];
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[s][e] = 0.f;

    // codes for k-chunk c (32 wide = two MFMA k-steps); loaded one chunk ahead of use
    // rows past the end read row 0 (always in bounds); their results are never stored
    uint4 zc0 = *reinterpret_cast<const uint4*>(zrow);
    uint4 zc1 = *reinterpret_cast<const uint4*>(zrow + 16);
    uint4 zn0 = zc0, zn1 = zc1;
    for (int c = 0; c < nkc; ++c) {
      if (c + 1 < nkc) {
        zn0 = *reinterpret_cast<const uint4*>(zrow + 32 * (c + 1));
        zn1 = *reinterpret_cast<const uint4*>(zrow + 32 * (c + 1) + 16);
      }
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const uint4 zv = ks == 0 ? zc0 : zc1;
        const bf16x8 bz = __builtin_bit_cast(bf16x8, zv);
        bf16x8 af[4];
#pragma unroll
        for (int s = 0; s < 4; ++s)
          af[s] = *reinterpret_cast<const bf16x8*>(fw + s * 32 * ldk + 32 * c + 16 * ks);
#pragma unroll
        for (int s = 0; s < 4; ++s)
          acc[s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[s], bz, acc[s], 0, 0, 0);
      }
      zc0 = zn0;
      zc1 = zn1;
    }

    if (!valid) continue;
    const float2* cs_row = rope ? p.rope + static_cast<int64_t>(row_position(p, row)) * half
                                : nullptr;
    auto finish_pair = [&](auto s_c, auto ps_c) {
      constexpr int S = decltype(s_c)::value;
      constexpr int SP = S + decltype(ps_c)::value;
      const int cl = wc * 128 + 32 * S + hl, clp = wc * 128 + 32 * SP + hl;  // local channels
      float a[16], b[16];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const uint4 ma = *reinterpret_cast<const uint4*>(mus + cl + 8 * h);
        const uint4 mb = *reinterpret_cast<const uint4*>(mus + clp + 8 * h);
        a[8 * h + 0] = bf16_lo(ma.x); a[8 * h + 1] = bf16_hi(ma.x);
        a[8 * h + 2] = bf16_lo(ma.y); a[8 * h + 3] = bf16_hi(ma.y);
        a[8 * h + 4] = bf16_lo(ma.z); a[8 * h + 5] = bf16_hi(ma.z);
        a[8 * h + 6] = bf16_lo(ma.w); a[8 * h + 7] = bf16_hi(ma.w);
        b[8 * h + 0] = bf16_lo(mb.x); b[8 * h + 1] = bf16_hi(mb.x);
        b[8 * h + 2] = bf16_lo(mb.y); b[8 * h + 3] = bf16_hi(mb.y);
        b[8 * h + 4] = bf16_lo(mb.z); b[8 * h + 5] = bf16_hi(mb.z);
        b[8 * h + 6] = bf16_lo(mb.w); b[8 * h + 7] = bf16_hi(mb.w);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        a[r] += acc[S][r];
        b[r] += acc[SP][r];
      }
      if (rope) {
        const int i0 = (32 * S + hl) & (half - 1);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float2 cs = cs_row[i0 + r];
          const float x = a[r], y = b[r];
          a[r] = x * cs.x - y * cs.y;
          b[r] = y * cs.x + x * cs.y;
        }
      }
      u32x4* da = reinterpret_cast<u32x4*>(C + row * N + n0 + cl);
      u32x4* db = reinterpret_cast<u32x4*>(C + row * N + n0 + clp);
      u32x4 o;
      o.x = pack_bf16x2(a[0], a[1]);   o.y = pack_bf16x2(a[2], a[3]);
      o.z = pack_bf16x2(a[4], a[5]);   o.w = pack_bf16x2(a[6], a[7]);
      __builtin_nontemporal_store(o, da);
      o.x = pack_bf16x2(a[8], a[9]);   o.y = pack_bf16x2(a[10], a[11]);
      o.z = pack_bf16x2(a[12], a[13]); o.w = pack_bf16x2(a[14], a[15]);
      __builtin_nontemporal_store(o, da + 1);
      o.x = pack_bf16x2(b[0], b[1]);   o.y = pack_bf16x2(b[2], b[3]);
      o.z = pack_bf16x2(b[4], b[5]);   o.w = pack_bf16x2(b[6], b[7]);
      __builtin_nontemporal_store(o, db);
      o.x = pack_bf16x2(b[8], b[9]);   o.y = pack_bf16x2(b[10], b[11]);
      o.z = pack_bf16x2(b[12], b[13]); o.w = pack_bf16x2(b[14], b[15]);
      __builtin_nontemporal_store(o, db + 1);
    };
    if (pstride == 2) {
      finish_pair(IntC<0>{}, IntC<2>{});
      finish_pair(IntC<1>{}, IntC<2>{});
    } else {
      finish_pair(IntC<0>{}, IntC<1>{});
      finish_pair(IntC<2>{}, IntC<1>{});
    }
  }
}

}  // namespace

size_t decode_bf16_lds_bytes(int nwc, int rank) {
  const int cn = 128 * nwc;
  return static_cast<size_t>(cn) * (rank + 8) * 2 + static_cast<size_t>(cn) * 2;
}

hipError_t launch_decode_bf16(int nwc, const GemmParams& p, hipStream_t stream) {
  if (p.total_tiles <= 0) return hipSuccess;
  int max_k = 0;
  for (int i = 0; i < p.n_jobs; ++i) max_k = p.jobs[i].k > max_k ? p.jobs[i].k : max_k;
  const size_t lds = decode_bf16_lds_bytes(nwc, max_k);
  if (nwc == 2) {
    hipLaunchKernelGGL(reuse_decode_bf16_kernel<2>, dim3(p.total_tiles), dim3(kThreads), lds,
                       stream, p);
  } else {
    hipLaunchKernelGGL(reuse_decode_bf16_kernel<1>, dim3(p.total_tiles), dim3(kThreads), lds,
                       stream, p);
  }
  return hipGetLastError();
}

}  // namespace scd
