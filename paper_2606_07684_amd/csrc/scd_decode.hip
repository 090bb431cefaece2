// Reuse decode (Section 4.3.2, Eq. decode_kv) on the bf16 path for gfx950:
//   K = RoPE(unrows(Z_K W_dec,K^T + mu_K)),  V = unrows(Z_V W_dec,V^T + mu_V)
// written straight into the consumer's KV cache.  The step is bound by HBM writes: every
// reconstructed element is written once and the codes are only r/w of that traffic.
//
// Work unit: NHG groups of 128 channels (CN = 128 * NHG) of one layer-branch x a group of
// tiles of 128 rows.  The workgroup copies its basis chunk (CN rows of W_dec, permuted so each
// MFMA accumulator lane ends with 16 consecutive channels of one row) into padded LDS rows with
// direct global->LDS loads.  Each of its 4 waves owns 32 rows of a tile: it loads their codes
// once, then for every 128-channel group runs v_mfma_f32_32x32x16_bf16 (basis as A, codes as
// B), adds the offset, rotates the keys and stores 16-byte vectors.
//
// Vector-memory instructions whose 64 lanes touch many cache lines are what limits this step, so
// the RoPE factors are built to need few of them: a row at position p with in-half offset
// d = (lane % 16) uses cos/sin((p - d) w) * cos/sin(d w).  The first factor is (nearly) the same
// row for the 16 lanes of a half-wave, so its loads broadcast; the second comes from table rows
// 0..15 staged once per workgroup in LDS.  Both factors are fp64-evaluated table entries; the
// product in fp32 is within a few ulp of cos/sin(p w).  Codes and factors are reused for every
// channel group.
#include "scd_device.h"

namespace scd {
namespace {

using namespace dev;

constexpr int kThreads = 256;
constexpr int kTT = kDecodeTileRows;  // rows per tile (4 waves x 32)
constexpr int kDRows = kRopeMinRows;  // in-half offsets d = 0..15

// Per-workgroup context of the decode kernel.
struct DecodeCtx {
  const uint16_t* Z;     // codes [M, K]
  uint16_t* C;           // output rows [M, N]
  int64_t M;
  int N, n0;             // row width, first channel of the chunk
  int64_t row_first;     // first row of the unit
  int n_tiles;           // tiles of the unit
};

// KCH = rank / 32, NHG = channel groups of 128, DH = head_dim, ROPE = key jobs, FULL = every
// tile of the unit is complete (only the last unit of a layer-branch can be partial).
template <int KCH, int NHG, int DH, bool ROPE, bool FULL>
__device__ __forceinline__ void decode_unit(const GemmParams& p, const LdsBatch& lb,
                                            const DecodeCtx& c, const uint16_t* Fs,
                                            const uint16_t* mus, const float2* dtab, int lane,
                                            int wave) {
  constexpr int K = 32 * KCH;
  constexpr int LDK = K + 8;
  constexpr int HALF = DH / 2;
  constexpr int PS = HALF / 32;  // blocks between RoPE partners: 2 (d_h 128) or 1 (d_h 64)
  constexpr int DSTRIDE = HALF + 2;  // padded LDS row of the in-half factor table (float2)
  const int h = lane >> 5;
  const int hl = 16 * h;
  const int d = lane & 15;

#pragma unroll 1
  for (int tile = 0; tile < c.n_tiles; ++tile) {
    // keep the compiler from hoisting loop-invariant LDS reads into registers across tiles
    asm volatile("" ::: "memory");
    // start every tile with the other waves of the workgroup, so that their stores go to
    // neighbouring rows at the same time (lone waves drifting apart cost DRAM locality)
    if (tile > 0) wave_lockstep();
    const int64_t row = c.row_first + static_cast<int64_t>(tile) * kTT + wave * 32 + (lane & 31);
    if (!FULL && c.row_first + static_cast<int64_t>(tile) * kTT >= c.M) break;  // uniform

    // codes: lane half h holds k = 16i + 8h + (0..7); rows past the end read row 0 (in bounds,
    // never stored)
    uint4 z[2 * KCH];
    {
      const uint16_t* zr = c.Z + (row < c.M ? row : 0) * K + 8 * h;
#pragma unroll
      for (int i = 0; i < 2 * KCH; ++i) z[i] = *reinterpret_cast<const uint4*>(zr + 16 * i);
    }

    // RoPE factors of this row for its pair indices i0(q) + r, q = 0, 1
    float2 cs[2][16];
    if constexpr (ROPE) {
      const int pos = row < c.M ? row_position_lds(p, lb, row) : d;
      const int base = pos - d;
      const float sgn = base < 0 ? -1.f : 1.f;  // cos/sin(-x) = (cos x, -sin x)
      const float2* brow = p.rope + static_cast<int64_t>(base < 0 ? -base : base) * HALF;
      const float2* drow = dtab + d * DSTRIDE;
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const int i0 = (32 * (PS == 2 ? q : 2 * q) + hl) & (HALF - 1);
#pragma unroll
        for (int r = 0; r < 16; r += 2) {
          const float4 b = *reinterpret_cast<const float4*>(brow + i0 + r);
          const float4 e = *reinterpret_cast<const float4*>(drow + i0 + r);
          const float bs0 = sgn * b.y, bs1 = sgn * b.w;
          cs[q][r] = make_float2(b.x * e.x - bs0 * e.y, bs0 * e.x + b.x * e.y);
          cs[q][r + 1] = make_float2(b.z * e.z - bs1 * e.w, bs1 * e.z + b.z * e.w);
        }
      }
    }

#pragma unroll
    for (int g = 0; g < NHG; ++g) {
      const uint16_t* fw = Fs + (g * 128 + (lane & 31)) * LDK + 8 * h;
      f32x16 acc[4];
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[s][e] = 0.f;
#pragma unroll
      for (int i = 0; i < 2 * KCH; ++i) {
        const bf16x8 bz = __builtin_bit_cast(bf16x8, z[i]);
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          const bf16x8 af = *reinterpret_cast<const bf16x8*>(fw + s * 32 * LDK + 16 * i);
          acc[s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, bz, acc[s], 0, 0, 0);
        }
      }
      if (FULL || row < c.M) {
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const int S = PS == 2 ? q : 2 * q;  // first-half block; its partner is S + PS
          const int cl = g * 128 + 32 * S + hl, clp = cl + 32 * PS;  // local channels
          float a[16], b[16];
#pragma unroll
          for (int k = 0; k < 2; ++k) {
            unpack8(*reinterpret_cast<const uint4*>(mus + cl + 8 * k), a + 8 * k);
            unpack8(*reinterpret_cast<const uint4*>(mus + clp + 8 * k), b + 8 * k);
          }
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            a[r] += acc[S][r];
            b[r] += acc[S + PS][r];
          }
          if constexpr (ROPE) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const float2 f = cs[q][r];
              const float x = a[r], y = b[r];
              a[r] = x * f.x - y * f.y;
              b[r] = y * f.x + x * f.y;
            }
          }
          u32x4* da = reinterpret_cast<u32x4*>(c.C + row * c.N + c.n0 + cl);
          u32x4* db = reinterpret_cast<u32x4*>(c.C + row * c.N + c.n0 + clp);
          da[0] = as_u32x4(pack8(a));
          da[1] = as_u32x4(pack8(a + 8));
          db[0] = as_u32x4(pack8(b));
          db[1] = as_u32x4(pack8(b + 8));
        }
      }
    }
  }
}

template <int KCH, int NHG, int DH, bool ROPE>
__global__ __launch_bounds__(kThreads, 2) void reuse_decode_bf16_kernel(GemmParams p) {
  constexpr int CN = 128 * NHG;
  constexpr int K = 32 * KCH;
  constexpr int LDK = K + 8;
  constexpr int HALF = DH / 2;
  constexpr int DSTRIDE = HALF + 2;
  extern __shared__ __attribute__((aligned(16))) uint16_t lds[];
  __shared__ LdsBatch lbatch;
  uint16_t* Fs = lds;                                                   // [CN][LDK]
  uint16_t* mus = Fs + CN * LDK;                                        // [CN]
  float2* dtab = reinterpret_cast<float2*>(mus + CN);                   // [kDRows][DSTRIDE]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;

  // unit -> (job, row group, channel chunk); channel chunk fastest
  const int unit = xcd_remap(blockIdx.x, gridDim.x);
  const GemmJob job = p.jobs[job_of(p, unit)];
  const int n_nc = job.n / CN;
  const int local = unit - job.tile_begin;
  const int nc = local % n_nc, tg = local / n_nc;
  const int tiles_per_unit = p.tiles_per_unit;

  DecodeCtx c;
  c.Z = static_cast<const uint16_t*>(job.a);
  c.C = static_cast<uint16_t*>(job.c);
  c.M = p.m;
  c.N = job.n;
  c.n0 = nc * CN;
  c.row_first = static_cast<int64_t>(tg) * tiles_per_unit * kTT;
  c.n_tiles = tiles_per_unit;
  const uint16_t* F = static_cast<const uint16_t*>(job.b);
  const uint16_t* mu = static_cast<const uint16_t*>(job.vec);
  const bool add_mu = (job.flags & kVecOut) != 0 && mu != nullptr;

  // basis chunk -> LDS (asynchronous); offsets, in-half RoPE factors and the batch -> LDS
  dma_rows(Fs, CN, K / 8, LDK / 8, wave, 4, lane,
           [&](int rho) { return F + static_cast<int64_t>(c.n0 + row_of_lds(rho)) * K; });
  if (tid < CN / 8) {
    const uint4 v = add_mu ? *reinterpret_cast<const uint4*>(mu + c.n0 + 8 * tid)
                           : make_uint4(0, 0, 0, 0);
    *reinterpret_cast<uint4*>(mus + 8 * tid) = v;
  }
  if (ROPE) {
    for (int i = tid; i < kDRows * HALF; i += kThreads) {
      const int r = i / HALF, k = i % HALF;
      dtab[r * DSTRIDE + k] = p.rope[static_cast<int64_t>(r) * HALF + k];
    }
  }
  stage_batch(p, lbatch, tid, kThreads);
  wait_vmem();
  __syncthreads();

  if (c.row_first + static_cast<int64_t>(tiles_per_unit) * kTT <= c.M)
    decode_unit<KCH, NHG, DH, ROPE, true>(p, lbatch, c, Fs, mus, dtab, lane, wave);
  else
    decode_unit<KCH, NHG, DH, ROPE, false>(p, lbatch, c, Fs, mus, dtab, lane, wave);
}

template <int NHG, int DH, bool ROPE>
hipError_t launch_kch(int kch, const GemmParams& p, size_t lds, hipStream_t stream) {
  const dim3 grid(p.total_tiles), block(kThreads);
  switch (kch) {
#define SCD_DECODE_CASE(KC)                                                                   \
  case KC:                                                                                    \
    hipLaunchKernelGGL((reuse_decode_bf16_kernel<KC, NHG, DH, ROPE>), grid, block, lds, stream, \
                       p);                                                                    \
    break;
    SCD_DECODE_CASE(1) SCD_DECODE_CASE(2) SCD_DECODE_CASE(3) SCD_DECODE_CASE(4)
    SCD_DECODE_CASE(5) SCD_DECODE_CASE(6) SCD_DECODE_CASE(7) SCD_DECODE_CASE(8)
#undef SCD_DECODE_CASE
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

int decode_channel_groups(int rank, int basis_width) {
  return (rank <= 128 && basis_width % 256 == 0) ? 2 : 1;
}

size_t decode_bf16_lds_bytes(int nhg, int rank, int head_dim) {
  const size_t cn = 128 * static_cast<size_t>(nhg);
  return cn * (rank + 8) * 2 + cn * 2 + static_cast<size_t>(kDRows) * (head_dim / 2 + 2) * 8;
}

hipError_t launch_decode_bf16(int nhg, const GemmParams& p, hipStream_t stream) {
  if (p.total_tiles <= 0) return hipSuccess;
  // every job of a launch has the same rank and branch
  const int rank = p.jobs[0].k;
  const bool rope = (p.jobs[0].flags & kRopeOut) != 0;
  for (int i = 1; i < p.n_jobs; ++i)
    if (p.jobs[i].k != rank || ((p.jobs[i].flags & kRopeOut) != 0) != rope)
      return hipErrorInvalidValue;
  if (rank % 32 != 0 || rank < 32 || rank > 256 || p.n_seqs > kMaxLdsSeqs ||
      p.tiles_per_unit < 1)
    return hipErrorInvalidValue;
  const size_t lds = decode_bf16_lds_bytes(nhg, rank, p.head_dim);
  const int kch = rank / 32;
#define SCD_DECODE_DISPATCH(NHG, DH)                                                    \
  if (nhg == NHG && p.head_dim == DH)                                                   \
    return rope ? launch_kch<NHG, DH, true>(kch, p, lds, stream)                        \
                : launch_kch<NHG, DH, false>(kch, p, lds, stream);
  SCD_DECODE_DISPATCH(2, 128)
  SCD_DECODE_DISPATCH(1, 128)
  SCD_DECODE_DISPATCH(2, 64)
  SCD_DECODE_DISPATCH(1, 64)
#undef SCD_DECODE_DISPATCH
  return hipErrorInvalidValue;
}

}  // namespace scd
