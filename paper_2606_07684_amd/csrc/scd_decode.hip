// Reuse decode (Section 4.3.2, Eq. decode_kv) on the bf16 path for gfx950:
//   K = RoPE(unrows(Z_K W_dec,K^T + mu_K)),  V = unrows(Z_V W_dec,V^T + mu_V)
// written straight into the consumer's KV cache.  The step is bound by HBM writes: every
// reconstructed element is written once and the codes are only r/w of that traffic.
//
// Work decomposition: a launch covers one branch (keys or values) of every layer of one rank, as
// one round of workgroups sized to the machine.  A workgroup owns a channel chunk of NHG x 128
// channels (512 for ranks up to 128: one workgroup of 8 waves per CU, whose basis chunk fills most
// of the LDS) and a contiguous, balanced share of the launch's row tiles, running across layers.
// It copies a layer-branch's basis chunk (CN rows of W_dec, permuted so each MFMA accumulator lane
// ends with 16 consecutive channels of one row) into padded LDS rows with direct global->LDS
// loads when its share enters that layer-branch.  Each wave owns 32 rows of a tile: it loads
// their codes once, then for every 128-channel group runs v_mfma_f32_32x32x16_bf16 (basis as A,
// codes as B), adds the offset, rotates the keys and stores 16-byte vectors.  The waves start
// every tile together, which keeps the workgroup's stores on neighbouring rows.
//
// Why this shape: the step writes ~8x what it reads, and HBM serves that write stream worst when
// reads are interleaved with it and when concurrent stores scatter over many rows.  A 512-channel
// chunk halves the code re-reads of a 256-channel one, the single round and the long shares
// leave almost no per-workgroup set-up (basis copy, waits) on the critical path, and the lockstep
// keeps the stores of a workgroup close together.
//
// RoPE factors are built to need few vector-memory instructions: a row at position p with
// in-half offset d = (lane % 16) uses cos/sin((p - d) w) * cos/sin(d w).  The first factor is
// (nearly) the same row for the 16 lanes of a half-wave, so its loads broadcast; the second comes
// from table rows 0..15 staged once per workgroup in LDS.  Both factors are fp64-evaluated table
// entries; the product in fp32 is within a few ulp of cos/sin(p w).  Codes and factors are reused
// for every channel group.
#include "scd_device.h"

namespace scd {
namespace {

using namespace dev;

// Waves per workgroup: 8 when the basis chunk (128 nhg channels x rank) takes more than half the
// LDS, so one workgroup holds the CU (512 channels up to rank 128, 256 channels above); 4 when
// two workgroups share a CU.  A tile is 32 rows per wave.
constexpr int waves_for(int nhg, int kch) {
  return 128 * nhg * (32 * kch + 8) * 2 > 80 * 1024 ? 8 : 4;
}
constexpr int kDRows = kRopeMinRows;  // in-half offsets d = 0..15

// The layer-branch a workgroup is working on.
struct DecodeCtx {
  const uint16_t* Z;     // codes [M, K]
  uint16_t* C;           // output rows [M, N]
  int64_t M;
  int N, n0;             // row width, first channel of the chunk
  bool silu;             // SiLU after the offset (the aligner's first product; never with RoPE)
};

// One tile: the TT rows from row t0 of the current layer-branch, channels [n0, n0 + 128 NHG).
// KCH = rank / 32, NHG = channel groups of 128, DH = head_dim, ROPE = key jobs, FULL = all TT
// rows exist (only the last tile of a layer-branch can be partial).
template <int KCH, int NHG, int DH, bool ROPE, bool FULL, int TT = 32 * waves_for(NHG, KCH)>
__device__ __forceinline__ void decode_tile(const GemmParams& p, const LdsBatch& lb,
                                            const DecodeCtx& c, int64_t t0, const uint16_t* Fs,
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

  {
    const int64_t row = t0 + wave * 32 + (lane & 31);

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
      // No row guard before the stores: the lane exchange below needs every lane.
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
        if constexpr (!ROPE) {
          if (c.silu) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              a[r] = silu_bf16(a[r]);
              b[r] = silu_bf16(b[r]);
            }
          }
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
        // Lane t and lane t + 16 (t % 32 < 16) swap halves (v_permlane16_swap): lane t keeps its
        // row's channels 0..7 of the 16 and takes row t + 16's, lane t + 16 takes row t's channels
        // 8..15 and keeps its own.  One store instruction then writes 16 rows x 64 contiguous bytes
        // (four lanes per row) instead of 32 rows x two separate 16-byte pieces, which halves the
        // write requests to L2 (32 -> 64 bytes each); the per-CU cache's queue of pending requests
        // was what held the stores back.
        const u32x4 ax = as_u32x4(pack8(a)), ay = as_u32x4(pack8(a + 8));
        const u32x4 bx = as_u32x4(pack8(b)), by = as_u32x4(pack8(b + 8));
        u32x4 alo, ahi, blo, bhi;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const auto sa = __builtin_amdgcn_permlane16_swap(ax[i], ay[i], false, false);
          const auto sb = __builtin_amdgcn_permlane16_swap(bx[i], by[i], false, false);
          alo[i] = sa[0];
          ahi[i] = sa[1];
          blo[i] = sb[0];
          bhi[i] = sb[1];
        }
        const int sub = 8 * ((lane >> 4) & 1);
        const int64_t r0 = t0 + wave * 32 + (lane & 15), r1 = r0 + 16;
        if (FULL || r0 < c.M) {
          *reinterpret_cast<u32x4*>(c.C + r0 * c.N + c.n0 + cl + sub) = alo;
          *reinterpret_cast<u32x4*>(c.C + r0 * c.N + c.n0 + clp + sub) = blo;
        }
        if (FULL || r1 < c.M) {
          *reinterpret_cast<u32x4*>(c.C + r1 * c.N + c.n0 + cl + sub) = ahi;
          *reinterpret_cast<u32x4*>(c.C + r1 * c.N + c.n0 + clp + sub) = bhi;
        }
      }
    }
  }
}

// Work decomposition: every launch covers one branch (keys or values) of every layer of one rank.
// The row tiles of all its layer-branches form one list (layer-major).  Workgroup u works on
// channel chunk u % n_nc of a contiguous, balanced share of that list (all its chunk siblings
// take the same share, on the same XCD), so a launch sized to the machine runs as one round
// with every workgroup busy to the end.  A workgroup stages a layer-branch's basis chunk once,
// when its share enters that layer-branch.
template <int KCH, int NHG, int DH, bool ROPE>
__device__ __forceinline__ void decode_body(const GemmParams& p, uint16_t* lds,
                                            LdsBatch& lbatch) {
  constexpr int kWaves = waves_for(NHG, KCH);
  constexpr int kThreads = 64 * kWaves;
  constexpr int kTT = 32 * kWaves;
  constexpr int CN = 128 * NHG;
  constexpr int K = 32 * KCH;
  constexpr int LDK = K + 8;
  constexpr int HALF = DH / 2;
  constexpr int DSTRIDE = HALF + 2;
  uint16_t* Fs = lds;                                                   // [CN][LDK]
  uint16_t* mus = Fs + CN * LDK;                                        // [CN]
  float2* dtab = reinterpret_cast<float2*>(mus + CN);                   // [kDRows][DSTRIDE]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;

  // workgroup -> (share of the row-tile list, channel chunk); chunk fastest
  const int u = xcd_remap(blockIdx.x, gridDim.x);
  const int N = p.jobs[0].n;  // every job of a launch has the basis width
  const int n_nc = N / CN;
  const int n_share = gridDim.x / n_nc;
  const int share = u / n_nc, nc = u % n_nc;
  const int64_t M = p.m;
  const int64_t tiles_per_job = (M + kTT - 1) / kTT;
  const int64_t n_tiles = tiles_per_job * p.n_jobs;
  const int64_t first = n_tiles * share / n_share, last = n_tiles * (share + 1) / n_share;

  // in-half RoPE factors and the batch -> LDS (once)
  if (ROPE) {
    for (int i = tid; i < kDRows * HALF; i += kThreads) {
      const int r = i / HALF, k = i % HALF;
      dtab[r * DSTRIDE + k] = p.rope[static_cast<int64_t>(r) * HALF + k];
    }
  }
  stage_batch(p, lbatch, tid, kThreads);

  DecodeCtx c;
  c.M = M;
  c.N = N;
  c.n0 = nc * CN;
  int cur = -1;
#pragma unroll 1
  for (int64_t gt = first; gt < last; ++gt) {
    // keep the compiler from hoisting the loop-invariant basis reads into registers across tiles
    asm volatile("" ::: "memory");
    const int j = static_cast<int>(gt / tiles_per_job);
    const int64_t t0 = (gt - static_cast<int64_t>(j) * tiles_per_job) * kTT;
    if (j != cur) {
      // entering a layer-branch: its basis chunk (rows permuted so each MFMA accumulator lane
      // ends with 16 consecutive channels of one row) and offsets -> LDS
      if (cur >= 0) lds_barrier();  // every wave is done reading the previous basis
      const GemmJob& job = p.jobs[j];
      c.Z = static_cast<const uint16_t*>(job.a);
      c.C = static_cast<uint16_t*>(job.c);
      const uint16_t* F = static_cast<const uint16_t*>(job.b);
      const uint16_t* mu = static_cast<const uint16_t*>(job.vec);
      const bool add_mu = (job.flags & kVecOut) != 0 && mu != nullptr;
      c.silu = (job.flags & kSiluOut) != 0;
      dma_rows(Fs, CN, K / 8, LDK / 8, wave, kWaves, lane,
               [&](int rho) { return F + static_cast<int64_t>(c.n0 + row_of_lds(rho)) * K; });
      if (tid < CN / 8) {
        const uint4 v = add_mu ? *reinterpret_cast<const uint4*>(mu + c.n0 + 8 * tid)
                               : make_uint4(0, 0, 0, 0);
        *reinterpret_cast<uint4*>(mus + 8 * tid) = v;
      }
      wait_vmem();
      __syncthreads();
      cur = j;
    } else {
      // start every tile with the other waves of the workgroup, so that their stores go to
      // neighbouring rows at the same time (lone waves drifting apart cost DRAM locality)
      wave_lockstep();
    }
    // one bounds-checked body for full and partial tiles (a second copy of the loop body costs
    // registers)
    decode_tile<KCH, NHG, DH, ROPE, false>(p, lbatch, c, t0, Fs, mus, dtab, lane, wave);
  }
}

template <int KCH, int NHG, int DH, bool ROPE>
__global__ __launch_bounds__(64 * waves_for(NHG, KCH), 2) void reuse_decode_bf16_kernel(
    GemmParams p) {
  extern __shared__ __attribute__((aligned(16))) uint16_t lds[];
  __shared__ LdsBatch lbatch;
  decode_body<KCH, NHG, DH, ROPE>(p, lds, lbatch);
}

// The aligner's first product (act = SiLU(z_h w1^T + b1)) on the same body: a short contraction
// whose time is writing its output, like the Reuse decode; its own symbol so that profiles keep
// the two steps apart.
template <int KCH, int NHG, int DH>
__global__ __launch_bounds__(64 * waves_for(NHG, KCH), 2) void patch_align_act_bf16_kernel(
    GemmParams p) {
  extern __shared__ __attribute__((aligned(16))) uint16_t lds[];
  __shared__ LdsBatch lbatch;
  decode_body<KCH, NHG, DH, false>(p, lds, lbatch);
}

template <int NHG, int DH>
hipError_t launch_align_kch(int kch, const GemmParams& p, int grid_size, size_t lds,
                            hipStream_t stream) {
  switch (kch) {
#define SCD_ALIGN_CASE(KC)                                                                     \
  case KC:                                                                                     \
    hipLaunchKernelGGL((patch_align_act_bf16_kernel<KC, NHG, DH>), dim3(grid_size),           \
                       dim3(64 * waves_for(NHG, KC)), lds, stream, p);                        \
    return hipGetLastError();
    SCD_ALIGN_CASE(1) SCD_ALIGN_CASE(2) SCD_ALIGN_CASE(3) SCD_ALIGN_CASE(4)
    default:
      break;
  }
  // ranks above 128 use at most two channel groups per workgroup (decode_channel_groups)
  if constexpr (NHG <= 2) {
    switch (kch) {
      SCD_ALIGN_CASE(5) SCD_ALIGN_CASE(6) SCD_ALIGN_CASE(7) SCD_ALIGN_CASE(8)
      default:
        break;
    }
  }
#undef SCD_ALIGN_CASE
  return hipErrorInvalidValue;
}

template <int NHG, int DH, bool ROPE>
hipError_t launch_kch(int kch, const GemmParams& p, int grid_size, size_t lds,
                      hipStream_t stream) {
  switch (kch) {
#define SCD_DECODE_CASE(KC)                                                                   \
  case KC:                                                                                    \
    hipLaunchKernelGGL((reuse_decode_bf16_kernel<KC, NHG, DH, ROPE>), dim3(grid_size),       \
                       dim3(64 * waves_for(NHG, KC)), lds, stream, p);                        \
    return hipGetLastError();
    SCD_DECODE_CASE(1) SCD_DECODE_CASE(2) SCD_DECODE_CASE(3) SCD_DECODE_CASE(4)
#undef SCD_DECODE_CASE
    default:
      break;
  }
  // ranks above 128 use at most two channel groups per workgroup (decode_channel_groups)
  if constexpr (NHG <= 2) {
    switch (kch) {
#define SCD_DECODE_CASE(KC)                                                                   \
  case KC:                                                                                    \
    hipLaunchKernelGGL((reuse_decode_bf16_kernel<KC, NHG, DH, ROPE>), dim3(grid_size),       \
                       dim3(64 * waves_for(NHG, KC)), lds, stream, p);                        \
    return hipGetLastError();
      SCD_DECODE_CASE(5) SCD_DECODE_CASE(6) SCD_DECODE_CASE(7) SCD_DECODE_CASE(8)
#undef SCD_DECODE_CASE
      default:
        break;
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace

int decode_channel_groups(int rank, int basis_width) {
  if (rank > 128) return basis_width % 256 == 0 ? 2 : 1;
  return basis_width % 512 == 0 ? 4 : (basis_width % 256 == 0 ? 2 : 1);
}

int decode_tile_rows(int nhg, int rank) { return 32 * waves_for(nhg, (rank + 31) / 32); }

// Compute units of the current device (queried once per device).
static hipError_t compute_units(int* out) {
  static int cache[64] = {0};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev >= 0 && dev < 64 && cache[dev] > 0) {
    *out = cache[dev];
    return hipSuccess;
  }
  int n = 0;
  e = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  if (n < 1) n = 1;
  if (dev >= 0 && dev < 64) cache[dev] = n;
  *out = n;
  return hipSuccess;
}

size_t decode_bf16_lds_bytes(int nhg, int rank, int head_dim) {
  const size_t cn = 128 * static_cast<size_t>(nhg);
  return cn * (rank + 8) * 2 + cn * 2 + static_cast<size_t>(kDRows) * (head_dim / 2 + 2) * 8;
}

hipError_t launch_decode_bf16(int nhg, const GemmParams& p, hipStream_t stream, bool align) {
  if (p.total_tiles <= 0) return hipSuccess;
  // every job of a launch has the same rank and branch
  const int rank = p.jobs[0].k;
  const bool rope = (p.jobs[0].flags & kRopeOut) != 0;
  for (int i = 1; i < p.n_jobs; ++i)
    if (p.jobs[i].k != rank || ((p.jobs[i].flags & kRopeOut) != 0) != rope)
      return hipErrorInvalidValue;
  const int cn = 128 * nhg;
  if (rank % 32 != 0 || rank < 32 || rank > 256 || p.n_seqs > kMaxLdsSeqs || p.n_jobs < 1 ||
      p.jobs[0].n % cn != 0)
    return hipErrorInvalidValue;
  for (int i = 1; i < p.n_jobs; ++i)
    if (p.jobs[i].n != p.jobs[0].n) return hipErrorInvalidValue;
  const size_t lds = decode_bf16_lds_bytes(nhg, rank, p.head_dim);
  const int kch = rank / 32;
  // one round of workgroups: as many as the compute units hold at once (LDS and the two waves per
  // SIMD the kernel is built for), in whole sets of channel-chunk siblings, at most one set per
  // row tile
  int cus = 0;
  const hipError_t e = compute_units(&cus);
  if (e != hipSuccess) return e;
  const int waves = waves_for(nhg, kch);
  const size_t lds_per_wg = lds + sizeof(LdsBatch);
  int per_cu = static_cast<int>((160 * 1024) / lds_per_wg);
  per_cu = per_cu < 8 / waves ? per_cu : 8 / waves;
  per_cu = per_cu < 1 ? 1 : per_cu;
  const int n_nc = p.jobs[0].n / cn;
  const int64_t tile_rows = 32 * waves;
  const int64_t row_tiles = (p.m + tile_rows - 1) / tile_rows * p.n_jobs;
  int64_t shares = static_cast<int64_t>(cus) * per_cu / n_nc;
  shares = shares < 1 ? 1 : (shares > row_tiles ? row_tiles : shares);
  const int grid_size = static_cast<int>(shares * n_nc);
  if (align && rope) return hipErrorInvalidValue;
#define SCD_DECODE_DISPATCH(NHG, DH)                                                    \
  if (nhg == NHG && p.head_dim == DH)                                                   \
    return align  ? launch_align_kch<NHG, DH>(kch, p, grid_size, lds, stream)           \
           : rope ? launch_kch<NHG, DH, true>(kch, p, grid_size, lds, stream)           \
                  : launch_kch<NHG, DH, false>(kch, p, grid_size, lds, stream);
  SCD_DECODE_DISPATCH(4, 128)
  SCD_DECODE_DISPATCH(2, 128)
  SCD_DECODE_DISPATCH(1, 128)
  SCD_DECODE_DISPATCH(4, 64)
  SCD_DECODE_DISPATCH(2, 64)
  SCD_DECODE_DISPATCH(1, 64)
#undef SCD_DECODE_DISPATCH
  return hipErrorInvalidValue;
}

}  // namespace scd
