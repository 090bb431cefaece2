// Offline Reuse fit of the SCD codec (Section 4.3.1 "Joint Subspace Learning"; Appendix F.1
// "Reuse: Layer-wise Stack-SVD with Ridge Regression").
//
// For one branch (keys or values) of every Reuse layer, the producer's and the consumer's caches of
// the same calibration prefixes give rows A, B [N, w] (keys de-rotated first).  The fit needs only
// the joint Gram G = X^T X of X = [A B] (2w x 2w) and the column sums 1^T X:
//   * the truncated SVD of the (centred) X is the eigendecomposition of the (centred) G, whose top-r
//     eigenvectors V_r give the latents Z = X V_r;
//   * the ridge encoder E = (A^T A + lam I)^-1 A^T Z needs A^T A and A^T Z = G[0:w, :] V_r;
//   * the ridge decoder F = (Z^T Z + lam I)^-1 Z^T B needs Z^T Z = V_r^T G V_r and
//     Z^T B = (G[w:2w, :] V_r)^T.
// The O(N w^2) part (the Gram) streams the caches once on the matrix cores; the O(w^3) part runs in
// fp64 as a sequence of launches over all layers at once (Householder tridiagonalisation,
// bisection and inverse iteration for the top r eigenpairs, Cholesky solves).
#include "scd_device.h"

#include <mutex>

namespace scd {

using namespace dev;

// Device-resident scratch of the allocation-free solve (scd_fit_solve_noalloc): the solve's fp64
// matrices for as many layers as fit, reused launch after launch.  Each GPU the
// library runs on holds its own copy for the life of the process.  Host code must never pass this
// name to a kernel (in host code it is a stand-in, not a device address): fit_scratch() looks up
// the device address once per device.
static __device__ __align__(256) double scratch[kFitScratchBytes / sizeof(double)];

namespace {

constexpr int kTB = kFitTile;
constexpr int kTileFloats = kTB * kTB + kTB;  // one partial tile: Gram block + column sums

__device__ inline int fit_position(const FitGramParams& p, int64_t row) {
  const int64_t t = row / p.g;
  int b = 0;
  int64_t local = t;
  if (p.cu_seqlens != nullptr) {
    int lo = 0, hi = p.n_seqs - 1;  // largest b with cu[b] <= t
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

// Upper tiles (ti <= tj) of the nt x nt tile grid, numbered row by row.
__device__ inline void tile_of(int tile, int nt, int& ti, int& tj) {
  int rem = tile;
  ti = 0;
  while (rem >= nt - ti) {
    rem -= nt - ti;
    ++ti;
  }
  tj = ti + rem;
}

// First column (inside a 128-column block) of chunk pair cp: VEC columns of one head's first half;
// their RoPE partners sit d_h/2 further on.  A block holds 128 / d_h heads of d_h / (2 VEC) pairs.
template <int DH, int VEC>
__device__ inline int pair_col(int cp) {
  constexpr int PER_HEAD = DH / 2 / VEC;
  return (cp / PER_HEAD) * DH + (cp % PER_HEAD) * VEC;
}

// Loads through the global address space.  The row pointers come out of the job table through a
// select between two sources, which hides their address space from the compiler; as generic (flat)
// loads they would also count against the LDS counter, so every LDS wait would drain them.
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) const u32x4 g_u32x4;
typedef __attribute__((address_space(1))) const f32x4 g_f32x4;
__device__ inline uint4 gload16(const char* p) {
  const u32x4 v = *(g_u32x4*)(p);
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ inline float4 gload_f4(const float2* p) {
  const f32x4 v = *(g_f32x4*)(p);
  return make_float4(v.x, v.y, v.z, v.w);
}

// Column sums of a staged dword (two bf16 values of one column): acc + lo + hi in one dot product.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ inline float add_bf16_pair(uint32_t v, float acc) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, v),
                                         __builtin_bit_cast(bf16x2_t, 0x3f803f80u), acc, false);
}

struct BlockSrc {
  const char* base;  // producer or consumer cache
  int col;           // column inside the w-wide row
};

// Source of the chunk pair starting at joint column jc (< 2w): columns [0, w) are the producer's,
// [w, 2w) the consumer's.  A head never straddles the two (w is a multiple of d_h).
__device__ inline BlockSrc block_src(const FitGramJob& j, int w, int jc, int eb) {
  BlockSrc s;
  s.base = static_cast<const char*>(jc < w ? j.a : j.b);
  s.col = (jc < w ? jc : jc - w) * eb;
  return s;
}

// ---------------------------------------------------------------------------------------------
// bf16 Gram: one workgroup of 4 waves per (job, upper 128 x 128 tile, row slice).  Each k-step
// stages 64 rows of the tile's two column blocks transposed in LDS ([column][row], so an MFMA
// operand fragment is 8 consecutive rows of one column) and runs v_mfma_f32_32x32x16_bf16 with the
// I block as A and the J block as B: C[m][n] = sum_rows X[row][I0+m] X[row][J0+n].  Keys are
// de-rotated in registers and rounded to bf16 once before the product (as the encoder does).
// Thread t stages row pair t % 32 and chunk pair t / 32 (8 columns + their RoPE partners).
//
// The step is bound by HBM latency, so rows travel two k-steps ahead in two register sets and the
// RoPE factors one step ahead; each is issued before the far data prefetch, so the in-order
// vector-memory counter never makes a step wait for rows it does not use yet.  The LDS tiles are
// double-buffered, which leaves one barrier per step, and that barrier waits for LDS only.
// PAIR: both rows of a thread's pair belong to one token (g even), so they share RoPE factors.
// ---------------------------------------------------------------------------------------------
//
// FULL (2w = 256 only): one workgroup owns the whole Gram of its (job, slice), so every row is read
// once.  Its two column blocks are the producer's (A) and the consumer's (B) columns; each wave
// computes one 128 x 128 tile (AA, AB, BB, and the mirror BA, which keeps the code uniform and is
// not stored), so a 64-row step is 64 MFMAs per wave against 32 KB of rows: about HBM speed.  The
// partial tiles keep the tile kernel's layout (AA, AB, BB), so the slice reduction is shared.
template <int DH, bool DEROPE, bool PAIR, bool FULL>
__device__ __forceinline__ void fit_gram_bf16_body(const FitGramParams& p) {
  constexpr int BK = kFitRowStep, S = BK + 8, HALF = DH / 2, NR = PAIR ? 1 : 2;
  constexpr int NA = FULL ? 4 : 2;  // accumulator blocks per wave and dimension
  __shared__ __attribute__((aligned(16))) uint16_t xt[2][2][kTB * S];  // [stage][block]

  const int nt = 2 * p.w / kTB, n_upper = nt * (nt + 1) / 2;
  // the tiles of one (job, slice) read the same rows: consecutive units on one XCD, so the second
  // read of a column block hits that XCD's L2
  int unit = xcd_remap(blockIdx.x, gridDim.x);
  const int tile = FULL ? 0 : unit % n_upper;
  if (!FULL) unit /= n_upper;
  const int slice = unit % p.n_slices;
  const int job = unit / p.n_slices;
  int ti = 0, tj = 1;
  if (!FULL) tile_of(tile, nt, ti, tj);
  const bool diag = ti == tj;
  const int nblk = diag ? 1 : 2;
  const FitGramJob& jb = p.jobs[job];
  const int64_t r0 = static_cast<int64_t>(slice) * p.slice_rows;
  const int64_t r1 = r0 + p.slice_rows < p.n_rows ? r0 + p.slice_rows : p.n_rows;
  const int64_t row_bytes = static_cast<int64_t>(p.w) * 2;
  const int tj_src = diag ? ti : tj;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // eight consecutive lanes cover the eight chunk pairs of one row pair: a load instruction reads
  // 8 rows x 128 contiguous bytes
  const int cp = tid & 7, rp = tid >> 3;
  const int c = pair_col<DH, 8>(cp);
  const int ri = c % DH;  // RoPE pair index of the first column (< d_h / 2)
  BlockSrc src[2];
  src[0] = block_src(jb, p.w, ti * kTB + c, 2);
  src[1] = block_src(jb, p.w, tj_src * kTB + c, 2);

  uint4 la[2][2][2], lb[2][2][2];  // [block][row of the pair][first half / partner]
  float4 rc[NR][4];                // RoPE (cos, sin) of the next step's rows, pairs ri .. ri+7
  constexpr int NCS = FULL ? 32 : 16;  // column sums kept: one or both blocks
  float csum[NCS];
#pragma unroll
  for (int i = 0; i < NCS; ++i) csum[i] = 0.f;
  f32x16 acc[NA][NA];
#pragma unroll
  for (int i = 0; i < NA; ++i)
#pragma unroll
    for (int j = 0; j < NA; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  const uint4 zero4 = make_uint4(0, 0, 0, 0);
  // Every step issues the same loads on every path (rows past the slice read its last row and are
  // zeroed when staged; a diagonal tile's J block re-reads its I block from L1/L2), so the
  // compiler's counter waits can leave the far prefetch in flight.
  auto issue_rows = [&](uint4 (&ld)[2][2][2], int64_t k0) {
#pragma unroll
    for (int rr = 0; rr < 2; ++rr) {
      int64_t n = k0 + 2 * rp + rr;
      n = n < r1 ? n : r1 - 1;
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const char* rowp = src[b].base + n * row_bytes + src[b].col;
        ld[b][rr][0] = gload16(rowp);
        ld[b][rr][1] = gload16(rowp + HALF * 2);
      }
    }
  };
  auto issue_rope = [&](int64_t k0) {
    if constexpr (DEROPE) {
#pragma unroll
      for (int q = 0; q < NR; ++q) {
        const int64_t n = k0 + 2 * rp + q;
        const float2* tab = p.rope + static_cast<int64_t>(n < r1 ? fit_position(p, n) : 0) * HALF + ri;
#pragma unroll
        for (int j = 0; j < 4; ++j) rc[q][j] = gload_f4(tab + 2 * j);
      }
    }
  };
  // de-rotate (keys), round, and write one k-step's rows into LDS stage sb; accumulate the diagonal
  // tile's column sums
  auto stage = [&](const uint4 (&ld)[2][2][2], int64_t k0, int sb) {
    if constexpr (!DEROPE) {
      // values: the staged dword of column j is the j-th bf16 of row 2rp (low half) and of row
      // 2rp + 1 (high half): one byte permute per dword, no conversions
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        if (b >= nblk) break;
        uint32_t* dst = reinterpret_cast<uint32_t*>(xt[sb][b]);
        const bool live0 = k0 + 2 * rp < r1, live1 = k0 + 2 * rp + 1 < r1;
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const uint4 a0 = live0 ? ld[b][0][q] : zero4, a1 = live1 ? ld[b][1][q] : zero4;
          const uint32_t w0[4] = {a0.x, a0.y, a0.z, a0.w}, w1[4] = {a1.x, a1.y, a1.z, a1.w};
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const uint32_t v = __builtin_amdgcn_perm(w1[j >> 1], w0[j >> 1],
                                                     (j & 1) ? 0x07060302u : 0x05040100u);
            if (FULL) csum[16 * b + 8 * q + j] = add_bf16_pair(v, csum[16 * b + 8 * q + j]);
            else if (b == 0 && diag) csum[8 * q + j] = add_bf16_pair(v, csum[8 * q + j]);
            const int col = c + q * HALF + j;
            dst[col * (S / 2) + ((((rp >> 2) ^ (col >> 3)) & 7) << 2) + (rp & 3)] = v;
          }
        }
      }
      return;
    }
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      if (b >= nblk) break;
      float f[2][2][8];
#pragma unroll
      for (int rr = 0; rr < 2; ++rr) {
        const bool live = k0 + 2 * rp + rr < r1;
        unpack8(live ? ld[b][rr][0] : zero4, f[rr][0]);
        unpack8(live ? ld[b][rr][1] : zero4, f[rr][1]);
        if constexpr (DEROPE) {
          const int q = PAIR ? 0 : rr;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float4 cs = rc[q][j];
            const float u0 = f[rr][0][2 * j], v0 = f[rr][1][2 * j];
            const float u1 = f[rr][0][2 * j + 1], v1 = f[rr][1][2 * j + 1];
            // inverse rotation by the position's angle
            f[rr][0][2 * j] = u0 * cs.x + v0 * cs.y;
            f[rr][1][2 * j] = v0 * cs.x - u0 * cs.y;
            f[rr][0][2 * j + 1] = u1 * cs.z + v1 * cs.w;
            f[rr][1][2 * j + 1] = v1 * cs.z - u1 * cs.w;
          }
        }
      }
      uint32_t* dst = reinterpret_cast<uint32_t*>(xt[sb][b]);
#pragma unroll
      for (int q = 0; q < 2; ++q)
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const uint32_t v = pack_bf16x2(f[0][q][j], f[1][q][j]);  // rows 2rp (low), 2rp+1 (high)
          if (FULL) csum[16 * b + 8 * q + j] = add_bf16_pair(v, csum[16 * b + 8 * q + j]);
          else if (b == 0 && diag) csum[8 * q + j] = add_bf16_pair(v, csum[8 * q + j]);
          const int col = c + q * HALF + j;
          dst[col * (S / 2) + ((((rp >> 2) ^ (col >> 3)) & 7) << 2) + (rp & 3)] = v;
        }
    }
  };

  const int wy = wave >> 1, wx = wave & 1;
  const int h = lane >> 5;
  // LDS tile layout: row group kg (8 rows) of column col sits at slot kg ^ ((col >> 3) & 7) of the
  // column's padded row, so neither the transposed writes nor the fragment reads conflict
  const int jblk = diag ? 0 : 1;
  auto frag = [&](const uint16_t* base, int col, int kg) {
    return *reinterpret_cast<const bf16x8*>(base + col * S + (((kg ^ (col >> 3)) & 7) << 3));
  };
  // FULL: waves 0..3 multiply (A block, B block) = (0,0), (0,1), (1,1), (1,0): tiles AA, AB, BB
  // and the mirror BA, which is not stored
  const int fa_blk = (wave == 2 || wave == 3) ? 1 : 0;
  const int fb_blk = (wave == 1 || wave == 2) ? 1 : 0;
  auto products = [&](int sb) {
    if constexpr (FULL) {
#pragma unroll
      for (int ks = 0; ks < BK / 16; ++ks) {
        bf16x8 fa[4], fb[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          fa[i] = frag(xt[sb][fa_blk], i * 32 + (lane & 31), 2 * ks + h);
          fb[i] = frag(xt[sb][fb_blk], i * 32 + (lane & 31), 2 * ks + h);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int ks = 0; ks < BK / 16; ++ks) {
        bf16x8 fa[2], fb[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          fa[i] = frag(xt[sb][0], wy * 64 + i * 32 + (lane & 31), 2 * ks + h);
          fb[i] = frag(xt[sb][jblk], wx * 64 + i * 32 + (lane & 31), 2 * ks + h);
        }
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
      }
    }
  };

  // prologue: rows of steps 0 and 1 in flight, RoPE of step 0 ahead of the step-1 rows.  Steps run
  // in pairs; a slice with an odd step count ends with a step of zeroed rows.
  // The scheduling fences keep each group of loads in issue order, so that the counter waits of a
  // step cover its own rows only.
  issue_rows(la, r0);
  __builtin_amdgcn_sched_barrier(0);
  issue_rope(r0);
  __builtin_amdgcn_sched_barrier(0);
  issue_rows(lb, r0 + BK);
  __builtin_amdgcn_sched_barrier(0);
  for (int64_t k0 = r0; k0 < r1; k0 += 2 * BK) {
    stage(la, k0, 0);
    __builtin_amdgcn_sched_barrier(0);
    issue_rope(k0 + BK);
    __builtin_amdgcn_sched_barrier(0);
    issue_rows(la, k0 + 2 * BK);
    __builtin_amdgcn_sched_barrier(0);
    lds_barrier();
    products(0);
    __builtin_amdgcn_sched_barrier(0);
    stage(lb, k0 + BK, 1);
    __builtin_amdgcn_sched_barrier(0);
    issue_rope(k0 + 2 * BK);
    __builtin_amdgcn_sched_barrier(0);
    issue_rows(lb, k0 + 3 * BK);
    __builtin_amdgcn_sched_barrier(0);
    lds_barrier();
    products(1);
    __builtin_amdgcn_sched_barrier(0);
  }

  float* out = p.partial + ((static_cast<int64_t>(job) * p.n_slices + slice) * n_upper + tile) *
                               static_cast<int64_t>(kTileFloats);
  if constexpr (FULL) {
    // waves 0, 1, 2 hold tiles AA, AB, BB (tile indices 0, 1, 2); wave 3's BA is the mirror of AB
    if (wave < 3) {
      float* to = out + wave * static_cast<int64_t>(kTileFloats);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int m = i * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
            const int n = j * 32 + (lane & 31);
            to[m * kTB + n] = acc[i][j][r];
          }
    }
  } else {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int m = wy * 64 + i * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
          const int n = wx * 64 + j * 32 + (lane & 31);
          out[m * kTB + n] = acc[i][j][r];
        }
  }
  if (FULL) {
    // both blocks' column sums: block 0 is tile AA's, block 1 tile BB's
#pragma unroll
    for (int i = 0; i < 32; ++i)
#pragma unroll
      for (int o = 8; o <= 32; o <<= 1) csum[i] += __shfl_xor(csum[i], o, 64);
    __syncthreads();
    float* red = reinterpret_cast<float*>(&xt[0][0][0]);  // [wave][cp][32]
    if (lane < 8) {
#pragma unroll
      for (int i = 0; i < 32; ++i) red[(wave * 8 + cp) * 32 + i] = csum[i];
    }
    __syncthreads();
    {
      const int pc = tid >> 5, i = tid & 31;  // 8 chunk pairs x 32 sums
      const float v = red[(0 * 8 + pc) * 32 + i] + red[(1 * 8 + pc) * 32 + i] +
                      red[(2 * 8 + pc) * 32 + i] + red[(3 * 8 + pc) * 32 + i];
      const int b = i >> 4, e = i & 15;
      const int cc = pair_col<DH, 8>(pc) + (e >> 3) * HALF + (e & 7);
      out[(b == 0 ? 0 : 2) * static_cast<int64_t>(kTileFloats) + kTB * kTB + cc] = v;
    }
  } else if (diag) {
    // a chunk pair's rows are spread over the lanes tid % 8 == cp of every wave: reduce in the
    // wave, then over the four waves through LDS (the tiles are no longer read)
#pragma unroll
    for (int i = 0; i < 16; ++i)
#pragma unroll
      for (int o = 8; o <= 32; o <<= 1) csum[i] += __shfl_xor(csum[i], o, 64);
    __syncthreads();
    float* red = reinterpret_cast<float*>(&xt[0][0][0]);  // [wave][cp][16]
    if (lane < 8) {
#pragma unroll
      for (int i = 0; i < 16; ++i) red[(wave * 8 + cp) * 16 + i] = csum[i];
    }
    __syncthreads();
    if (tid < 8 * 16) {
      const int pc = tid >> 4, i = tid & 15;
      const float v = red[(0 * 8 + pc) * 16 + i] + red[(1 * 8 + pc) * 16 + i] +
                      red[(2 * 8 + pc) * 16 + i] + red[(3 * 8 + pc) * 16 + i];
      const int cc = pair_col<DH, 8>(pc) + (i >> 3) * HALF + (i & 7);
      out[kTB * kTB + cc] = v;
    }
  }
}

template <int DH, bool DEROPE, bool PAIR>
__global__ __launch_bounds__(256, 2) void fit_gram_bf16_kernel(const FitGramParams p) {
  fit_gram_bf16_body<DH, DEROPE, PAIR, false>(p);
}

template <int DH, bool DEROPE, bool PAIR>
__global__ __launch_bounds__(256, 1) void fit_gram_full_bf16_kernel(const FitGramParams p) {
  fit_gram_bf16_body<DH, DEROPE, PAIR, true>(p);
}

// ---------------------------------------------------------------------------------------------
// fp32 Gram on the vector units (the fp32 path takes no reduced-precision products): 16-row
// k-steps staged row-major in LDS, each thread accumulates an 8 x 8 block of the tile.  Thread t
// stages row t % 16 and chunk pair t / 16 (4 columns + their RoPE partners).
// ---------------------------------------------------------------------------------------------
template <int DH, bool DEROPE>
__global__ __launch_bounds__(256) void fit_gram_f32_kernel(const FitGramParams p) {
  constexpr int BK = 16, LD = kTB + 4, HALF = DH / 2;
  __shared__ __attribute__((aligned(16))) float xs[2][BK * LD];

  const int nt = 2 * p.w / kTB, n_upper = nt * (nt + 1) / 2;
  // the tiles of one (job, slice) read the same rows: consecutive units on one XCD, so the second
  // read of a column block hits that XCD's L2
  int unit = xcd_remap(blockIdx.x, gridDim.x);
  const int tile = unit % n_upper;
  unit /= n_upper;
  const int slice = unit % p.n_slices;
  const int job = unit / p.n_slices;
  int ti, tj;
  tile_of(tile, nt, ti, tj);
  const bool diag = ti == tj;
  const int nblk = diag ? 1 : 2;
  const FitGramJob& jb = p.jobs[job];
  const int64_t r0 = static_cast<int64_t>(slice) * p.slice_rows;
  const int64_t r1 = r0 + p.slice_rows < p.n_rows ? r0 + p.slice_rows : p.n_rows;
  const int64_t row_bytes = static_cast<int64_t>(p.w) * 4;

  const int tid = threadIdx.x;
  const int lr = tid & 15, cp = tid >> 4;
  const int c = pair_col<DH, 4>(cp);
  const int ri = c % DH;
  BlockSrc src[2];
  src[0] = block_src(jb, p.w, ti * kTB + c, 4);
  src[1] = block_src(jb, p.w, tj * kTB + c, 4);
  const int ty = tid >> 4, tx = tid & 15;

  float acc[8][8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = 0.f;
  float csum[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) csum[i] = 0.f;

  for (int64_t k0 = r0; k0 < r1; k0 += BK) {
    const int64_t n = k0 + lr;
    float f[2][2][4];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      if (b >= nblk) break;
      float4 u = make_float4(0.f, 0.f, 0.f, 0.f), v = u;
      if (n < r1) {
        const char* rowp = src[b].base + n * row_bytes + src[b].col;
        const uint4 ui = gload16(rowp), vi = gload16(rowp + HALF * 4);
        u = make_float4(__uint_as_float(ui.x), __uint_as_float(ui.y), __uint_as_float(ui.z),
                        __uint_as_float(ui.w));
        v = make_float4(__uint_as_float(vi.x), __uint_as_float(vi.y), __uint_as_float(vi.z),
                        __uint_as_float(vi.w));
      }
      f[b][0][0] = u.x; f[b][0][1] = u.y; f[b][0][2] = u.z; f[b][0][3] = u.w;
      f[b][1][0] = v.x; f[b][1][1] = v.y; f[b][1][2] = v.z; f[b][1][3] = v.w;
      if constexpr (DEROPE) {
        if (n < r1) {
          const float2* tab = p.rope + static_cast<int64_t>(fit_position(p, n)) * HALF + ri;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float2 cs = tab[j];
            const float a0 = f[b][0][j], b0 = f[b][1][j];
            f[b][0][j] = a0 * cs.x + b0 * cs.y;
            f[b][1][j] = b0 * cs.x - a0 * cs.y;
          }
        }
      }
      if (b == 0 && diag) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          csum[j] += f[0][0][j];
          csum[4 + j] += f[0][1][j];
        }
      }
    }
    __syncthreads();
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      if (b >= nblk) break;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        xs[b][lr * LD + c + j] = f[b][0][j];
        xs[b][lr * LD + c + HALF + j] = f[b][1][j];
      }
    }
    __syncthreads();
    const float* xi = xs[0];
    const float* xj = xs[diag ? 0 : 1];
#pragma unroll 4
    for (int k = 0; k < BK; ++k) {
      float av[8], bv[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        av[i] = xi[k * LD + ty + 16 * i];
        bv[i] = xj[k * LD + tx + 16 * i];
      }
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
    }
  }

  float* out = p.partial + ((static_cast<int64_t>(job) * p.n_slices + slice) * n_upper + tile) *
                               static_cast<int64_t>(kTileFloats);
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) out[(ty + 16 * i) * kTB + tx + 16 * j] = acc[i][j];
  if (diag) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int o = 8; o >= 1; o >>= 1) csum[i] += __shfl_xor(csum[i], o, 64);
    if (lr == 0) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        out[kTB * kTB + c + j] = csum[j];
        out[kTB * kTB + c + HALF + j] = csum[4 + j];
      }
    }
  }
}

// Sums each job's partial tiles over its slices in slice order (so the result does not depend on
// scheduling) and writes the full symmetric Gram and the column sums.  A workgroup owns one 32 x 32
// sub-block of an upper tile: it reads the partials coalesced, writes the block in place and its
// mirror image through an LDS transpose.  Inside a diagonal tile only sub-blocks on or above its
// diagonal run, and a diagonal sub-block takes element (min, max) for both (i, j) and (j, i), so the
// Gram is exactly symmetric.
__global__ __launch_bounds__(256) void fit_gram_reduce_kernel(const FitGramParams p) {
  const int n2 = 2 * p.w, nt = n2 / kTB, n_upper = nt * (nt + 1) / 2;
  const int job = blockIdx.y;
  const int tile = blockIdx.x / 16, sub = blockIdx.x % 16, sr = sub / 4, sc = sub % 4;
  int ti, tj;
  tile_of(tile, nt, ti, tj);
  const bool diag = ti == tj;
  if (diag && sr > sc) return;
  const FitGramJob& jb = p.jobs[job];
  const float* base = p.partial + (static_cast<int64_t>(job) * p.n_slices * n_upper + tile) *
                                      static_cast<int64_t>(kTileFloats);
  const int64_t slice_stride = static_cast<int64_t>(n_upper) * kTileFloats;
  __shared__ float blk[32][33];
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int r = ty + 8 * k;
    const int off = (sr * 32 + r) * kTB + sc * 32 + tx;
    float v = 0.f;
    for (int sl = 0; sl < p.n_slices; ++sl) v += base[sl * slice_stride + off];
    blk[r][tx] = v;
  }
  __syncthreads();
  const int i0 = ti * kTB + sr * 32, j0 = tj * kTB + sc * 32;
  const bool dsub = diag && sr == sc;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int r = ty + 8 * k;
    const float up = dsub && r > tx ? blk[tx][r] : blk[r][tx];
    jb.gram[static_cast<int64_t>(i0 + r) * n2 + j0 + tx] = up;      // G[i][j], i <= j
    if (!dsub) jb.gram[static_cast<int64_t>(j0 + r) * n2 + i0 + tx] = blk[tx][r];  // G[j][i]
  }
  if (diag && sub == 0 && threadIdx.x < kTB) {
    float v = 0.f;
    for (int sl = 0; sl < p.n_slices; ++sl) v += base[sl * slice_stride + kTB * kTB + threadIdx.x];
    jb.colsum[ti * kTB + threadIdx.x] = v;
  }
}

// ---------------------------------------------------------------------------------------------
// fp64 solve.  Every stage is one launch over all layers of the call (the last grid dimension is
// the layer), so each stage spreads over the whole GPU:
//   prep      the centred Gram G_c and the offsets;
//   tridiag   Householder reduction Q^T G_c Q = T (tridiagonal), one launch per column: the launch
//             for column k + 1 applies reflector k to the trailing block, forms reflector k + 1
//             from the updated column and the product p = tau A v that the next launch needs.  Two
//             matrix copies take turns as source and destination, so no workgroup reads what
//             another workgroup of the same launch writes.  The last steps (a trailing block of at
//             most 128 rows) run in one launch with the block in LDS;
//   bisect    the r largest eigenvalues of T by bisection on Sturm counts;
//   inverse   their eigenvectors of T by inverse iteration (three solves with T - lambda I under
//             partial pivoting); eigenvalues closer than 1e-7 ||T|| form a cluster, whose vectors
//             one thread computes in turn, each orthogonalised against the cluster's earlier ones
//             (for 2w <= 256 the working vectors live in LDS);
//   back      V_r = Q Y, each column's largest-magnitude entry then made positive;
//   project   P = G_c V_r;
//   normal    Z^T Z + lam I = V_r^T P + lam I and A^T A + lam I;
//   chol      right-looking Cholesky of both, one launch per column (sizes up to 128: one
//             launch, the matrix in LDS);
//   out       the triangular solves for E and F and the outputs, rounded once.
// ---------------------------------------------------------------------------------------------
constexpr int kSolveThreads = 256;
constexpr int kSolveRows = 16;  // rows per workgroup of the prep and of a tridiagonal step, n <= 512
// Rows per workgroup of a tridiagonal step for n > 512 and of a per-column Cholesky step: the
// trailing block is then large and one layer's 16-row workgroups would leave most CUs idle, each
// workgroup bound by its CU's share of the memory bandwidth.
constexpr int kSolveRowsWide = 4;
// columns of Y per workgroup of the back-transformation: 8 for n <= 512 (many layers, short
// chains), 2 above (one layer's few workgroups carry long chains)
constexpr int kBackColsNarrow = 8, kBackColsWide = 2;
constexpr int kMaxN = 2 * kFitMaxSolveWidth;
constexpr int kInverseSolves = 3;
constexpr double kEps = 2.220446049250313e-16;  // 2^-52
constexpr double kClusterTol = 1e-7;            // relative to ||T||: eigenvalues closer cluster
constexpr double kNaN = __builtin_nan("");

// Per-layer table that the prep launch writes into the layer's workspace for the later launches
// (whose argument block stays small).
struct SolveJob {
  const float* gram;
  const float* colsum;
  void* w_enc;
  void* w_dec;
  void* mu_enc;
  void* mu_dec;
  int64_t rank;
  double tnorm;  // Gershgorin bound of ||T||, written by the bisection launch
};

struct SolveArgs {
  double* work;
  double rows;
  double lambda;
  int32_t w;
  int32_t step;
  int32_t center;
  int32_t bf16;
};

// One layer's workspace (fp64, n = 2w): four n x n matrices Z, X, Y, M, then 8n scalars.
struct Slots {
  double *z, *x, *y, *m;
  double *d, *e, *tau, *p0, *p1, *lam, *ldiag;
  SolveJob* job;
};

__device__ inline Slots slots(double* work, int w, int layer) {
  const int64_t n = 2 * w, n2 = n * n;
  double* b = work + layer * fit_solve_layer_doubles(w);
  Slots s;
  s.z = b;
  s.x = b + n2;
  s.y = b + 2 * n2;
  s.m = b + 3 * n2;
  double* v = b + 4 * n2;
  s.d = v;
  s.e = v + n;
  s.tau = v + 2 * n;
  s.p0 = v + 3 * n;
  s.p1 = v + 4 * n;
  s.lam = v + 5 * n;
  s.ldiag = v + 6 * n;  // Cholesky diagonals: A^T A block [w], then Z^T Z block [r]
  s.job = reinterpret_cast<SolveJob*>(v + 7 * n);
  return s;
}

// Centred Gram entry G[i][j] - s_i s_j / N in fp64; every stage that needs G_c evaluates it with
// this one expression, so all see the same values.
__device__ inline double centred(const float* gram, const float* cs, int n, int i, int j, double rows,
                                 bool center) {
  double g = static_cast<double>(gram[static_cast<int64_t>(i) * n + j]);
  if (center) g -= static_cast<double>(cs[i]) * static_cast<double>(cs[j]) / rows;
  return g;
}

__device__ inline double wave_sum(double v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ inline void store_out(void* dst, int64_t i, double v, bool bf16) {
  if (bf16) static_cast<__bf16*>(dst)[i] = static_cast<__bf16>(static_cast<float>(v));
  else static_cast<float*>(dst)[i] = static_cast<float>(v);
}

// Reflector j lives in row j of X (j odd) or Y (j even), entries j+1 .. n-1 (the first one 1).
__device__ inline double* reflector_rows(const Slots& s, int j) { return (j & 1) ? s.x : s.y; }

// ---- prep: G_c into Z, the offsets, the job table --------------------------------------------
__global__ __launch_bounds__(kSolveThreads) void fit_prep_kernel(const FitSolveParams p) {
  const int layer = blockIdx.y, n = 2 * p.w;
  const FitSolveJob& jb = p.jobs[layer];
  const Slots s = slots(p.work, p.w, layer);
  const double rows = static_cast<double>(p.n_rows);
  const bool center = p.center != 0, bf16 = p.bf16 != 0;
  const int i0 = blockIdx.x * kSolveRows;
  for (int e = threadIdx.x; e < kSolveRows * n; e += kSolveThreads) {
    const int i = i0 + e / n, j = e % n;
    if (i < n) s.z[static_cast<int64_t>(i) * n + j] = centred(jb.gram, jb.colsum, n, i, j, rows, center);
  }
  if (blockIdx.x != 0) return;
  if (threadIdx.x == 0)
    *s.job = SolveJob{jb.gram, jb.colsum, jb.w_enc, jb.w_dec, jb.mu_enc, jb.mu_dec, jb.rank, 0.0};
  if (center) {
    for (int i = threadIdx.x; i < p.w; i += kSolveThreads) {
      store_out(jb.mu_enc, i, static_cast<double>(jb.colsum[i]) / rows, bf16);
      store_out(jb.mu_dec, i, static_cast<double>(jb.colsum[p.w + i]) / rows, bf16);
    }
  }
}

// ---- one Householder step ----------------------------------------------------------------------
// Launch k (k = -1 .. n-3), with A^(k) the matrix after reflectors 0 .. k-1 (A^(0) = G_c):
//   w_k = p_k - (tau_k / 2)(p_k . v_k) v_k;  A^(k+1) = A^(k) - v_k w_k^T - w_k v_k^T on the block
//   [k+1, n)^2 (launch -1 has no reflector to apply);
//   column k+1 of A^(k+1) gives d_{k+1}, and its part below the diagonal, x, gives reflector k+1:
//   beta = -sign(x_0) ||x||, tau = (beta - x_0) / beta, v = x / (x_0 - beta) with v_0 = 1, so that
//   (I - tau v v^T) x = beta e_0 (e_{k+1} = beta; x with nothing below x_0 takes tau = 0);
//   p_{k+1} = tau_{k+1} A^(k+1) v_{k+1} on rows [k+2, n), this workgroup's rows only.
// Source A^(k): G_c (Z) for k <= 0, else the previous launch's destination; destination: X for even
// k, Y for odd k.  Reflector k+1 goes into row k+1 of the destination, a row no later launch
// writes; p alternates between two vectors.
// Every global load of a launch is issued at its start (the reflector and p of the previous launch,
// row k+1 and, for n <= 64 PRE, this workgroup's rows of the source), so the launch waits on one
// round of loads rather than three.
template <int PRE, int ROWS>
__device__ __forceinline__ void tridiag_step(const SolveArgs& a) {
  __shared__ double vk[kMaxN], wk[kMaxN], vn[kMaxN];
  __shared__ double red[2][kSolveThreads / 64];
  const int layer = blockIdx.y, n = 2 * a.w, k = a.step, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  constexpr int kWaves = kSolveThreads / 64, kRowsPerWave = ROWS / kWaves;
  static_assert(ROWS % kWaves == 0, "whole rows per wave");
  const Slots s = slots(a.work, a.w, layer);
  const double* src = k <= 0 ? s.z : ((k - 1) & 1 ? s.y : s.x);
  double* dst = (k & 1) ? s.y : s.x;  // k = -1 is odd: Y (only its reflector row is written)
  double* p_next = ((k + 1) & 1) ? s.p1 : s.p0;
  const int r0 = k + 2 + blockIdx.x * ROWS;
  // loads: reflector k and p_k into vk / wk, row k+1 of the source into vn, own rows to registers
  if (k >= 0) {
    const double* vrow = reflector_rows(s, k) + static_cast<int64_t>(k) * n;
    const double* p_cur = (k & 1) ? s.p1 : s.p0;
    for (int i = k + 1 + tid; i < n; i += kSolveThreads) {
      vk[i] = vrow[i];
      wk[i] = p_cur[i];
    }
  } else {
    for (int i = tid; i < n; i += kSolveThreads) vk[i] = wk[i] = 0.0;
  }
  const double* row1 = src + static_cast<int64_t>(k + 1) * n;
  for (int i = k + 1 + tid; i < n; i += kSolveThreads) vn[i] = row1[i];
  double pre[PRE > 0 ? kRowsPerWave : 1][PRE > 0 ? PRE : 1];
  if constexpr (PRE > 0) {
    for (int q = 0; q < kRowsPerWave; ++q) {
      const int i = r0 + wave + kWaves * q;
      for (int u = 0; u < PRE; ++u) {
        const int j = k + 2 + lane + 64 * u;
        pre[q][u] = (i < n && j < n) ? src[static_cast<int64_t>(i) * n + j] : 0.0;
      }
    }
  }
  __syncthreads();
  // w_k = p_k - (tau_k / 2)(p_k . v_k) v_k (zero for launch -1)
  double kk = 0.0;
  if (k >= 0) {
    double dot = 0.0;
    for (int i = k + 1 + tid; i < n; i += kSolveThreads) dot += wk[i] * vk[i];
    dot = wave_sum(dot);
    if (lane == 0) red[0][wave] = dot;
    __syncthreads();
    double t = 0.0;
    for (int q = 0; q < kWaves; ++q) t += red[0][q];
    kk = 0.5 * s.tau[k] * t;
  }
  const double vk1 = vk[k + 1], wk1 = wk[k + 1] - kk * vk1;
  // column k+1 of A^(k+1) (row k+1, the matrix being symmetric) and w_k, own entries only
  double sig = 0.0;
  for (int i = k + 1 + tid; i < n; i += kSolveThreads) {
    const double wi = wk[i] - kk * vk[i];
    if (i > k + 1) wk[i] = wi;  // entry k+1 stays p_k's: every thread reads it above
    const double c = vn[i] - vk1 * wi - wk1 * vk[i];
    vn[i] = c;
    if (i >= k + 3) sig += c * c;
  }
  sig = wave_sum(sig);
  if (lane == 0) red[1][wave] = sig;
  __syncthreads();
  double sigma = 0.0;
  for (int q = 0; q < kWaves; ++q) sigma += red[1][q];
  const double d_next = vn[k + 1], alpha = vn[k + 2];
  double tau = 0.0, beta = alpha, scale = 0.0;
  if (!(sigma == 0.0)) {
    const double norm = sqrt(alpha * alpha + sigma);
    beta = alpha >= 0.0 ? -norm : norm;
    tau = (beta - alpha) / beta;
    scale = 1.0 / (alpha - beta);
  }
  // v_{k+1}: entries past its first scaled in place; its first entry (1) is never stored in vn,
  // so alpha stays readable
  for (int i = k + 3 + tid; i < n; i += kSolveThreads) vn[i] *= scale;
  __syncthreads();
  // this workgroup's rows of A^(k+1) and of p_{k+1}
  for (int q = 0; q < kRowsPerWave; ++q) {
    const int i = r0 + wave + kWaves * q;
    if (i >= n || i >= r0 + ROWS) break;
    const double* arow = src + static_cast<int64_t>(i) * n;
    double* orow = dst + static_cast<int64_t>(i) * n;
    const double vi = vk[i], wi = wk[i];
    double acc = 0.0;
    auto entry = [&](int j, double x) {
      const double v = x - vi * wk[j] - wi * vk[j];
      if (k >= 0) orow[j] = v;
      if (k == n - 3) s.d[n - 1] = v;  // the last launch: i = j = n - 1
      acc += v * (j == k + 2 ? 1.0 : vn[j]);
    };
    if constexpr (PRE > 0) {
#pragma unroll
      for (int u = 0; u < PRE; ++u) {
        const int j = k + 2 + lane + 64 * u;
        if (j < n) entry(j, pre[q][u]);
      }
    } else {
      for (int j = k + 2 + lane; j < n; j += 64) entry(j, arow[j]);
    }
    acc = wave_sum(acc);
    if (lane == 0) p_next[i] = tau * acc;
  }
  if (blockIdx.x == 0) {
    double* vrow = dst + static_cast<int64_t>(k + 1) * n;
    for (int i = k + 2 + tid; i < n; i += kSolveThreads) vrow[i] = i == k + 2 ? 1.0 : vn[i];
    if (tid == 0) {
      s.d[k + 1] = d_next;
      s.e[k + 1] = beta;
      s.tau[k + 1] = tau;
    }
  }
}

constexpr int kTridiagPre = 8;  // row entries per lane held in registers: n <= 512
__global__ __launch_bounds__(kSolveThreads) void fit_tridiag_pre_kernel(const SolveArgs a) {
  tridiag_step<kTridiagPre, kSolveRows>(a);
}
__global__ __launch_bounds__(kSolveThreads) void fit_tridiag_kernel(const SolveArgs a) {
  tridiag_step<0, kSolveRowsWide>(a);
}

// The last steps, from step k0 on (trailing block of at most kTailN rows), in one launch: one
// workgroup per layer holds the block [k0 + 1, n)^2 of A^(k0) in LDS and applies the same steps as
// the per-column launches (the same expressions, reflectors and p in the same places), the
// workgroup barriers standing in for the launch boundaries.  k0 = -1 starts from G_c itself.
constexpr int kTailN = 128, kTailThreads = 1024;
__global__ __launch_bounds__(kTailThreads) void fit_tridiag_tail_kernel(const SolveArgs a) {
  constexpr int LD = kTailN + 1, kWaves = kTailThreads / 64;
  __shared__ double am[kTailN * LD];
  __shared__ double vk[kTailN], wk[kTailN], vn[kTailN], pk[kTailN];
  __shared__ double red[2][kWaves];
  const int layer = blockIdx.x, n = 2 * a.w, k0 = a.step, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const Slots s = slots(a.work, a.w, layer);
  const int o = k0 + 1;  // global index of local row / column 0
  const int m0 = n - o;  // rows of the block (<= kTailN)
  {
    const double* src = k0 <= 0 ? s.z : ((k0 - 1) & 1 ? s.y : s.x);
    for (int e = tid; e < m0 * m0; e += kTailThreads) {
      const int i = e / m0, j = e % m0;
      am[i * LD + j] = src[static_cast<int64_t>(o + i) * n + o + j];
    }
    if (k0 >= 0) {
      const double* vrow = reflector_rows(s, k0) + static_cast<int64_t>(k0) * n;
      const double* p_cur = (k0 & 1) ? s.p1 : s.p0;
      for (int i = tid; i < m0; i += kTailThreads) {
        vk[i] = vrow[o + i];
        pk[i] = p_cur[o + i];
      }
    } else {
      for (int i = tid; i < m0; i += kTailThreads) vk[i] = pk[i] = 0.0;
    }
  }
  __syncthreads();
  auto block_sum = [&](double v, int slot) {
    v = wave_sum(v);
    if (lane == 0) red[slot][wave] = v;
    __syncthreads();
    double t = 0.0;
    for (int q = 0; q < kWaves; ++q) t += red[slot][q];
    return t;
  };
  double tau_k = k0 >= 0 ? s.tau[k0] : 0.0;
  for (int k = k0; k <= n - 3; ++k) {
    // local indices: global i is local i - o; the step touches global [k + 1, n)
    const int b = k + 1 - o;  // local index of global k + 1
    // w_k = p_k - (tau_k / 2)(p_k . v_k) v_k
    double kk = 0.0;
    if (k >= 0) {
      double dot = 0.0;
      for (int i = b + tid; i < m0; i += kTailThreads) dot += pk[i] * vk[i];
      kk = 0.5 * tau_k * block_sum(dot, 0);
    }
    const double vk1 = vk[b], wk1 = pk[b] - kk * vk1;
    double sig = 0.0;
    for (int i = b + tid; i < m0; i += kTailThreads) {
      const double wi = pk[i] - kk * vk[i];
      wk[i] = wi;
      const double c = am[b * LD + i] - vk1 * wi - wk1 * vk[i];
      vn[i] = c;
      if (i >= b + 2) sig += c * c;
    }
    const double sigma = block_sum(sig, 1);  // its barrier also publishes wk and vn
    const double d_next = vn[b], alpha = vn[b + 1];
    double tau = 0.0, beta = alpha, scale = 0.0;
    if (!(sigma == 0.0)) {
      const double norm = sqrt(alpha * alpha + sigma);
      beta = alpha >= 0.0 ? -norm : norm;
      tau = (beta - alpha) / beta;
      scale = 1.0 / (alpha - beta);
    }
    __syncthreads();  // every thread has read alpha and used pk
    for (int i = b + 2 + tid; i < m0; i += kTailThreads) vn[i] *= scale;
    __syncthreads();
    // rows k + 2 .. n - 1 of A^(k+1) (in place) and of p_{k+1}
    for (int i = b + 1 + wave; i < m0; i += kWaves) {
      const double vi = vk[i], wi = wk[i];
      double acc = 0.0;
      for (int j = b + 1 + lane; j < m0; j += 64) {
        const double v = am[i * LD + j] - vi * wk[j] - wi * vk[j];
        am[i * LD + j] = v;
        if (k == n - 3 && tid == 0) s.d[n - 1] = v;  // the last step: i = j = n - 1
        acc += v * (j == b + 1 ? 1.0 : vn[j]);
      }
      acc = wave_sum(acc);
      if (lane == 0) pk[i] = tau * acc;
    }
    // reflector k + 1 where the per-column launches keep it, and T's entries
    double* vrow = ((k + 1) & 1 ? s.x : s.y) + static_cast<int64_t>(k + 1) * n;
    for (int i = b + 1 + tid; i < m0; i += kTailThreads) vrow[o + i] = i == b + 1 ? 1.0 : vn[i];
    if (tid == 0) {
      s.d[k + 1] = d_next;
      s.e[k + 1] = beta;
      s.tau[k + 1] = tau;
    }
    __syncthreads();  // pk and am are the next step's
    // the next step's reflector: v_{k+1} (first entry 1)
    for (int i = b + 1 + tid; i < m0; i += kTailThreads) vk[i] = i == b + 1 ? 1.0 : vn[i];
    tau_k = tau;
    __syncthreads();
  }
}

// ---- bisection -------------------------------------------------------------------------------
// Number of eigenvalues of T below x (Sturm count of the LDL^T pivots of T - x I); a pivot smaller
// in magnitude than pivmin counts as -pivmin.
__device__ inline int sturm_count(const double* d, const double* e2, int n, double x, double pivmin) {
  double q = d[0] - x;
  if (fabs(q) < pivmin) q = -pivmin;
  int c = q < 0.0 ? 1 : 0;
  for (int i = 1; i < n; ++i) {
    q = (d[i] - x) - e2[i - 1] / q;
    if (fabs(q) < pivmin) q = -pivmin;
    c += q < 0.0 ? 1 : 0;
  }
  return c;
}

// Gershgorin interval of T, over the workgroup (64 threads, one wave).
__device__ inline void gershgorin(const double* d, const double* ae, int n, double& lo, double& hi) {
  lo = INFINITY;
  hi = -INFINITY;
  for (int i = threadIdx.x; i < n; i += 64) {
    const double rad = (i > 0 ? ae[i - 1] : 0.0) + (i < n - 1 ? ae[i] : 0.0);
    lo = fmin(lo, d[i] - rad);
    hi = fmax(hi, d[i] + rad);
  }
  for (int o = 32; o > 0; o >>= 1) {
    lo = fmin(lo, __shfl_xor(lo, o, 64));
    hi = fmax(hi, __shfl_xor(hi, o, 64));
  }
}

// One wave per workgroup, four eigenvalues per wave, each by 16 lanes: lam[j] = the (j+1)-th
// largest.  Every round the 16 lanes take Sturm counts at 16 evenly spaced interior points of the
// bracket, which then shrinks to the pair of neighbouring points (ends included) between which the
// count passes j's ascending index: a 17-fold cut per round, until the bracket is below an absolute
// 2^-52 ||T|| plus a relative 2^-51.
constexpr int kSectionLanes = 16;
__global__ __launch_bounds__(64) void fit_bisect_kernel(const SolveArgs a) {
  __shared__ double d[kMaxN], e2[kMaxN], ae[kMaxN];
  const int layer = blockIdx.y, n = 2 * a.w;
  const Slots s = slots(a.work, a.w, layer);
  const int r = static_cast<int>(s.job->rank);
  for (int i = threadIdx.x; i < n; i += 64) {
    d[i] = s.d[i];
    const double e = i < n - 1 ? s.e[i] : 0.0;
    e2[i] = e * e;
    ae[i] = fabs(e);
  }
  __syncthreads();
  double lo0, hi0;
  gershgorin(d, ae, n, lo0, hi0);
  // a floor keeps the tolerances positive for an all-zero matrix
  const double tnorm = fmax(fmax(fabs(lo0), fabs(hi0)), 1e-280);
  if (blockIdx.x == 0 && threadIdx.x == 0) s.job->tnorm = tnorm;
  const int lane = threadIdx.x & (kSectionLanes - 1);
  const int j = blockIdx.x * (64 / kSectionLanes) + threadIdx.x / kSectionLanes;
  // the 16 lanes of an eigenvalue share every branch below; whole groups past r are idle
  const bool live = j < r;
  const double atol = kEps * tnorm, pivmin = kEps * tnorm;
  const int t = n - 1 - j;  // ascending index
  double lo = lo0 - atol, hi = hi0 + atol;
  for (int it = 0; it < 64; ++it) {
    if (hi - lo <= atol + 2.0 * kEps * fmax(fabs(lo), fabs(hi))) break;
    // point k = 1 .. 16 at lo + k step; the new ends are points (or the old ends), so the counts
    // already taken there hold for them
    const double step = (hi - lo) * (1.0 / (kSectionLanes + 1));
    const double x = lo + step * (lane + 1);
    const bool below = live && sturm_count(d, e2, n, x, pivmin) <= t;
    // lanes of this group whose point lies below the eigenvalue (a prefix of the group)
    const uint64_t m = __ballot(below);
    const int group = threadIdx.x & ~(kSectionLanes - 1);
    const int kb = __popcll((m >> group) & ((1ull << kSectionLanes) - 1));
    const double nlo = kb > 0 ? lo + step * kb : lo;
    const double nhi = kb < kSectionLanes ? lo + step * (kb + 1) : hi;
    lo = nlo;
    hi = nhi;
  }
  if (live && lane == 0) s.lam[j] = 0.5 * (lo + hi);
}

// ---- inverse iteration --------------------------------------------------------------------------
__device__ inline double start_entry(int i, int m) {
  uint32_t x = static_cast<uint32_t>(i) * 0x9E3779B1u ^ (static_cast<uint32_t>(m) + 0x7F4A7C15u) * 0x85EBCA77u;
  x ^= x >> 16;
  x *= 0x7FEB352Du;
  x ^= x >> 15;
  x *= 0x846CA68Bu;
  x ^= x >> 16;
  return static_cast<double>(x >> 8) * (1.0 / 16777216.0) - 0.5;
}

// A pivot smaller than tol in magnitude becomes +-tol (NaN stays NaN).
__device__ inline double guard_pivot(double c, double tol) {
  return !(fabs(c) <= tol) ? c : (c >= 0.0 ? tol : -tol);
}

// Strided view of one vector: entry i at p[i * stride].
struct Strided {
  double* p;
  int64_t stride;
  __device__ double& operator[](int i) const { return p[i * stride]; }
};

// The four vectors one eigenvector's inverse iteration works on: the vector and its LU factors.
struct InverseWork {
  Strided y, u0, u1, u2;
};

// Inverse iteration for the cluster of eigenvalues lam[j .. last] (one thread).  Member m works in
// work(m); every finished vector m is stored at out(m) (Y[i][m] of the layer), which is also where
// the orthogonalisation reads the earlier members.
template <typename WorkFn, typename OutFn>
__device__ inline void inverse_cluster(const double* d, const double* e, int n, const double* lam,
                                       int j, int last, double tnorm, WorkFn work, OutFn out) {
  const double pert = 10.0 * kEps * tnorm, ptol = kEps * tnorm;
  double sigma = 0.0;
  for (int m = j; m <= last; ++m) {
    const InverseWork wk = work(m);
    const Strided y = wk.y, u0 = wk.u0, u1 = wk.u1, u2 = wk.u2;
    // shifts inside a cluster step down by at least pert, so the solves stay independent
    sigma = m == j ? lam[m] : fmin(lam[m], sigma - pert);
    for (int i = 0; i < n; ++i) y[i] = start_entry(i, m);
    double sc = 2.0;  // the start vector's entries lie in [-1/2, 1/2)
    for (int it = 0; it < kInverseSolves; ++it) {
      // forward elimination of (T - sigma I) y = b / max|b| with partial pivoting; rows hold
      // (c0, c1) on the diagonal and the superdiagonal, the right-hand side rides along
      double c0 = d[0] - sigma, c1 = n > 1 ? e[0] : 0.0;
      double yc = y[0] * sc;
      for (int i = 0; i < n - 1; ++i) {
        const double sub = e[i], a1 = d[i + 1] - sigma, b1 = i + 1 < n - 1 ? e[i + 1] : 0.0;
        const double nb = y[i + 1] * sc;
        if (fabs(c0) >= fabs(sub)) {
          const double piv = guard_pivot(c0, ptol);
          const double mult = sub / piv;
          u0[i] = piv;
          u1[i] = c1;
          u2[i] = 0.0;
          y[i] = yc;
          yc = nb - mult * yc;
          c0 = a1 - mult * c1;
          c1 = b1;
        } else {
          const double mult = c0 / sub;
          u0[i] = sub;
          u1[i] = a1;
          u2[i] = b1;
          y[i] = nb;
          yc = yc - mult * nb;
          c0 = c1 - mult * a1;
          c1 = -mult * b1;
        }
      }
      u0[n - 1] = guard_pivot(c0, ptol);
      y[n - 1] = yc;
      // back substitution, in place
      double x1 = 0.0, x2 = 0.0;
      for (int i = n - 1; i >= 0; --i) {
        double v = y[i];
        if (i + 1 < n) v -= u1[i] * x1;
        if (i + 2 < n) v -= u2[i] * x2;
        v /= u0[i];
        y[i] = v;
        x2 = x1;
        x1 = v;
      }
      // orthogonalise against the cluster's earlier vectors, then normalise
      for (int q = j; q < m; ++q) {
        const Strided yq = out(q);
        double dot = 0.0;
        for (int i = 0; i < n; ++i) dot += yq[i] * y[i];
        for (int i = 0; i < n; ++i) y[i] -= dot * yq[i];
      }
      double ss = 0.0, mx = 0.0;
      for (int i = 0; i < n; ++i) {
        ss += y[i] * y[i];
        mx = fmax(mx, fabs(y[i]));
      }
      const double inv = 1.0 / sqrt(ss);
      for (int i = 0; i < n; ++i) y[i] *= inv;
      sc = mx > 0.0 ? 1.0 / (mx * inv) : 1.0;  // 1 / max|y| of the normalised vector
    }
    const Strided o = out(m);
    if (o.p != y.p)
      for (int i = 0; i < n; ++i) o[i] = y[i];
  }
}

// One thread per eigenvalue; only the first thread of a cluster works (it takes the whole
// cluster in order).  Returns false for threads with nothing to do.
__device__ inline bool cluster_of(const double* lam, int r, int j, double ctol, int* last) {
  if (j >= r || (j > 0 && !(lam[j - 1] - lam[j] > ctol))) return false;
  int l = j;
  while (l + 1 < r && !(lam[l] - lam[l + 1] > ctol)) ++l;
  *last = l;
  return true;
}

// Inverse iteration, one eigenvector per working thread: the thread keeps its vector and the LU
// factors of T - sigma I in LDS ([i][thread], THREADS interleaved, so the threads' accesses fall in
// distinct banks) and copies each finished vector to Y[i][m].  Two instances: 16 threads per
// workgroup for n <= 256, and one thread per workgroup (96 KiB of LDS) for larger n; the chain of
// dependent accesses would otherwise wait on global memory at each link.
constexpr int kInverseLdsN = 256, kInverseLdsThreads = 16;
template <int N, int THREADS>
__global__ __launch_bounds__(64) void fit_inverse_lds_kernel(const SolveArgs a) {
  __shared__ double d[N], e[N];
  __shared__ double vec[4 * N * THREADS];
  const int layer = blockIdx.y, n = 2 * a.w;
  const Slots s = slots(a.work, a.w, layer);
  const int r = static_cast<int>(s.job->rank);
  for (int i = threadIdx.x; i < n; i += 64) {
    d[i] = s.d[i];
    e[i] = i < n - 1 ? s.e[i] : 0.0;
  }
  __syncthreads();
  const int t = threadIdx.x;
  const int j = blockIdx.x * THREADS + t;
  if (t >= THREADS) return;
  const double tnorm = s.job->tnorm;
  int last;
  if (!cluster_of(s.lam, r, j, kClusterTol * tnorm, &last)) return;
  constexpr int64_t kPlane = static_cast<int64_t>(N) * THREADS;
  auto lds = [&](int q) { return Strided{vec + q * kPlane + t, THREADS}; };
  inverse_cluster(
      d, e, n, s.lam, j, last, tnorm,
      [&](int) { return InverseWork{lds(0), lds(1), lds(2), lds(3)}; },
      [&](int m) { return Strided{s.z + m, r}; });
}

// ---- back-transformation and sign ---------------------------------------------------------------
// kBackCols columns of Y per workgroup, held in LDS while the reflectors n-3 .. 0 are applied in
// turn (Y <- (I - tau_j v_j v_j^T) Y); thread t keeps rows i = t / kBackCols (mod kSolveThreads /
// kBackCols) of column t % kBackCols.  Then each column's first entry of largest magnitude is made
// positive.  Each reflector costs every column about 3n LDS accesses, so few columns per
// workgroup (and more workgroups) shorten the chain.
template <int kBackCols>
__global__ __launch_bounds__(kSolveThreads) void fit_back_kernel(const SolveArgs a) {
  __shared__ double yc[kMaxN * kBackCols];
  __shared__ double vb[kMaxN];
  __shared__ double red[kSolveThreads / 64][kBackCols];
  __shared__ int redi[kSolveThreads / 64][kBackCols];
  const int layer = blockIdx.y, n = 2 * a.w, tid = threadIdx.x;
  const Slots s = slots(a.work, a.w, layer);
  const int r = static_cast<int>(s.job->rank);
  const int c0 = blockIdx.x * kBackCols;
  if (c0 >= r) return;
  constexpr int kGroups = kSolveThreads / kBackCols;  // row groups
  const int c = tid % kBackCols, g = tid / kBackCols, lane = tid & 63, wave = tid >> 6;
  const bool live = c0 + c < r;
  for (int e = tid; e < n * kBackCols; e += kSolveThreads) {
    const int i = e / kBackCols, cc = e % kBackCols;
    yc[e] = c0 + cc < r ? s.z[static_cast<int64_t>(i) * r + c0 + cc] : 0.0;
  }
  // Reflector jr - 1 (its tau and this thread's entries of its row) is loaded into registers while
  // reflector jr is applied, so the chain of n - 2 reflectors does not wait on a global load at
  // each link; the barriers inside the chain only order LDS accesses (lds_barrier), so the loads
  // stay in flight across them.
  constexpr int kPer = kMaxN / kSolveThreads;
  double nxt[kPer];
  double tnext = 0.0;
  auto fetch = [&](int jr) {
    if (jr < 0) return;
    tnext = s.tau[jr];
    const double* vrow = reflector_rows(s, jr) + static_cast<int64_t>(jr) * n;
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      const int i = jr + 1 + tid + q * kSolveThreads;
      nxt[q] = i < n ? vrow[i] : 0.0;
    }
  };
  __syncthreads();  // Y is in LDS
  fetch(n - 3);
  for (int jr = n - 3; jr >= 0; --jr) {
    const double t = tnext;
    double cur[kPer];
#pragma unroll
    for (int q = 0; q < kPer; ++q) cur[q] = nxt[q];
    fetch(jr - 1);
    if (t == 0.0) continue;
    lds_barrier();  // the previous reflector's vb and red reads are done
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      const int i = jr + 1 + tid + q * kSolveThreads;
      if (i < n) vb[i] = cur[q];
    }
    lds_barrier();
    double part = 0.0;
    for (int i = jr + 1 + g; i < n; i += kGroups) part += vb[i] * yc[i * kBackCols + c];
    // the row groups of a wave that share column c sit kBackCols lanes apart
    for (int o = kBackCols; o < 64; o <<= 1) part += __shfl_xor(part, o, 64);
    if (lane < kBackCols) red[wave][lane] = part;
    lds_barrier();
    double dot = 0.0;
    for (int q = 0; q < kSolveThreads / 64; ++q) dot += red[q][c];
    const double f = t * dot;
    for (int i = jr + 1 + g; i < n; i += kGroups) yc[i * kBackCols + c] -= f * vb[i];
  }
  // sign: the first entry of largest magnitude of each column made positive
  __syncthreads();  // the last reflector's red reads and Y updates are done
  double best = -1.0;
  int bi = 0;
  for (int i = g; i < n; i += kGroups) {
    const double v = fabs(yc[i * kBackCols + c]);
    if (v > best) {
      best = v;
      bi = i;
    }
  }
  for (int o = kBackCols; o < 64; o <<= 1) {
    const double ob = __shfl_xor(best, o, 64);
    const int oi = __shfl_xor(bi, o, 64);
    if (ob > best || (ob == best && oi < bi)) {
      best = ob;
      bi = oi;
    }
  }
  if (lane < kBackCols) {
    red[wave][lane] = best;
    redi[wave][lane] = bi;
  }
  __syncthreads();
  best = red[0][c];
  bi = redi[0][c];
  for (int q = 1; q < kSolveThreads / 64; ++q) {
    if (red[q][c] > best || (red[q][c] == best && redi[q][c] < bi)) {
      best = red[q][c];
      bi = redi[q][c];
    }
  }
  const double sg = yc[bi * kBackCols + c] < 0.0 ? -1.0 : 1.0;
  if (live)
    for (int i = g; i < n; i += kGroups)
      s.z[static_cast<int64_t>(i) * r + c0 + c] = sg * yc[i * kBackCols + c];
}

// ---- fp64 tiled products ------------------------------------------------------------------------
// 64 x 64 output tile per workgroup, 4 x 4 per thread, k-steps of 16 through LDS.  ta(kk, i) and
// tb(kk, j) give the operands' entries for reduction index kk (0 outside the matrix).
template <typename FA, typename FB, typename FC>
__device__ inline void tile_product(int kdim, FA ta, FB tb, FC out) {
  __shared__ double as[16][64 + 1], bs[16][64 + 1];
  const int tid = threadIdx.x, tx = tid % 16, ty = tid / 16;
  double acc[4][4] = {};
  for (int k0 = 0; k0 < kdim; k0 += 16) {
    for (int e = tid; e < 16 * 64; e += kSolveThreads) {
      const int kk = e / 64, x = e % 64;
      as[kk][x] = k0 + kk < kdim ? ta(k0 + kk, x) : 0.0;
      bs[kk][x] = k0 + kk < kdim ? tb(k0 + kk, x) : 0.0;
    }
    __syncthreads();
    for (int kk = 0; kk < 16; ++kk) {
      double av[4], bv[4];
      for (int q = 0; q < 4; ++q) {
        av[q] = as[kk][ty + 16 * q];
        bv[q] = bs[kk][tx + 16 * q];
      }
      for (int q = 0; q < 4; ++q)
        for (int u = 0; u < 4; ++u) acc[q][u] += av[q] * bv[u];
    }
    __syncthreads();
  }
  for (int q = 0; q < 4; ++q)
    for (int u = 0; u < 4; ++u) out(ty + 16 * q, tx + 16 * u, acc[q][u]);
}

// P = G_c V_r [n, r] into M (grid: n / 64 x ceil(r_max / 64) tiles, layers)
__global__ __launch_bounds__(kSolveThreads) void fit_project_kernel(const SolveArgs a) {
  const int layer = blockIdx.z, n = 2 * a.w;
  const Slots s = slots(a.work, a.w, layer);
  const SolveJob jb = *s.job;
  const int r = static_cast<int>(jb.rank);
  const int i0 = blockIdx.x * 64, m0 = blockIdx.y * 64;
  if (m0 >= r) return;
  const bool center = a.center != 0;
  tile_product(
      n,
      // G_c is symmetric: its column i0 + x read as a row, so the loads run along rows
      [&](int kk, int x) { return centred(jb.gram, jb.colsum, n, kk, i0 + x, a.rows, center); },
      [&](int kk, int x) {
        return m0 + x < r ? s.z[static_cast<int64_t>(kk) * r + m0 + x] : 0.0;
      },
      [&](int x, int y, double v) {
        if (m0 + y < r) s.m[static_cast<int64_t>(i0 + x) * r + m0 + y] = v;
      });
}

// Z^T Z + lam I = V_r^T P + lam I [r, r] into Y (grid.x = tiles of it), and A^T A + lam I [w, w]
// into X (grid.y = 1: w / 64 x w / 64 tiles over grid.x)
__global__ __launch_bounds__(kSolveThreads) void fit_normal_kernel(const SolveArgs a) {
  const int layer = blockIdx.z, n = 2 * a.w, w = a.w;
  const Slots s = slots(a.work, a.w, layer);
  const SolveJob jb = *s.job;
  const int r = static_cast<int>(jb.rank);
  if (blockIdx.y == 0) {
    const int nt = (r + 63) / 64;
    if (static_cast<int>(blockIdx.x) >= nt * nt) return;
    const int k0 = (blockIdx.x / nt) * 64, l0 = (blockIdx.x % nt) * 64;
    tile_product(
        n,
        [&](int i, int x) { return k0 + x < r ? s.z[static_cast<int64_t>(i) * r + k0 + x] : 0.0; },
        [&](int i, int x) { return l0 + x < r ? s.m[static_cast<int64_t>(i) * r + l0 + x] : 0.0; },
        [&](int x, int y, double v) {
          const int k = k0 + x, l = l0 + y;
          if (k < r && l < r) s.y[static_cast<int64_t>(k) * r + l] = v + (k == l ? a.lambda : 0.0);
        });
  } else {
    const int nt = w / 64;
    if (static_cast<int>(blockIdx.x) >= nt * nt) return;
    const int i0 = (blockIdx.x / nt) * 64, j0 = (blockIdx.x % nt) * 64;
    const bool center = a.center != 0;
    for (int e = threadIdx.x; e < 64 * 64; e += kSolveThreads) {
      const int i = i0 + e / 64, j = j0 + e % 64;
      s.x[static_cast<int64_t>(i) * w + j] =
          centred(jb.gram, jb.colsum, n, i, j, a.rows, center) + (i == j ? a.lambda : 0.0);
    }
  }
}

// ---- Cholesky, one column per launch --------------------------------------------------------------
// grid.y = 0: A^T A + lam I (X, size w), 1: Z^T Z + lam I (Y, size r).  Step k reads column k on and
// below the diagonal, updates rows (k, s) of the lower triangle (a workgroup's kSolveRowsWide rows),
// and stores L[i][k] twice, in places nothing reads before the solves: at [k][i] in the upper
// triangle (column k of L as a row) and at [i][k] of a row-major copy of L just past the matrix.
// L[k][k] goes to ldiag.  A non-positive pivot leaves NaN, which reaches every output of the layer.
__global__ __launch_bounds__(kSolveThreads) void fit_chol_kernel(const SolveArgs a) {
  __shared__ double lc[kFitMaxSolveWidth];
  const int layer = blockIdx.z, w = a.w, k = a.step, tid = threadIdx.x;
  const Slots s = slots(a.work, a.w, layer);
  const int r = static_cast<int>(s.job->rank);
  const bool zz = blockIdx.y == 1;
  const int sz = zz ? r : w;
  if (k >= sz) return;
  double* mat = zz ? s.y : s.x;
  double* ldiag = s.ldiag + (zz ? w : 0);
  const double piv = mat[static_cast<int64_t>(k) * sz + k];
  const double lkk = piv > 0.0 ? sqrt(piv) : kNaN;
  for (int i = k + 1 + tid; i < sz; i += kSolveThreads) lc[i] = mat[static_cast<int64_t>(i) * sz + k] / lkk;
  __syncthreads();
  const int lane = tid & 63, wave = tid >> 6;
  const int r0 = k + 1 + blockIdx.x * kSolveRowsWide;
  for (int i = r0 + wave; i < r0 + kSolveRowsWide && i < sz; i += kSolveThreads / 64) {
    const double li = lc[i];
    double* row = mat + static_cast<int64_t>(i) * sz;
    for (int j = k + 1 + lane; j <= i; j += 64) row[j] -= li * lc[j];
    if (lane == 0) {
      mat[static_cast<int64_t>(k) * sz + i] = li;
      mat[static_cast<int64_t>(sz) * sz + static_cast<int64_t>(i) * sz + k] = li;
    }
  }
  if (blockIdx.x == 0 && tid == 0) ldiag[k] = lkk;
}

// The same factorisation for sizes up to kCholLdsN, one workgroup per matrix with the matrix in
// LDS: one launch instead of one per column, and bit-identical to it (the same operations on every
// entry in the same order).  grid.x = 0: A^T A + lam I, 1: Z^T Z + lam I.
constexpr int kCholLdsN = 128, kCholThreads = 1024;
__global__ __launch_bounds__(kCholThreads) void fit_chol_lds_kernel(const SolveArgs a) {
  constexpr int LD = kCholLdsN + 1;
  __shared__ double m[kCholLdsN * LD];
  __shared__ double lc[kCholLdsN];
  const int layer = blockIdx.y, w = a.w, tid = threadIdx.x;
  const Slots s = slots(a.work, a.w, layer);
  const int r = static_cast<int>(s.job->rank);
  const bool zz = blockIdx.x == 1;
  const int sz = zz ? r : w;
  double* mat = zz ? s.y : s.x;
  double* ldiag = s.ldiag + (zz ? w : 0);
  for (int e = tid; e < sz * sz; e += kCholThreads) {
    const int i = e / sz, j = e % sz;
    if (j <= i) m[i * LD + j] = mat[static_cast<int64_t>(i) * sz + j];
  }
  __syncthreads();
  for (int k = 0; k < sz; ++k) {
    const double piv = m[k * LD + k];
    const double lkk = piv > 0.0 ? sqrt(piv) : kNaN;
    for (int i = k + 1 + tid; i < sz; i += kCholThreads) lc[i] = m[i * LD + k] / lkk;
    if (tid == 0) ldiag[k] = lkk;
    __syncthreads();
    // rows by wave, the row's columns by lane
    for (int i = k + 1 + (tid >> 6); i < sz; i += kCholThreads / 64) {
      const double li = lc[i];
      for (int j = k + 1 + (tid & 63); j <= i; j += 64) m[i * LD + j] -= li * lc[j];
    }
    // column k of L, as the per-column launches store it: the upper triangle and the row-major copy
    for (int i = k + 1 + tid; i < sz; i += kCholThreads) {
      mat[static_cast<int64_t>(k) * sz + i] = lc[i];
      mat[static_cast<int64_t>(sz) * sz + static_cast<int64_t>(i) * sz + k] = lc[i];
    }
    __syncthreads();
  }
}

// ---- triangular solves and outputs --------------------------------------------------------------
__device__ inline double readlane_f64(double v, int lane) {
  const int64_t b = __double_as_longlong(v);
  const int lo = __builtin_amdgcn_readlane(static_cast<int>(b), lane);
  const int hi = __builtin_amdgcn_readlane(static_cast<int>(b >> 32), lane);
  return __longlong_as_double((static_cast<int64_t>(hi) << 32) | static_cast<uint32_t>(lo));
}

// One wave solves (L L^T) x = b for one right-hand side held in LDS (xs[i], lane i % 64 owns
// entry i, so every LDS access is the lane's own).  Forward L y = b column by column: y_i =
// b_i / L_ii, then b_j -= L[j][i] y_i for j > i with column i of L read as row i of the upper
// triangle (`lu`, contiguous).  Backward L^T x = y the same way from the bottom: x_i = y_i / L_ii,
// then y_j -= L[i][j] x_i for j < i with row i of L read from the row-major copy (`lr`).  The
// entry of step i is broadcast from its owner lane.
__device__ inline void wave_chol_solve(const double* lu, const double* lr, const double* diag,
                                       int sz, double* xs) {
  const int lane = threadIdx.x & 63;
  for (int i = 0; i < sz; ++i) {
    double own = 0.0;
    if ((i & 63) == lane) {
      own = xs[i] / diag[i];
      xs[i] = own;
    }
    const double yi = readlane_f64(own, i & 63);
    const double* col = lu + static_cast<int64_t>(i) * sz;
    for (int j = i + 1 + ((lane - i - 1) & 63); j < sz; j += 64) xs[j] -= col[j] * yi;
  }
  for (int i = sz - 1; i >= 0; --i) {
    double own = 0.0;
    if ((i & 63) == lane) {
      own = xs[i] / diag[i];
      xs[i] = own;
    }
    const double xi = readlane_f64(own, i & 63);
    const double* row = lr + static_cast<int64_t>(i) * sz;
    for (int j = lane; j < i; j += 64) xs[j] -= row[j] * xi;
  }
}

// One wave per right-hand side, four per workgroup.  Waves [0, r): encoder column m,
// E[:, m] = (A^T A + lam I)^-1 P[0:w, m] -> w_enc[m, :]; waves [r, r + w): decoder row j,
// F[:, j] = (Z^T Z + lam I)^-1 P[w + j, :]^T -> w_dec[j, :].
__global__ __launch_bounds__(kSolveThreads) void fit_out_kernel(const SolveArgs a) {
  __shared__ double xs_all[kSolveThreads / 64][kFitMaxSolveWidth];
  const int layer = blockIdx.y, w = a.w, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const Slots s = slots(a.work, a.w, layer);
  const SolveJob jb = *s.job;
  const int r = static_cast<int>(jb.rank);
  const bool bf16 = a.bf16 != 0;
  const int t = blockIdx.x * (kSolveThreads / 64) + wave;
  double* xs = xs_all[wave];
  if (t < r) {
    for (int i = lane; i < w; i += 64) xs[i] = s.m[static_cast<int64_t>(i) * r + t];
    wave_chol_solve(s.x, s.x + static_cast<int64_t>(w) * w, s.ldiag, w, xs);
    for (int i = lane; i < w; i += 64) store_out(jb.w_enc, static_cast<int64_t>(t) * w + i, xs[i], bf16);
  } else if (t < r + w) {
    const int j = t - r;
    const double* b = s.m + static_cast<int64_t>(w + j) * r;
    for (int l = lane; l < r; l += 64) xs[l] = b[l];
    wave_chol_solve(s.y, s.y + static_cast<int64_t>(r) * r, s.ldiag + w, r, xs);
    for (int l = lane; l < r; l += 64) store_out(jb.w_dec, static_cast<int64_t>(j) * r + l, xs[l], bf16);
  }
}

template <int DH>
hipError_t launch_gram_dh(bool bf16, bool derope, const FitGramParams& p, dim3 grid,
                          hipStream_t stream) {
  if (bf16 && fit_full_gram(true, p.w)) {
    if (!derope) hipLaunchKernelGGL((fit_gram_full_bf16_kernel<DH, false, true>), grid, dim3(256), 0, stream, p);
    else if (p.g % 2 == 0) hipLaunchKernelGGL((fit_gram_full_bf16_kernel<DH, true, true>), grid, dim3(256), 0, stream, p);
    else hipLaunchKernelGGL((fit_gram_full_bf16_kernel<DH, true, false>), grid, dim3(256), 0, stream, p);
  } else if (bf16) {
    if (!derope) hipLaunchKernelGGL((fit_gram_bf16_kernel<DH, false, true>), grid, dim3(256), 0, stream, p);
    else if (p.g % 2 == 0) hipLaunchKernelGGL((fit_gram_bf16_kernel<DH, true, true>), grid, dim3(256), 0, stream, p);
    else hipLaunchKernelGGL((fit_gram_bf16_kernel<DH, true, false>), grid, dim3(256), 0, stream, p);
  } else {
    if (derope) hipLaunchKernelGGL((fit_gram_f32_kernel<DH, true>), grid, dim3(256), 0, stream, p);
    else hipLaunchKernelGGL((fit_gram_f32_kernel<DH, false>), grid, dim3(256), 0, stream, p);
  }
  return hipGetLastError();
}

}  // namespace

int64_t fit_upper_tiles(int w) {
  const int64_t nt = 2 * static_cast<int64_t>(w) / kTB;
  return nt * (nt + 1) / 2;
}

bool fit_full_gram(bool bf16, int w) { return bf16 && 2 * w == 2 * kTB; }

int64_t fit_units_per_slice(bool bf16, int w, int n_jobs) {
  return static_cast<int64_t>(n_jobs) * (fit_full_gram(bf16, w) ? 1 : fit_upper_tiles(w));
}

hipError_t launch_fit_gram(bool bf16, const FitGramParams& p, hipStream_t stream) {
  const int64_t units = static_cast<int64_t>(p.n_jobs) * fit_units_per_slice(bf16, p.w, 1) *
                        p.n_slices;
  const dim3 grid(static_cast<unsigned>(units));
  hipError_t e;
  switch (p.head_dim) {
    case 32: e = launch_gram_dh<32>(bf16, p.derope != 0, p, grid, stream); break;
    case 64: e = launch_gram_dh<64>(bf16, p.derope != 0, p, grid, stream); break;
    case 128: e = launch_gram_dh<128>(bf16, p.derope != 0, p, grid, stream); break;
    default: return hipErrorInvalidValue;
  }
  if (e != hipSuccess) return e;
  const int64_t bx = fit_upper_tiles(p.w) * 16;  // 32 x 32 sub-blocks of every upper tile
  hipLaunchKernelGGL(fit_gram_reduce_kernel, dim3(static_cast<unsigned>(bx), p.n_jobs), dim3(256),
                     0, stream, p);
  return hipGetLastError();
}

hipError_t fit_scratch(double** ptr) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static double* addr[kMaxDevices] = {};
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (addr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    addr[dev] = static_cast<double*>(p);
  }
  *ptr = addr[dev];
  return hipSuccess;
}

hipError_t launch_fit_solve(const FitSolveParams& p, hipStream_t stream) {
  const int n = 2 * p.w, layers = p.n_jobs;
  int rmax = 0;
  for (int l = 0; l < layers; ++l) rmax = p.jobs[l].rank > rmax ? p.jobs[l].rank : rmax;
  const dim3 block(kSolveThreads), wave(64);
  SolveArgs a{p.work, static_cast<double>(p.n_rows), p.lambda, p.w, 0, p.center, p.bf16};
  hipLaunchKernelGGL(fit_prep_kernel, dim3((n + kSolveRows - 1) / kSolveRows, layers), block, 0,
                     stream, p);
  // steps k0 .. n-3 (a trailing block of n - k0 - 1 <= kTailN rows) in one launch
  const int k0 = n - 1 - kTailN > -1 ? n - 1 - kTailN : -1;
  for (int k = -1; k < k0; ++k) {
    a.step = k;
    const int rows = n - k - 2;
    const int rpw = n <= 64 * kTridiagPre ? kSolveRows : kSolveRowsWide;
    const dim3 grid((rows + rpw - 1) / rpw, layers);
    if (n <= 64 * kTridiagPre) hipLaunchKernelGGL(fit_tridiag_pre_kernel, grid, block, 0, stream, a);
    else hipLaunchKernelGGL(fit_tridiag_kernel, grid, block, 0, stream, a);
  }
  a.step = k0;
  hipLaunchKernelGGL(fit_tridiag_tail_kernel, dim3(layers), dim3(kTailThreads), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const unsigned rt = static_cast<unsigned>((rmax + 63) / 64);
  hipLaunchKernelGGL(fit_bisect_kernel, dim3((rmax + 3) / 4, layers), wave, 0, stream, a);
  if (n <= kInverseLdsN)
    hipLaunchKernelGGL((fit_inverse_lds_kernel<kInverseLdsN, kInverseLdsThreads>),
                       dim3((rmax + kInverseLdsThreads - 1) / kInverseLdsThreads, layers), wave, 0,
                       stream, a);
  else
    hipLaunchKernelGGL((fit_inverse_lds_kernel<kMaxN, 1>), dim3(rmax, layers), wave, 0, stream, a);
  if (n <= 512)
    hipLaunchKernelGGL(fit_back_kernel<kBackColsNarrow>,
                       dim3((rmax + kBackColsNarrow - 1) / kBackColsNarrow, layers), block, 0,
                       stream, a);
  else
    hipLaunchKernelGGL(fit_back_kernel<kBackColsWide>,
                       dim3((rmax + kBackColsWide - 1) / kBackColsWide, layers), block, 0, stream,
                       a);
  hipLaunchKernelGGL(fit_project_kernel, dim3(n / 64, rt, layers), block, 0, stream, a);
  const unsigned tw = static_cast<unsigned>(p.w / 64);
  hipLaunchKernelGGL(fit_normal_kernel, dim3(rt * rt > tw * tw ? rt * rt : tw * tw, 2, layers),
                     block, 0, stream, a);
  const int sz = p.w > rmax ? p.w : rmax;
  if (sz <= kCholLdsN) {
    hipLaunchKernelGGL(fit_chol_lds_kernel, dim3(2, layers), dim3(kCholThreads), 0, stream, a);
  } else {
    for (int k = 0; k < sz; ++k) {
      a.step = k;
      const int rows = sz - k - 1;
      const int gx = rows > 0 ? (rows + kSolveRowsWide - 1) / kSolveRowsWide : 1;
      hipLaunchKernelGGL(fit_chol_kernel, dim3(gx, 2, layers), block, 0, stream, a);
    }
  }
  constexpr int kWaves = kSolveThreads / 64;
  hipLaunchKernelGGL(fit_out_kernel, dim3((rmax + p.w + kWaves - 1) / kWaves, layers), block, 0,
                     stream, a);
  return hipGetLastError();
}

}  // namespace scd
