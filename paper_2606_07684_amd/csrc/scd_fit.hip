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
// fp64 in one workgroup per layer (parallel cyclic Jacobi, then Cholesky solves).
#include "scd_device.h"

#include <mutex>

namespace scd {

using namespace dev;

// Device-resident scratch of the allocation-free solve (scd_fit_solve_noalloc): the solve's fp64
// Jacobi and solve matrices for as many layers as fit, reused launch after launch.  Each GPU the
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
__device__ inline int upper_index(int ti, int tj, int nt) {
  return ti * nt - ti * (ti - 1) / 2 + (tj - ti);
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
// fp64 solve, one workgroup of 1024 threads per layer.
// ---------------------------------------------------------------------------------------------
constexpr int kSolveThreads = 1024;

// Pair k of round `round` of the cyclic ("round-robin") ordering of n indices: the n/2 pairs of a
// round are disjoint and the n - 1 rounds visit every pair once.
__device__ inline void jacobi_pair(int round, int k, int n, int& lo, int& hi) {
  // round < m and k < n / 2 <= m, so both sums lie in [0, 2m): one conditional subtraction
  // replaces the modulo
  const int m = n - 1;
  int a, b;
  if (k == 0) {
    a = m;
    b = round;
  } else {
    a = round + k;
    a = a >= m ? a - m : a;
    b = round - k + m;
    b = b >= m ? b - m : b;
  }
  lo = a < b ? a : b;
  hi = a < b ? b : a;
}

// In-place Cholesky factor (lower triangle) of the dim x dim matrix at a (row stride ld).  A
// non-positive pivot leaves NaN, which then reaches every output of the solve.
__device__ void cholesky(double* a, int dim, int ld, double* piv) {
  const int tid = threadIdx.x;
  for (int k = 0; k < dim; ++k) {
    if (tid == 0) {
      const double d = a[k * ld + k];
      *piv = d > 0.0 ? sqrt(d) : __longlong_as_double(0x7ff8000000000000ll);
      a[k * ld + k] = *piv;
    }
    __syncthreads();
    const double pv = *piv;
    for (int i = k + 1 + tid; i < dim; i += kSolveThreads) a[i * ld + k] /= pv;
    __syncthreads();
    const int rem = dim - k - 1;
    for (int e = tid; e < rem * rem; e += kSolveThreads) {
      const int i = k + 1 + e / rem, j = k + 1 + e % rem;
      if (j <= i) a[i * ld + j] -= a[i * ld + k] * a[j * ld + k];
    }
    __syncthreads();
  }
}

// Solves (L L^T) x = b for one right-hand side held at x[0], x[xs], ... (in place).
__device__ void chol_solve(const double* l, int dim, int ld, double* x, int xs) {
  for (int i = 0; i < dim; ++i) {
    double s = x[i * xs];
    for (int j = 0; j < i; ++j) s -= l[i * ld + j] * x[j * xs];
    x[i * xs] = s / l[i * ld + i];
  }
  for (int i = dim - 1; i >= 0; --i) {
    double s = x[i * xs];
    for (int j = i + 1; j < dim; ++j) s -= l[j * ld + i] * x[j * xs];
    x[i * xs] = s / l[i * ld + i];
  }
}

__device__ inline void store_out(void* dst, int64_t i, double v, bool bf16) {
  if (bf16) static_cast<__bf16*>(dst)[i] = static_cast<__bf16>(static_cast<float>(v));
  else static_cast<float*>(dst)[i] = static_cast<float>(v);
}

__global__ __launch_bounds__(kSolveThreads) void fit_solve_kernel(const FitSolveParams p) {
  const int job = blockIdx.x;
  const FitSolveJob& jb = p.jobs[job];
  const int w = p.w, n = 2 * w, r = jb.rank, half = n / 2;
  const int tid = threadIdx.x;
  const bool bf16 = p.bf16 != 0;
  double* gc = p.work + static_cast<int64_t>(job) * 3 * n * n;  // centred Gram (kept)
  double* mj = gc + static_cast<int64_t>(n) * n;                 // Jacobi matrix, then V_r
  double* vj = mj + static_cast<int64_t>(n) * n;                 // eigenvectors, then G V_r
  const double rows = static_cast<double>(p.n_rows);

  __shared__ double rot_c[kFitMaxSolveWidth], rot_s[kFitMaxSolveWidth];
  __shared__ int sel[2 * kFitMaxSolveWidth];
  __shared__ int changed;
  __shared__ double piv, trace;

  // centred Gram G - s s^T / N (the Gram of the rows minus their mean), V = I, offsets
  for (int e = tid; e < n * n; e += kSolveThreads) {
    const int i = e / n, j = e % n;
    double g = jb.gram[e];
    if (p.center) g -= static_cast<double>(jb.colsum[i]) * static_cast<double>(jb.colsum[j]) / rows;
    gc[e] = g;
    mj[e] = g;
    vj[e] = i == j ? 1.0 : 0.0;
  }
  if (p.center) {
    for (int i = tid; i < w; i += kSolveThreads) {
      store_out(jb.mu_enc, i, static_cast<double>(jb.colsum[i]) / rows, bf16);
      store_out(jb.mu_dec, i, static_cast<double>(jb.colsum[w + i]) / rows, bf16);
    }
  }
  if (tid == 0) {
    trace = 0.0;
    changed = 0;
  }
  __syncthreads();
  if (tid == 0) {
    double t = 0.0;
    for (int i = 0; i < n; ++i) t += fabs(gc[i * n + i]);
    trace = t;
  }
  __syncthreads();
  // Rotations below these thresholds change the eigenvectors far below fp32 precision; lower
  // thresholds would keep rotating on roundoff (off-diagonal entries of about eps * lambda_max)
  // and never report convergence.
  const double floor_abs = 1e-15 * trace;

  // parallel cyclic Jacobi: every round applies n/2 disjoint rotations at once
  for (int sweep = 0; sweep < p.max_sweeps; ++sweep) {
    for (int round = 0; round < n - 1; ++round) {
      for (int k = tid; k < half; k += kSolveThreads) {
        int a, b;
        jacobi_pair(round, k, n, a, b);
        const double app = mj[a * n + a], aqq = mj[b * n + b], apq = mj[a * n + b];
        double cr = 1.0, sr = 0.0;
        if (fabs(apq) > floor_abs && fabs(apq) > 1e-12 * sqrt(fabs(app * aqq))) {
          // zero the (a, b) entry of J^T M J with J = [[c, s], [-s, c]] on (a, b)
          const double th = (aqq - app) / (2.0 * apq);
          const double t = (th >= 0.0 ? 1.0 : -1.0) / (fabs(th) + sqrt(th * th + 1.0));
          cr = 1.0 / sqrt(t * t + 1.0);
          sr = t * cr;
          changed = 1;
        }
        rot_c[k] = cr;
        rot_s[k] = sr;
      }
      __syncthreads();
      for (int e = tid; e < half * half; e += kSolveThreads) {
        const int P = e / half, Q = e % half;
        int p0, q0, p1, q1;
        jacobi_pair(round, P, n, p0, q0);
        jacobi_pair(round, Q, n, p1, q1);
        const double cP = rot_c[P], sP = rot_s[P], cQ = rot_c[Q], sQ = rot_s[Q];
        const double m00 = mj[p0 * n + p1], m01 = mj[p0 * n + q1];
        const double m10 = mj[q0 * n + p1], m11 = mj[q0 * n + q1];
        const double r0a = cP * m00 - sP * m10, r0b = cP * m01 - sP * m11;
        const double r1a = sP * m00 + cP * m10, r1b = sP * m01 + cP * m11;
        mj[p0 * n + p1] = cQ * r0a - sQ * r0b;
        mj[p0 * n + q1] = sQ * r0a + cQ * r0b;
        mj[q0 * n + p1] = cQ * r1a - sQ * r1b;
        mj[q0 * n + q1] = sQ * r1a + cQ * r1b;
      }
      for (int e = tid; e < n * half; e += kSolveThreads) {
        const int i = e / half, Q = e % half;
        int p1, q1;
        jacobi_pair(round, Q, n, p1, q1);
        const double cQ = rot_c[Q], sQ = rot_s[Q];
        const double a = vj[i * n + p1], b = vj[i * n + q1];
        vj[i * n + p1] = cQ * a - sQ * b;
        vj[i * n + q1] = sQ * a + cQ * b;
      }
      __syncthreads();
    }
    const int any = changed;
    __syncthreads();
    if (!any) break;
    if (tid == 0) changed = 0;
    __syncthreads();
  }

  // the r largest eigenvalues in decreasing order.  The order is total (NaN counts as -inf and
  // ties go to the lower index), so the ranks are a permutation of [0, n) and every sel[k], k < r,
  // is written even when non-finite inputs reached the matrix.
  for (int i = tid; i < n; i += kSolveThreads) {
    const double di = mj[i * n + i];
    const double li = isnan(di) ? -INFINITY : di;
    int cnt = 0;
    for (int j = 0; j < n; ++j) {
      const double dj = mj[j * n + j];
      const double lj = isnan(dj) ? -INFINITY : dj;
      cnt += (lj > li || (lj == li && j < i)) ? 1 : 0;
    }
    if (cnt < r) sel[cnt] = i;
  }
  __syncthreads();
  // V_r [n, r] (into the Jacobi matrix's storage), each column's largest-magnitude entry positive
  double* vr = mj;
  for (int k = tid; k < r; k += kSolveThreads) {
    const int col = sel[k];
    int imax = 0;
    double best = -1.0;
    for (int i = 0; i < n; ++i) {
      const double a = fabs(vj[i * n + col]);
      if (a > best) {
        best = a;
        imax = i;
      }
    }
    const double sg = vj[imax * n + col] < 0.0 ? -1.0 : 1.0;
    for (int i = 0; i < n; ++i) vr[i * r + k] = sg * vj[i * n + col];
  }
  __syncthreads();
  // P = G_c V_r [n, r]: rows [0, w) are A^T Z, rows [w, 2w) are (Z^T B)^T
  double* pm = vj;
  for (int e = tid; e < n * r; e += kSolveThreads) {
    const int i = e / r, k = e % r;
    double s = 0.0;
    for (int j = 0; j < n; ++j) s += gc[i * n + j] * vr[j * r + k];
    pm[e] = s;
  }
  __syncthreads();
  // Z^T Z + lam I = V_r^T P + lam I (r x r, in the centred Gram's lower-right block) and
  // A^T A + lam I (its upper-left block)
  double* c2 = gc + static_cast<int64_t>(w) * n + w;
  for (int e = tid; e < r * r; e += kSolveThreads) {
    const int k = e / r, l = e % r;
    double s = 0.0;
    for (int i = 0; i < n; ++i) s += vr[i * r + k] * pm[i * r + l];
    c2[k * n + l] = s + (k == l ? p.lambda : 0.0);
  }
  for (int i = tid; i < w; i += kSolveThreads) gc[i * n + i] += p.lambda;
  __syncthreads();
  cholesky(gc, w, n, &piv);
  cholesky(c2, r, n, &piv);
  // encoder E = (A^T A + lam I)^-1 A^T Z: column k of P's first w rows, in place
  for (int k = tid; k < r; k += kSolveThreads) chol_solve(gc, w, n, pm + k, r);
  // decoder F = (Z^T Z + lam I)^-1 Z^T B: column j of F is row w + j of P, in place
  for (int j = tid; j < w; j += kSolveThreads) chol_solve(c2, r, n, pm + static_cast<int64_t>(w + j) * r, 1);
  __syncthreads();
  // W_enc [r, w] = E^T and W_dec [w, r] = F^T, each rounded once
  for (int e = tid; e < r * w; e += kSolveThreads) {
    const int k = e / w, cc = e % w;
    store_out(jb.w_enc, e, pm[cc * r + k], bf16);
  }
  for (int e = tid; e < w * r; e += kSolveThreads)
    store_out(jb.w_dec, e, pm[static_cast<int64_t>(w) * r + e], bf16);
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
  hipLaunchKernelGGL(fit_solve_kernel, dim3(p.n_jobs), dim3(kSolveThreads), 0, stream, p);
  return hipGetLastError();
}

}  // namespace scd
