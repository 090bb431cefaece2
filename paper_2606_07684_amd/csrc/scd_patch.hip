// Patch KV regeneration (Section 4.4.2, Eq. kv_from_patch) as a bf16 MFMA GEMM for gfx950:
//   K = RoPE(H_hat W_K^T + b_K),  V = H_hat W_V^T + b_V   written straight into the KV cache.
// The same body regenerates a Patch layer from the aligner's hidden activations through the folded
// projections (act W_fold^T + c) and runs the aligner's own products.
//
// One workgroup computes a 256 (channels n) x 256 (tokens t) tile of C^T = W * H_hat^T with four
// waves, each owning 128 channels x 128 tokens as 8 x 8 blocks of v_mfma_f32_16x16x32_bf16.  The
// 16 x 16 x 32 shape does the same work per cycle as the 32 x 32 x 16 one with the same operand
// traffic, and this part holds a clearly higher clock under it: at equal MFMA-busy fractions, a
// build on the 32 x 32 shape ran this product at 1.6-1.7 GHz where the 16 x 16 shape ran at 1.9-2.0.
// The weight tile is the MFMA A operand, so an accumulator holds four channels of one token;
// weight rows are placed in LDS in a permuted order that gives each lane 8 consecutive channels of
// one token across a pair of blocks.  A wave's 128 channels are whole heads, so every RoPE pair
// (i, i + d_h/2) meets in one lane: bias, rotation and bf16 rounding happen in registers and each
// lane stores 16-byte vectors.
//
// K advances 64 at a time.  An operand tile of one 64-wide step (256 rows x 64 bf16 = 32 KiB, its
// 16-byte chunks XOR-swizzled so MFMA operand reads are conflict-free) fills one slot of a ring of
// five, the whole 160 KiB of LDS.  Both operand tiles travel global -> LDS directly
// (buffer_load_dwordx4 ... lds), eight lanes of a copy instruction reading one row's whole 128-byte
// line.  Each step is two 32-wide k-slices; the workgroup barrier sits between them, so the
// operand reads of the next step's first slice run under MFMAs.  The copies are spread over the
// step, one every four MFMAs after the slice's operand reads: the token tile of step k + 2 in the
// first slice (into the slot the previous barrier released) and the weight tile of step k + 2 in
// the second (into the slot this step's barrier released).  Issued in one burst, the 64 copies of
// a step (64 KiB per CU) would queue behind the texture path, and each stalled copy holds up the
// MFMAs behind it in the wave's instruction stream.
//
// The epilogue first stages the tile's RoPE factors (256 tokens x d_h/2 pairs, fp32) and bias in
// the then free LDS, so its stores never queue behind global loads (on this part loads and stores
// share one counter: a load issued after stores can only be waited for together with them).
#include "scd_device.h"

namespace scd {
namespace {

using namespace dev;

constexpr int kBM = kPatchBM;   // tokens per tile
constexpr int kBN = kPatchBN;   // channels per tile
constexpr int kBK = 64;                     // contraction step
constexpr int kLDK = kBK;                   // LDS row (bf16 elements): 8 16-byte chunks, swizzled
constexpr int kChunks = kBK / 8;
constexpr int kSlot = kBN * kLDK;           // elements per ring slot (one operand tile of a step)
constexpr int kRing = 5;                    // slots
constexpr int kWaves = 4;                   // one wave per SIMD
constexpr int kThreads = 64 * kWaves;
constexpr int kDmaIters = kBN * kChunks / kThreads;  // copy instructions per wave per operand tile
constexpr int kWaveTok = 128;               // tokens per wave (each wave owns 128 channels)
constexpr int kUB = kWaveTok / 16;          // 16-token MFMA blocks per wave
constexpr int kSB = 128 / 16;               // 16-channel MFMA blocks per wave
static_assert(kBN == kBM, "square tiles: both operand tiles fill one slot");
static_assert(kRing * kSlot * 2 <= 160 * 1024, "LDS");
static_assert(kBM * 32 * 16 + kBN * 2 <= kRing * kSlot * 2, "epilogue staging fits the ring");
// Fourth word of a raw buffer resource on gfx9-family parts: 32-bit data format, no swizzle.
constexpr int kBufferFlags = 0x00020000;

// Chunk c of LDS row r sits at chunk position c ^ swz(r).  A swizzle must depend on r % 16 only
// (fragment reads take it from the lane's row within a 16-row block); for 128-byte rows, r & 7 is
// conflict-free for the MFMA operand reads (eight lanes of a read hit eight distinct chunk
// positions of eight rows, all 32 banks once).
__device__ __forceinline__ int swz(int r) { return r & 7; }

// Weight row (within the tile) held by LDS row rho.  Element i of a 16 x 16 MFMA accumulator of
// lane l is output row 4 (l / 16) + i of its block; with this order, blocks 2p and 2p + 1 of a
// wave's 128 rows give lane l the channels 32p + 8 (l / 16) + (0..7), eight consecutive ones.
__device__ __forceinline__ int weight_row_of_lds(int rho) {
  const int s = (rho >> 4) & 7, m = rho & 15;
  return (rho & 128) | (32 * (s >> 1) + 8 * (m >> 2) + 4 * (s & 1) + (m & 3));
}

// s_waitcnt immediates: at most n vector-memory operations outstanding (optionally with every LDS
// access completed), or every LDS access completed.
constexpr int vmcnt_imm(int n, bool lds_done = false) {
  return (n & 15) | ((n >> 4) << 14) | (0x7 << 4) | ((lds_done ? 0 : 0xF) << 8);
}
constexpr int kLgkmDone = 0xF | (0x3 << 14) | (0x7 << 4);

// Scheduling groups for one slice of 64 MFMAs, in two halves of 32 with a scheduling fence
// between them (one solver region of all 64 MFMAs, 16 reads and 8 copies is not ordered as asked):
// in the first half one LDS read (operands of the next slice, which do not feed these MFMAs) after
// every second MFMA, in the second half one copy after every fourth.  (The compiler cannot tell
// that the copies and the reads touch different LDS slots, so it keeps them in program order:
// reads first.)
template <int I = 0>
__device__ __forceinline__ void interleave_reads() {
  if constexpr (I < 16) {
    __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    interleave_reads<I + 1>();
  }
}
template <int C, int I = 0>
__device__ __forceinline__ void interleave_copies() {
  static_assert(C >= 0 && C <= 8, "at most one copy per four MFMAs");
  if constexpr (I < C) {
    __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
    __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
    interleave_copies<C, I + 1>();
  } else if constexpr (C < 8) {
    __builtin_amdgcn_sched_group_barrier(0x008, 4 * (8 - C), 0);
  }
}

// The product C = A B^T of one launch (both operands row-major with the contraction contiguous,
// 256 x 256 tiles), with the epilogue the job flags select.  Two kernels run it: the Patch KV
// regeneration and the aligner in front of it, so profiles attribute each step to its own symbol.
__device__ __forceinline__ void patch_gemm_bf16(const GemmParams& p, uint16_t* smem) {

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wn = wave >> 1, wt = wave & 1;  // channel half, token half

  const int unit = xcd_remap(blockIdx.x, gridDim.x);
  const GemmJob job = p.jobs[job_of(p, unit)];
  const int local = unit - job.tile_begin;
  const int N = job.n, K = job.k;
  const int64_t M = p.m;
  const int ntn = (N + kBN - 1) / kBN;
  const int64_t t0 = static_cast<int64_t>(local / ntn) * kBM;
  const int n0 = (local % ntn) * kBN;
  const uint16_t* W = static_cast<const uint16_t*>(job.b);
  const uint16_t* Hh = static_cast<const uint16_t*>(job.a);
  const int nk = K / kBK;

  // Operand tile of step kc -> ring slot, asynchronously (buffer_load_dwordx4 ... lds).  A tile is
  // 256 rows x 8 chunks of 16 bytes = kDmaIters wave-wide instructions per wave; lane i of
  // instruction j of wave w fills chunk position (4j + w) * 64 + i (row / 8, position % 8) with the
  // chunk that belongs there.  Weight rows past N repeat row N - 1 and token rows past M repeat row
  // M - 1 (they only feed accumulators that are never stored), so no copy leaves the matrices.  The
  // buffer resources start at the tile's first weight row and first token row; a lane's byte
  // offsets then fit in 32 bits and the step's offset is one scalar.
  auto records = [](int64_t bytes) { return static_cast<int>(bytes < 0x7fffffff ? bytes : 0x7fffffff); };
  const __amdgpu_buffer_rsrc_t wres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(W + static_cast<int64_t>(n0) * K), 0,
      records(static_cast<int64_t>(N - n0) * K * 2), kBufferFlags);
  const __amdgpu_buffer_rsrc_t hres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(Hh + t0 * K), 0, records((M - t0) * K * 2), kBufferFlags);
  uint32_t woff[kDmaIters], hoff[kDmaIters];
#pragma unroll
  for (int j = 0; j < kDmaIters; ++j) {
    const int slot = (kWaves * j + wave) * 64 + lane;
    const int rho = slot / kChunks, c = (slot % kChunks) ^ swz(slot / kChunks);
    const int n = weight_row_of_lds(rho) < N - n0 ? weight_row_of_lds(rho) : N - n0 - 1;
    const int t = t0 + rho < M ? rho : static_cast<int>(M - 1 - t0);
    woff[j] = static_cast<uint32_t>((n * K + 8 * c) * 2);
    hoff[j] = static_cast<uint32_t>((t * K + 8 * c) * 2);
  }
  constexpr bool kTokens = true, kWeights = false;
  // copies j0 .. j1-1 of an operand tile (the whole tile is 0 .. kDmaIters-1)
  auto copy_part = [&](bool tokens, int kc, int slot, int j0, int j1) {
    uint16_t* dst = smem + slot * kSlot;
    const int kb = kc * kBK * 2;
#pragma unroll
    for (int j = j0; j < j1; ++j)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(tokens ? hres : wres,
                                               (lds_void_t)(dst + 8 * ((kWaves * j + wave) * 64)), 16,
                                               tokens ? hoff[j] : woff[j], kb, 0, 0);
  };
  auto copy_tile = [&](bool tokens, int kc, int slot) { copy_part(tokens, kc, slot, 0, kDmaIters); };

  f32x4 acc[kSB][kUB];
#pragma unroll
  for (int s = 0; s < kSB; ++s)
#pragma unroll
    for (int u = 0; u < kUB; ++u)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[s][u][e] = 0.f;

  const int lr = lane & 15, lq = lane >> 4;
  // Fragments of k-slice ks (32 wide) of the current stage: 8 weight blocks, 8 token blocks.  Lane
  // group q = l / 16 reads chunk 4 ks + q of its row; every block starts at a multiple of 16 rows,
  // so the row's swizzle is swz(lane % 16).
  auto frags = [&](const uint16_t* wb, const uint16_t* hb, int ks, bf16x8* af, bf16x8* bfr) {
    const int co = 8 * ((4 * ks + lq) ^ swz(lr));
#pragma unroll
    for (int s = 0; s < kSB; ++s)
      af[s] = *reinterpret_cast<const bf16x8*>(wb + s * 16 * kLDK + co);
#pragma unroll
    for (int u = 0; u < kUB; ++u)
      bfr[u] = *reinterpret_cast<const bf16x8*>(hb + u * 16 * kLDK + co);
  };
  // half h of a slice's MFMAs: weight blocks 4h .. 4h + 3 against every token block
  auto mma = [&](const bf16x8* af, const bf16x8* bfr, int h) {
#pragma unroll
    for (int s = 4 * h; s < 4 * h + 4; ++s)
#pragma unroll
      for (int u = 0; u < kUB; ++u)
        acc[s][u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[s], bfr[u], acc[s][u], 0, 0, 0);
  };

  // Copies in issue order: T0 W0 T1 W1 T2 W2 ... (token and weight tiles); the i-th goes to slot
  // i mod 5.  Step kc reads slots of T(kc) and W(kc); its first slice issues token tile kc + 2 into
  // the slot of weight tile kc - 1 (released at the previous barrier) and its second slice weight
  // tile kc + 2 into the slot of token tile kc (released at its own barrier).  At the barrier of
  // step kc only token tile kc + 2 may still be in flight.  A step index past the end re-copies
  // the last step into a slot that is never read for data (its reads only feed the discarded
  // look-ahead of the final step), so every step issues the same copies and one counter
  // threshold holds throughout.
  auto clamp = [&](int kc) { return kc < nk ? kc : nk - 1; };
  copy_tile(kTokens, 0, 0);
  copy_tile(kWeights, 0, 1);
  copy_tile(kTokens, clamp(1), 2);
  copy_tile(kWeights, clamp(1), 3);
  // step 0's two tiles have landed once at most the last two copies are pending
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(2 * kDmaIters, true));
  lds_barrier();
  const uint16_t* wrow = smem + (wn * 128 + lr) * kLDK;
  const uint16_t* hrow = smem + (wt * kWaveTok + lr) * kLDK;
  bf16x8 a0[kSB], b0[kUB], a1[kSB], b1[kUB];
  int sh = 0, sw = 1, sfree = 4;  // slots of step kc's token and weight tiles; slot for T(kc+2)
  frags(wrow + sw * kSlot, hrow + sh * kSlot, 0, a0, b0);
  for (int kc = 0; kc < nk; ++kc) {
    const int next_h = sh + 2 >= kRing ? sh + 2 - kRing : sh + 2;
    const int next_w = sw + 2 >= kRing ? sw + 2 - kRing : sw + 2;
    __builtin_amdgcn_s_waitcnt(kLgkmDone);
    __builtin_amdgcn_sched_barrier(0);
    mma(a0, b0, 0);
    frags(wrow + sw * kSlot, hrow + sh * kSlot, 1, a1, b1);
    interleave_reads();
    __builtin_amdgcn_sched_barrier(0);
    mma(a0, b0, 1);
    copy_tile(kTokens, clamp(kc + 2), sfree);
    interleave_copies<kDmaIters>();
    __builtin_amdgcn_sched_barrier(0);
    // Step kc + 1's tiles have landed once at most token tile kc + 2's copies are pending.
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(kDmaIters, true));
    lds_barrier();
    __builtin_amdgcn_sched_barrier(0);
    mma(a1, b1, 0);
    frags(wrow + next_w * kSlot, hrow + next_h * kSlot, 0, a0, b0);
    interleave_reads();
    __builtin_amdgcn_sched_barrier(0);
    mma(a1, b1, 1);
    copy_tile(kWeights, clamp(kc + 2), sh);
    interleave_copies<kDmaIters>();
    __builtin_amdgcn_sched_barrier(0);
    sfree = sw;
    sh = next_h;
    sw = next_w;
  }
  // drain the look-ahead copies and every wave's operand reads: the ring is free from here on
  wait_vmem();
  lds_barrier();

  // Epilogue.  Lane l holds, for blocks (2p + b, u), token t0 + wt*kWaveTok + 16u + l%16 and
  // channels n0 + wn*128 + 32p + 8*(l/16) + 4b + i, i = 0..3.
  const bool rope = (job.flags & kRopeOut) != 0;
  const bool silu = (job.flags & kSiluOut) != 0;
  const bool add_vec = (job.flags & kVecOut) != 0 && job.vec != nullptr;
  const uint16_t* bias = static_cast<const uint16_t*>(job.vec);
  uint16_t* C = static_cast<uint16_t*>(job.c);
  const int dh = p.head_dim, half = dh >> 1;
  // Block pairs p that hold (i, i + d_h/2): (0,2),(1,3) for d_h = 128; (0,1),(2,3) for 64.
  const int pstride = half >> 5;  // 2 or 1
  const int nw = n0 + wn * 128;
  const int ql = 8 * lq;
  // The tile's RoPE factors and bias are staged in the (now free) LDS first, so the epilogue's
  // stores never wait behind global loads.  Factors: 16-byte chunk c (pairs 2c, 2c + 1) of token
  // r's table row at byte (c * 256 + r) * 16, so the lanes of a read (consecutive tokens) hit
  // consecutive chunks; one DMA instruction fills 64 consecutive chunk slots, and a lane always
  // fetches the same token (its row position is looked up once).  Bias: 256 bf16 after them.
  unsigned char* stage = reinterpret_cast<unsigned char*>(smem);
  uint16_t* sbias = reinterpret_cast<uint16_t*>(stage + kBM * 32 * 16);
  if (rope) {
    const int nchunk = half / 2;  // chunks per token row
    const int r = ((wave % (kBM / 64)) * 64) + lane;
    const int64_t tr = t0 + r < M ? t0 + r : M - 1;
    const float2* src = p.rope + static_cast<int64_t>(row_position(p, tr)) * half;
    for (int j = 0; j < nchunk * kBM / (64 * kWaves); ++j) {
      const int slot = (j * kWaves + wave) * 64;  // first chunk slot of this instruction
      const int c = slot / kBM;
      __builtin_amdgcn_global_load_lds(src + 2 * c, (lds_void_t)(stage + 16 * slot), 16, 0, 0);
    }
  }
  if (add_vec && tid < kBN / 8) {
    const int nb = n0 + 8 * tid;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (nb < N) v = *reinterpret_cast<const uint4*>(bias + nb);
    *reinterpret_cast<uint4*>(sbias + 8 * tid) = v;
  }
  wait_vmem();
  lds_barrier();

  auto load8 = [&](int nb, float* v) {
    if (add_vec) {
      const uint4 x = *reinterpret_cast<const uint4*>(sbias + (nb - n0));
      v[0] = bf16_lo(x.x); v[1] = bf16_hi(x.x);
      v[2] = bf16_lo(x.y); v[3] = bf16_hi(x.y);
      v[4] = bf16_lo(x.z); v[5] = bf16_hi(x.z);
      v[6] = bf16_lo(x.w); v[7] = bf16_hi(x.w);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = 0.f;
    }
  };
  auto store8 = [&](int64_t t, int nb, const float* y) {
    if (nb >= N) return;
    uint4 o;
    o.x = pack_bf16x2(y[0], y[1]);
    o.y = pack_bf16x2(y[2], y[3]);
    o.z = pack_bf16x2(y[4], y[5]);
    o.w = pack_bf16x2(y[6], y[7]);
    *reinterpret_cast<uint4*>(C + t * N + nb) = o;
  };

  // One pair of block pairs (P, P + PS) holds channels (i, i + d_h/2); P and PS are compile-time so
  // the accumulators stay in registers.  rl is the token's row within the tile.
  auto finish_pair = [&](auto p_c, auto ps_c, int u, int64_t t, int rl) {
    constexpr int P = decltype(p_c)::value;
    constexpr int PP = P + decltype(ps_c)::value;
    const int nb = nw + 32 * P + ql, nbp = nw + 32 * PP + ql;
    float a[8], b[8];
    load8(nb, a);
    load8(nbp, b);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      a[i] += acc[2 * P][u][i];
      a[4 + i] += acc[2 * P + 1][u][i];
      b[i] += acc[2 * PP][u][i];
      b[4 + i] += acc[2 * PP + 1][u][i];
    }
    if (silu) {
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        a[r] = silu_bf16(a[r]);
        b[r] = silu_bf16(b[r]);
      }
    }
    if (rope) {
      const int c0 = ((32 * P + ql) & (half - 1)) >> 1;  // chunk of the pair of channel r = 0
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 cs = *reinterpret_cast<const float4*>(stage + ((c0 + q) * kBM + rl) * 16);
        const float x0 = a[2 * q], y0 = b[2 * q], x1 = a[2 * q + 1], y1 = b[2 * q + 1];
        a[2 * q] = x0 * cs.x - y0 * cs.y;
        b[2 * q] = y0 * cs.x + x0 * cs.y;
        a[2 * q + 1] = x1 * cs.z - y1 * cs.w;
        b[2 * q + 1] = y1 * cs.z + x1 * cs.w;
      }
    }
    store8(t, nb, a);
    store8(t, nbp, b);
  };

#pragma unroll
  for (int u = 0; u < kUB; ++u) {
    const int rl = wt * kWaveTok + 16 * u + lr;
    const int64_t t = t0 + rl;
    if (t >= M) continue;
    if (pstride == 2) {
      finish_pair(IntC<0>{}, IntC<2>{}, u, t, rl);
      finish_pair(IntC<1>{}, IntC<2>{}, u, t, rl);
    } else {
      finish_pair(IntC<0>{}, IntC<1>{}, u, t, rl);
      finish_pair(IntC<2>{}, IntC<1>{}, u, t, rl);
    }
  }
}

constexpr int kSmemElems = kRing * kSlot;
__global__ __launch_bounds__(kThreads, 1) void patch_kv_bf16_kernel(GemmParams p) {
  __shared__ __attribute__((aligned(16))) uint16_t smem[kSmemElems];
  patch_gemm_bf16(p, smem);
}

__global__ __launch_bounds__(kThreads, 1) void patch_align_bf16_kernel(GemmParams p) {
  __shared__ __attribute__((aligned(16))) uint16_t smem[kSmemElems];
  patch_gemm_bf16(p, smem);
}

}  // namespace

hipError_t launch_patch_bf16(const GemmParams& p, hipStream_t stream) {
  if (p.total_tiles <= 0) return hipSuccess;
  hipLaunchKernelGGL(patch_kv_bf16_kernel, dim3(p.total_tiles), dim3(kThreads), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_align_bf16(const GemmParams& p, hipStream_t stream) {
  if (p.total_tiles <= 0) return hipSuccess;
  hipLaunchKernelGGL(patch_align_bf16_kernel, dim3(p.total_tiles), dim3(kThreads), 0, stream, p);
  return hipGetLastError();
}

}  // namespace scd
