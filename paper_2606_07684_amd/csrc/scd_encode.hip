// Producer encode (Section 4.3.2, Eq. encode_z_kv; Section 4.4.1) on the bf16 path for gfx950:
//   Z_K = (rows(deRoPE(K)) - mu_K) W_enc,K^T,   Z_V = (rows(V) - mu_V) W_enc,V^T,   Z_H = H W_enc,H^T
// The step is bound by HBM reads of the K/V/H inputs (the codes are r/w of that traffic).
//
// A workgroup of 4 waves owns 128 input rows of one layer-branch and produces up to 128 code
// columns for them (RB*32; a rank above 128 takes two workgroups per row tile, so every instance
// keeps two waves per SIMD).  Every wave streams its 32 rows straight from HBM into registers, 128 input
// columns (one chunk) at a time, one chunk ahead of use.  With deRoPE each lane loads the same
// 8 columns of both halves of a head, so every rotation pair meets in one lane; the rotated values
// are rounded to bf16 and used directly as the B operand of v_mfma_f32_32x32x16_bf16 (without
// deRoPE the loaded bf16 values are the operand as they are).  Each lane keeps the cosines and
// sines of its row in registers for all heads.  The encoder weight chunk (all code rows x 128
// columns, rows permuted so each lane ends with 16 consecutive code columns of one row) is
// double-buffered in LDS and shared by the four waves.  Both operands visit the columns of a chunk
// in the same order, so the contraction is unchanged.
//
// The offset is folded into the product: (X - 1 mu^T) E^T = X E^T - 1 (E mu)^T.  E mu is one more
// MFMA per k-step with mu as a B operand broadcast to all 32 columns; wave w computes it for the
// code blocks b = w (mod 4), the workgroup shares it through LDS and every lane subtracts it from
// its fp32 accumulators.  The offset therefore costs no per-element work and is never rounded.
#include "scd_device.h"

namespace scd {
namespace {

using namespace dev;

constexpr int kThreads = 256;
constexpr int kChunk = 128;          // input columns per chunk
constexpr int kLdcPad = kChunk + 8;  // padded LDS row of a weight chunk (elements)

// Column (within a chunk) that lane half h supplies to MFMA k-step s (0..7).  With deRoPE, even
// steps take the first half of a head and odd steps the matching second half:
//   d_h = 128: step s -> offset o = 16*(s/2), half (s&1);  d_h = 64: two heads per chunk.
template <int DH>
__device__ constexpr int chunk_col(int s, int h, bool derope) {
  if (!derope) return 16 * s + 8 * h;
  constexpr int steps_per_head = DH / 16;
  const int hc = s / steps_per_head, sw = s % steps_per_head;
  return hc * DH + (sw & 1) * (DH / 2) + 16 * (sw >> 1) + 8 * h;
}

// RB = code blocks of 32 (rank <= 32*RB); DH = head_dim (64 or 128, used with deRoPE);
// DEROPE = key jobs; MU = every job of the launch has an offset.
template <int RB, int DH, bool DEROPE, bool MU, int DEPTH>
__global__ __launch_bounds__(kThreads) void encode_bf16_kernel(GemmParams p) {
  constexpr int kMuBlocks = (RB + 3) / 4;  // offset blocks per wave (waves past RB idle)
  extern __shared__ __attribute__((aligned(16))) uint16_t lds[];
  // Weight chunk rows: padded (DEPTH 1) or swizzled without padding (DEPTH 2, where every wave must
  // issue a fixed number of copies so its waits can be counted).
  constexpr bool kSwz = DEPTH == 2;
  constexpr int kLdc = kSwz ? kChunk : kLdcPad;
  uint16_t* Es = lds;                               // [2][RB*32][kLdc]
  uint16_t* mus = lds + 2 * RB * 32 * kLdc;         // [K] (deRoPE'd-space offset)
  float* emu = reinterpret_cast<float*>(mus + (MU ? p.jobs[0].k : 0));  // [RB*32]: E mu

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int h = lane >> 5;

  const int unit = xcd_remap(blockIdx.x, gridDim.x);
  const GemmJob job = p.jobs[job_of(p, unit)];
  // A rank above RB*32 takes two workgroups per row tile, units 2i and 2i + 1, each producing
  // RB*32 (or the remaining) code columns of the same rows: consecutive units run on one XCD at
  // about the same time, so the second read of the rows mostly hits L2.
  const int n_split = (job.n + RB * 32 - 1) / (RB * 32);  // 1 or 2
  const int local = unit - job.tile_begin;
  const int code0 = (local % n_split) * RB * 32;
  const int R = job.n - code0 < RB * 32 ? job.n - code0 : RB * 32;  // code columns here
  const int K = job.k;
  const int64_t M = p.m;
  const int64_t row = static_cast<int64_t>(local / n_split) * 128 + wave * 32 + (lane & 31);
  const bool valid = row < M;
  constexpr bool derope = DEROPE;
  const uint16_t* X = static_cast<const uint16_t*>(job.a);
  const uint16_t* E = static_cast<const uint16_t*>(job.b) + static_cast<int64_t>(code0) * K;
  const uint16_t* mu = static_cast<const uint16_t*>(job.vec);
  const int nchunks = K / kChunk;

  // offsets -> LDS (whole row width)
  if (MU) {
    for (int q = tid; q < K / 8; q += kThreads)
      *reinterpret_cast<uint4*>(mus + 8 * q) = *reinterpret_cast<const uint4*>(mu + 8 * q);
  }

  // weight chunk c -> LDS buffer b, asynchronously; code rows beyond R read row 0 and only feed
  // accumulator blocks that are never stored.  Swizzled: RB*32 rows x 16 chunks of 16 bytes, chunk
  // q of row rho at q ^ (rho & 7), exactly 2*RB copies per wave.  Padded: rows of 17 slots, the
  // pad slot masked off.
  constexpr int kEDma = RB * 32 * (kChunk / 8) / kThreads;
  auto stage_weights = [&](int c, int b) {
    uint16_t* dst = Es + b * RB * 32 * kLdc;
    if constexpr (kSwz) {
#pragma unroll
      for (int j = 0; j < kEDma; ++j) {
        const int slot = (4 * j + wave) * 64 + lane;
        const int rho = slot >> 4, q = (slot & 15) ^ (rho & 7);
        const int r = row_of_lds(rho);
        __builtin_amdgcn_global_load_lds(
            E + static_cast<int64_t>(r < R ? r : 0) * K + c * kChunk + 8 * q,
            (lds_void_t)(dst + 8 * ((4 * j + wave) * 64)), 16, 0, 0);
      }
    } else {
      dma_rows(dst, RB * 32, kChunk / 8, kLdc / 8, wave, 4, lane, [&](int rho) {
        const int r = row_of_lds(rho);
        return E + static_cast<int64_t>(r < R ? r : 0) * K + c * kChunk;
      });
    }
  };
  // MFMA A fragment of weight block b at chunk column col (a multiple of 8) for this lane's row
  auto efrag = [&](const uint16_t* eb, int b, int col) {
    const int q = kSwz ? ((col >> 3) ^ (lane & 7)) : (col >> 3);
    return *reinterpret_cast<const bf16x8*>(eb + b * 32 * kLdc + 8 * q);
  };

  // this lane's rotation factors for every pair index it touches: i = 16*o + 8*h + e
  constexpr int kNo = DH / 32;  // 16-wide offsets per half head
  float cs_c[kNo][8], cs_s[kNo][8];
  if (derope) {
    const float2* cs_row = p.rope + static_cast<int64_t>(valid ? row_position(p, row) : 0) * (DH / 2);
#pragma unroll
    for (int o = 0; o < kNo; ++o)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float2 v = cs_row[16 * o + 8 * h + e];
        cs_c[o][e] = v.x;
        cs_s[o][e] = v.y;
      }
  }

  const uint16_t* xrow = X + (valid ? row : 0) * K;
  // rows past the end read row 0 (always in bounds); their codes are never stored
  auto load_x = [&](int c, uint4* dst) {
#pragma unroll
    for (int s = 0; s < 8; ++s)
      dst[s] = *reinterpret_cast<const uint4*>(xrow + c * kChunk + chunk_col<DH>(s, h, derope));
  };

  f32x16 acc[RB], accm[kMuBlocks];
#pragma unroll
  for (int b = 0; b < RB; ++b)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[b][e] = 0.f;
#pragma unroll
  for (int i = 0; i < kMuBlocks; ++i)
#pragma unroll
    for (int e = 0; e < 16; ++e) accm[i][e] = 0.f;

  // One chunk's MFMAs for input registers x (8 loads of this lane's row) against weight buffer buf.
  // Each weight fragment of k-step s + 1 (and the offset's) is read into the register its MFMA of
  // step s has just consumed, one read after each MFMA, so each LDS read has most of a step of
  // MFMAs to land instead of stalling the MFMA that needs it, with no second register set.
  // B operands come in (first half, second half) pairs: deRoPE in fp32 and one bf16 rounding
  // (keys), or the loaded values themselves.  Both operands visit the chunk's columns in the same
  // order, so the contraction is unchanged.  Every wave computes kMuBlocks offset blocks (blocks
  // past RB repeat block 0 and are never used), so every step has the same instructions.
  // The read-ahead keeps a step's fragments live across the next step's deRoPE; the key kernels
  // with four or more code blocks would then need more than half a SIMD's registers and drop to one
  // wave per SIMD, which costs more than the reads' latency (the second wave hides it), so they
  // read each step's fragments right before its MFMAs.
  constexpr bool kReadAhead = !(DEROPE && RB >= 4);
  constexpr int kStepMfma = RB + (MU ? kMuBlocks : 0);
  constexpr int kStepReads = RB + (MU ? kMuBlocks + 1 : 0);
  constexpr int kPairs = kStepMfma < kStepReads ? kStepMfma : kStepReads;
  auto compute_chunk = [&](int c, int buf, const uint4* x) {
    const uint16_t* eb = Es + buf * RB * 32 * kLdc + (lane & 31) * kLdc;
    bf16x8 f[RB], m[kMuBlocks], mu;
    auto read_step = [&](int s) {
      const int col = chunk_col<DH>(s, h, derope);
#pragma unroll
      for (int b = 0; b < RB; ++b) f[b] = efrag(eb, b, col);
      if constexpr (MU) {
#pragma unroll
        for (int i = 0; i < kMuBlocks; ++i) {
          const int b = wave + 4 * i;
          m[i] = efrag(eb, b < RB ? b : 0, col);
        }
        mu = *reinterpret_cast<const bf16x8*>(mus + c * kChunk + col);
      }
    };
    if constexpr (kReadAhead) read_step(0);
    bf16x8 bu, bv;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      if ((s & 1) == 0) {
        if constexpr (DEROPE) {
          float u[8], v[8];
          unpack8(x[s], u);
          unpack8(x[s + 1], v);
          constexpr int spH = DH / 16;
          const int o = (s % spH) >> 1;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float cc = cs_c[o][e], sn = cs_s[o][e];
            const float a = u[e], b = v[e];
            u[e] = a * cc + b * sn;
            v[e] = b * cc - a * sn;
          }
          bu = __builtin_bit_cast(bf16x8, pack8(u));
          bv = __builtin_bit_cast(bf16x8, pack8(v));
        } else {
          bu = __builtin_bit_cast(bf16x8, x[s]);
          bv = __builtin_bit_cast(bf16x8, x[s + 1]);
        }
      }
      const bf16x8 bx = (s & 1) ? bv : bu;
      if constexpr (!kReadAhead) {
        // each fragment read right before its MFMA (short-lived registers)
        const int col = chunk_col<DH>(s, h, derope);
#pragma unroll
        for (int b = 0; b < RB; ++b)
          acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(efrag(eb, b, col), bx, acc[b], 0, 0, 0);
        if constexpr (MU) {
          const bf16x8 mu_s = *reinterpret_cast<const bf16x8*>(mus + c * kChunk + col);
#pragma unroll
          for (int i = 0; i < kMuBlocks; ++i) {
            const int b = wave + 4 * i;
            if (b < RB)
              accm[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(efrag(eb, b, col), mu_s, accm[i],
                                                                0, 0, 0);
          }
        }
        continue;
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int b = 0; b < RB; ++b)
        acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[b], bx, acc[b], 0, 0, 0);
      if constexpr (MU) {
        // E mu for this wave's offset blocks: mu (same columns as the inputs) in every B column
#pragma unroll
        for (int i = 0; i < kMuBlocks; ++i)
          accm[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(m[i], mu, accm[i], 0, 0, 0);
      }
      if (kReadAhead && s + 1 < 8) {
        read_step(s + 1);
#pragma unroll
        for (int i = 0; i < kPairs; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
        if constexpr (kStepMfma > kPairs)
          __builtin_amdgcn_sched_group_barrier(0x008, kStepMfma - kPairs, 0);
        if constexpr (kStepReads > kPairs)
          __builtin_amdgcn_sched_group_barrier(0x100, kStepReads - kPairs, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  if constexpr (DEPTH == 1) {
  uint4 xc[8], xn[8];
  stage_weights(0, 0);
  load_x(0, xc);
  wait_vmem();
  lds_barrier();

  for (int c = 0; c < nchunks; ++c) {
    const int buf = c & 1;
    if (c + 1 < nchunks) {
      stage_weights(c + 1, buf ^ 1);
      load_x(c + 1, xn);
    }
    compute_chunk(c, buf, xc);
    wait_vmem();
    lds_barrier();
#pragma unroll
    for (int s = 0; s < 8; ++s) xc[s] = xn[s];
  }

  } else {
  // inputs two chunks ahead in a ring of three register sets; the chunk loop is unrolled by three
  // so every set keeps its registers (no copies of registers whose loads are in flight)
  constexpr int kWait8 = 8 | (0x7 << 4) | (0xF << 8);  // at most the 8 input loads of chunk c + 2
  uint4 x0[8], x1[8], x2[8];
  stage_weights(0, 0);
  load_x(0, x0);
  load_x(nchunks > 1 ? 1 : 0, x1);
  __builtin_amdgcn_s_waitcnt(kWait8);
  lds_barrier();
  const int last = nchunks - 1;
  auto step = [&](int c, uint4 (&xcur)[8], uint4 (&xfar)[8]) {
    const int buf = c & 1;
    // weights of chunk c + 1 and inputs of chunk c + 2 (past the end: in-bounds re-loads that are
    // never used, so every step issues the same loads and the compiler's counter waits can leave
    // the far inputs in flight)
    stage_weights(c + 1 < last ? c + 1 : last, buf ^ 1);
    __builtin_amdgcn_sched_barrier(0);
    load_x(c + 2 < last ? c + 2 : last, xfar);
    __builtin_amdgcn_sched_barrier(0);
    if (c < nchunks) compute_chunk(c, buf, xcur);
    // chunk c + 1's weights and inputs have landed once only chunk c + 2's 8 input loads are
    // pending; the barrier makes that true for every wave and retires this chunk's LDS reads.  The
    // scheduling fences keep each step's loads on their side of the count.
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(kWait8);
    lds_barrier();
    __builtin_amdgcn_sched_barrier(0);
  };
  // chunks run in threes; steps past the last chunk only keep the load pattern uniform
  for (int c = 0; c < nchunks; c += 3) {
    step(c, x0, x2);
    step(c + 1, x1, x0);
    step(c + 2, x2, x1);
  }
  wait_vmem();
  }
  if constexpr (MU) {
    // every B column of the offset product is the same: lanes 0 and 32 publish their 16 values
#pragma unroll
    for (int i = 0; i < kMuBlocks; ++i) {
      const int b = wave + 4 * i;
      if (b < RB && (lane & 31) == 0) {
#pragma unroll
        for (int e = 0; e < 16; ++e) emu[32 * b + 16 * h + e] = accm[i][e];
      }
    }
    __syncthreads();
#pragma unroll
    for (int b = 0; b < RB; ++b)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[b][e] -= emu[32 * b + 16 * h + e];
  }
  if (!valid) return;
  // lane holds, for block b, code columns code0 + 32*b + 16*h + (0..15) of its row
  uint16_t* Zo = static_cast<uint16_t*>(job.c) + row * job.n + code0;
#pragma unroll
  for (int b = 0; b < RB; ++b) {
    const int c0 = 32 * b + 16 * h;
    if (c0 >= R) continue;
    float y[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) y[e] = acc[b][e];
    uint4* d = reinterpret_cast<uint4*>(Zo + c0);
    d[0] = pack8(y);
    d[1] = pack8(y + 8);
  }
}

template <int RB, bool DEROPE, bool MU>
hipError_t launch_rb(int head_dim, const GemmParams& p, size_t lds, hipStream_t stream) {
  // long rows without deRoPE or offset (the H branch) prefetch two chunks ahead
  if constexpr (!DEROPE && !MU) {
    if (p.jobs[0].k >= 2048) {
      if (head_dim == 128)
        hipLaunchKernelGGL((encode_bf16_kernel<RB, 128, DEROPE, MU, 2>), dim3(p.total_tiles),
                           dim3(kThreads), lds, stream, p);
      else
        hipLaunchKernelGGL((encode_bf16_kernel<RB, 64, DEROPE, MU, 2>), dim3(p.total_tiles),
                           dim3(kThreads), lds, stream, p);
      return hipGetLastError();
    }
  }
  if (head_dim == 128)
    hipLaunchKernelGGL((encode_bf16_kernel<RB, 128, DEROPE, MU, 1>), dim3(p.total_tiles),
                       dim3(kThreads), lds, stream, p);
  else
    hipLaunchKernelGGL((encode_bf16_kernel<RB, 64, DEROPE, MU, 1>), dim3(p.total_tiles),
                       dim3(kThreads), lds, stream, p);
  return hipGetLastError();
}


template <int RB>
hipError_t launch_kind(bool derope, bool mu, int head_dim, const GemmParams& p, size_t lds,
                       hipStream_t stream) {
  if (derope)
    return mu ? launch_rb<RB, true, true>(head_dim, p, lds, stream)
              : launch_rb<RB, true, false>(head_dim, p, lds, stream);
  return mu ? launch_rb<RB, false, true>(head_dim, p, lds, stream)
            : launch_rb<RB, false, false>(head_dim, p, lds, stream);
}

}  // namespace

// Code blocks of 32 the kernel instance for `max_rank` computes (a template parameter); ranks
// above 128 take two workgroups of 4 blocks per row tile.
int encode_code_blocks(int max_rank) { return max_rank <= 64 ? 2 : 4; }

size_t encode_bf16_lds_bytes(int code_blocks, int k, bool mu) {
  return static_cast<size_t>(2) * code_blocks * 32 * kLdcPad * 2 +
         (mu ? static_cast<size_t>(k) * 2 + static_cast<size_t>(code_blocks) * 32 * 4 : 0);
}

hipError_t launch_encode_bf16(const GemmParams& p, hipStream_t stream) {
  if (p.total_tiles <= 0) return hipSuccess;
  // every job of a launch has the same width, the same deRoPE flag and an offset either on every
  // job or on none
  const int k = p.jobs[0].k;
  const bool derope = (p.jobs[0].flags & kDeropeIn) != 0;
  const bool mu = (p.jobs[0].flags & kVecIn) != 0 && p.jobs[0].vec != nullptr;
  int max_r = 0;
  for (int i = 0; i < p.n_jobs; ++i) {
    const GemmJob& j = p.jobs[i];
    if (j.k != k || ((j.flags & kDeropeIn) != 0) != derope ||
        (((j.flags & kVecIn) != 0 && j.vec != nullptr) != mu))
      return hipErrorInvalidValue;
    max_r = j.n > max_r ? j.n : max_r;
  }
  const int rb = encode_code_blocks(max_r);
  const size_t lds = encode_bf16_lds_bytes(rb, k, mu);
  if (rb == 2) return launch_kind<2>(derope, mu, p.head_dim, p, lds, stream);
  return launch_kind<4>(derope, mu, p.head_dim, p, lds, stream);
}

}  // namespace scd
