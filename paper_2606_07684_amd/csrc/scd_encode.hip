// Producer encode (Section 4.3.2, Eq. encode_z_kv; Section 4.4.1) on the bf16 path for gfx950:
//   Z_K = (rows(deRoPE(K)) - mu_K) W_enc,K^T,   Z_V = (rows(V) - mu_V) W_enc,V^T,   Z_H = H W_enc,H^T
// The step is bound by HBM reads of the K/V/H inputs (the codes are r/w of that traffic).
//
// A workgroup of 4 waves owns 128 input rows of one layer-branch and produces all RB*32 code
// columns for them.  Every wave streams its 32 rows straight from HBM into registers, 128 input
// columns (one chunk) at a time, one chunk ahead of use.  With deRoPE each lane loads the same
// 8 columns of both halves of a head, so every rotation pair meets in one lane; the rotated,
// offset-subtracted values are rounded to bf16 and used directly as the B operand of
// v_mfma_f32_32x32x16_bf16.  Each lane keeps the cosines and sines of its row in registers for
// all heads.  The encoder weight chunk (all code rows x 128 columns, rows permuted so each lane
// ends with 16 consecutive code columns of one row) is double-buffered in LDS and shared by the
// four waves.  Both operands visit the columns of a chunk in the same order, so the contraction
// is unchanged.
#include "scd_device.h"

namespace scd {
namespace {

using namespace dev;

constexpr int kThreads = 256;
constexpr int kChunk = 128;          // input columns per chunk
constexpr int kLdc = kChunk + 8;     // padded LDS row of a weight chunk (elements)

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

// RB = code blocks of 32 (rank <= 32*RB); DH = head_dim (64 or 128, used with deRoPE).
template <int RB, int DH>
__global__ __launch_bounds__(kThreads) void encode_bf16_kernel(GemmParams p) {
  extern __shared__ __attribute__((aligned(16))) uint16_t lds[];
  uint16_t* Es = lds;                               // [2][RB*32][kLdc]
  uint16_t* mus = lds + 2 * RB * 32 * kLdc;         // [K] (deRoPE'd-space offset)

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int h = lane >> 5;

  const int unit = xcd_remap(blockIdx.x, gridDim.x);
  const GemmJob job = p.jobs[job_of(p, unit)];
  const int R = job.n, K = job.k;
  const int64_t M = p.m;
  const int64_t row = static_cast<int64_t>(unit - job.tile_begin) * 128 + wave * 32 + (lane & 31);
  const bool valid = row < M;
  const bool derope = (job.flags & kDeropeIn) != 0;
  const bool sub_mu = (job.flags & kVecIn) != 0 && job.vec != nullptr;
  const uint16_t* X = static_cast<const uint16_t*>(job.a);
  const uint16_t* E = static_cast<const uint16_t*>(job.b);
  const uint16_t* mu = static_cast<const uint16_t*>(job.vec);
  const int nchunks = K / kChunk;

  // offsets -> LDS (whole row width)
  if (sub_mu) {
    for (int q = tid; q < K / 8; q += kThreads)
      *reinterpret_cast<uint4*>(mus + 8 * q) = *reinterpret_cast<const uint4*>(mu + 8 * q);
  }

  // weight chunk c -> LDS buffer b, asynchronously; code rows beyond R read row 0 and only feed
  // accumulator blocks that are never stored
  auto stage_weights = [&](int c, int b) {
    dma_rows(Es + b * RB * 32 * kLdc, RB * 32, kChunk / 8, kLdc / 8, wave, 4, lane, [&](int rho) {
      const int r = row_of_lds(rho);
      return E + static_cast<int64_t>(r < R ? r : 0) * K + c * kChunk;
    });
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
  uint4 xc[8], xn[8];
  // rows past the end read row 0 (always in bounds); their codes are never stored
  auto load_x = [&](int c, uint4* dst) {
#pragma unroll
    for (int s = 0; s < 8; ++s)
      dst[s] = *reinterpret_cast<const uint4*>(xrow + c * kChunk + chunk_col<DH>(s, h, derope));
  };

  f32x16 acc[RB];
#pragma unroll
  for (int b = 0; b < RB; ++b)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[b][e] = 0.f;

  stage_weights(0, 0);
  load_x(0, xc);
  wait_vmem();
  __syncthreads();

  for (int c = 0; c < nchunks; ++c) {
    const int buf = c & 1;
    if (c + 1 < nchunks) {
      stage_weights(c + 1, buf ^ 1);
      load_x(c + 1, xn);
    }
    // B operands, one (first half, second half) pair of k-steps at a time: deRoPE and offset in
    // fp32, one bf16 rounding, then the MFMAs of both steps.
    const uint16_t* eb = Es + buf * RB * 32 * kLdc + (lane & 31) * kLdc;
#pragma unroll
    for (int s = 0; s < 8; s += 2) {
      bf16x8 bu, bv;
      if (derope || sub_mu) {
        float u[8], v[8];
        unpack8(xc[s], u);
        unpack8(xc[s + 1], v);
        const int cu = c * kChunk + chunk_col<DH>(s, h, derope);
        const int cv = c * kChunk + chunk_col<DH>(s + 1, h, derope);
        if (derope) {
          constexpr int spH = DH / 16;
          const int o = (s % spH) >> 1;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float cc = cs_c[o][e], sn = cs_s[o][e];
            const float a = u[e], b = v[e];
            u[e] = a * cc + b * sn;
            v[e] = b * cc - a * sn;
          }
        }
        if (sub_mu) {
          float mu_u[8], mu_v[8];
          unpack8(*reinterpret_cast<const uint4*>(mus + cu), mu_u);
          unpack8(*reinterpret_cast<const uint4*>(mus + cv), mu_v);
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            u[e] -= mu_u[e];
            v[e] -= mu_v[e];
          }
        }
        bu = __builtin_bit_cast(bf16x8, pack8(u));
        bv = __builtin_bit_cast(bf16x8, pack8(v));
      } else {
        bu = __builtin_bit_cast(bf16x8, xc[s]);
        bv = __builtin_bit_cast(bf16x8, xc[s + 1]);
      }
      const int colu = chunk_col<DH>(s, h, derope), colv = chunk_col<DH>(s + 1, h, derope);
#pragma unroll
      for (int b = 0; b < RB; ++b) {
        const bf16x8 ae = *reinterpret_cast<const bf16x8*>(eb + b * 32 * kLdc + colu);
        acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ae, bu, acc[b], 0, 0, 0);
      }
#pragma unroll
      for (int b = 0; b < RB; ++b) {
        const bf16x8 ae = *reinterpret_cast<const bf16x8*>(eb + b * 32 * kLdc + colv);
        acc[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ae, bv, acc[b], 0, 0, 0);
      }
    }
    wait_vmem();
    __syncthreads();
#pragma unroll
    for (int s = 0; s < 8; ++s) xc[s] = xn[s];
  }

  if (!valid) return;
  // lane holds, for block b, code columns 32*b + 16*h + (0..15) of its row
  uint16_t* Zo = static_cast<uint16_t*>(job.c) + row * R;
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

template <int RB>
hipError_t launch_rb(int head_dim, const GemmParams& p, size_t lds, hipStream_t stream) {
  if (head_dim == 128)
    hipLaunchKernelGGL((encode_bf16_kernel<RB, 128>), dim3(p.total_tiles), dim3(kThreads), lds,
                       stream, p);
  else
    hipLaunchKernelGGL((encode_bf16_kernel<RB, 64>), dim3(p.total_tiles), dim3(kThreads), lds,
                       stream, p);
  return hipGetLastError();
}

}  // namespace

// Code blocks of 32 the kernel instance for `max_rank` computes (a template parameter).
int encode_code_blocks(int max_rank) {
  const int rb = (max_rank + 31) / 32;
  return rb <= 2 ? 2 : (rb <= 4 ? 4 : 8);
}

size_t encode_bf16_lds_bytes(int code_blocks, int k) {
  return static_cast<size_t>(2) * code_blocks * 32 * kLdc * 2 + static_cast<size_t>(k) * 2;
}

hipError_t launch_encode_bf16(const GemmParams& p, hipStream_t stream) {
  if (p.total_tiles <= 0) return hipSuccess;
  int max_r = 0, max_k = 0;
  for (int i = 0; i < p.n_jobs; ++i) {
    max_r = p.jobs[i].n > max_r ? p.jobs[i].n : max_r;
    max_k = p.jobs[i].k > max_k ? p.jobs[i].k : max_k;
  }
  const int rb = encode_code_blocks(max_r);
  const size_t lds = encode_bf16_lds_bytes(rb, max_k);
  if (rb == 2) return launch_rb<2>(p.head_dim, p, lds, stream);
  if (rb == 4) return launch_rb<4>(p.head_dim, p, lds, stream);
  return launch_rb<8>(p.head_dim, p, lds, stream);
}

}  // namespace scd
