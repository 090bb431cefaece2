// Device helpers shared by the bf16 kernels of the SCD codec (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "scd_kernels.h"

namespace scd {
namespace dev {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void* lds_void_t;

constexpr int kNumXcd = 8;

template <int V> struct IntC { static constexpr int value = V; };

// Workgroups are dispatched round-robin over the XCDs; renumber them so that each XCD receives a
// contiguous range of work units (neighbouring units share operands through that XCD's L2).
__device__ inline int xcd_remap(int bid, int nb) {
  const int q = nb / kNumXcd, rem = nb % kNumXcd;
  const int x = bid % kNumXcd, i = bid / kNumXcd;
  return (x < rem ? x * (q + 1) : rem * (q + 1) + (x - rem) * q) + i;
}

// Index of the job that owns work unit `unit` (jobs are ordered by tile_begin).
__device__ inline int job_of(const GemmParams& p, int unit) {
  int j = 0;
  while (j + 1 < p.n_jobs && unit >= p.jobs[j + 1].tile_begin) ++j;
  return j;
}

// RoPE table row of code row `row` (token row / g): the token's position within its own request,
// clamped to the table.
__device__ inline int row_position(const GemmParams& p, int64_t row) {
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

// Request boundaries staged in LDS so that position lookups never wait on vector memory.
// A single request without cu_seqlens is staged as cu = {0, T} so every lookup takes one path.
struct LdsBatch {
  int cu[kMaxLdsSeqs + 1];
  int p0[kMaxLdsSeqs];
};

// Copies the batch descriptor into LDS.  Requires n_seqs <= kMaxLdsSeqs.
__device__ inline void stage_batch(const GemmParams& p, LdsBatch& b, int tid, int nthreads) {
  const int64_t n_tokens = p.m / p.g;
  for (int i = tid; i <= p.n_seqs; i += nthreads)
    b.cu[i] = p.cu_seqlens != nullptr ? p.cu_seqlens[i] : (i == 0 ? 0 : static_cast<int>(n_tokens));
  for (int i = tid; i < p.n_seqs; i += nthreads) b.p0[i] = p.pos0 != nullptr ? p.pos0[i] : 0;
}

// RoPE table row of code row `row` from the staged descriptor (see row_position).
__device__ inline int row_position_lds(const GemmParams& p, const LdsBatch& lb, int64_t row) {
  const int t = static_cast<int>(row / p.g);
  int lo = 0, hi = p.n_seqs - 1;  // largest b with cu[b] <= t
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (lb.cu[mid] <= t) lo = mid; else hi = mid - 1;
  }
  int64_t pos = static_cast<int64_t>(t - lb.cu[lo]) + lb.p0[lo];
  pos = pos < 0 ? 0 : (pos >= p.max_pos ? p.max_pos - 1 : pos);
  return static_cast<int>(pos);
}

// MFMA 32x32 output rows are (8a + 4h + b) for accumulator element r = 4a + b of lane half h.
// Storing operand row 16h + 4a + b at LDS row 8a + 4h + b of each 32-row block makes element r of
// lane half h hold operand row 16h + r: 16 consecutive rows (output channels) per lane.  This is
// the operand row held by LDS row rho.
__device__ inline int row_of_lds(int rho) {
  const int o = rho & 31;
  return (rho & ~31) | (16 * ((o >> 2) & 1) + 4 * (o >> 3) + (o & 3));
}

// SiLU x / (1 + e^-x) for outputs rounded to bf16 next: the hardware exponential and reciprocal
// (each within about an ulp of fp32, far inside that rounding) instead of an IEEE division, which
// costs about ten instructions per element.  For very negative x, e^-x overflows to inf and its
// reciprocal is 0, so the result is the limit -0.
__device__ inline float silu_bf16(float x) { return x * __builtin_amdgcn_rcpf(1.f + __expf(-x)); }

__device__ inline float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ inline uint32_t pack_bf16x2(float a, float b) {
  const uint32_t lo = __builtin_bit_cast(uint16_t, static_cast<__bf16>(a));
  const uint32_t hi = __builtin_bit_cast(uint16_t, static_cast<__bf16>(b));
  return lo | (hi << 16);
}
__device__ inline void unpack8(const uint4& v, float* f) {
  f[0] = bf16_lo(v.x); f[1] = bf16_hi(v.x); f[2] = bf16_lo(v.y); f[3] = bf16_hi(v.y);
  f[4] = bf16_lo(v.z); f[5] = bf16_hi(v.z); f[6] = bf16_lo(v.w); f[7] = bf16_hi(v.w);
}
__device__ inline uint4 pack8(const float* f) {
  uint4 v;
  v.x = pack_bf16x2(f[0], f[1]); v.y = pack_bf16x2(f[2], f[3]);
  v.z = pack_bf16x2(f[4], f[5]); v.w = pack_bf16x2(f[6], f[7]);
  return v;
}
__device__ inline u32x4 as_u32x4(const uint4& v) { return u32x4{v.x, v.y, v.z, v.w}; }

// Direct global -> LDS copy of `nrows` rows of `chunks` 16-byte pieces into LDS rows of
// `stride` 16-byte slots (stride > chunks pads each row so MFMA operand reads hit distinct banks).
// Every wave of `nwaves` issues global_load_lds_dwordx4 for its share: lane i of one instruction
// fills slot base + i of the region, so the LDS address is uniform per instruction and padding
// slots are masked off.  LDS row rho receives the row src_row(rho) points to.  The copies complete
// asynchronously (vmcnt); wait for them and barrier before reading.
template <typename SrcRow>
__device__ inline void dma_rows(uint16_t* dst, int nrows, int chunks, int stride, int wave,
                                int nwaves, int lane, SrcRow src_row) {
  const int total = nrows * stride;
  for (int base = wave * 64; base < total; base += nwaves * 64) {
    const int slot = base + lane;
    const int rho = slot / stride, cc = slot - rho * stride;
    if (slot < total && cc < chunks)
      __builtin_amdgcn_global_load_lds(src_row(rho) + 8 * cc, (lds_void_t)(dst + 8 * base), 16,
                                       0, 0);
  }
}

// Wait until every vector-memory operation of this wave (loads, stores, LDS DMA) has completed.
__device__ inline void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Workgroup barrier that waits for this wave's LDS accesses only.  __syncthreads() carries a
// workgroup fence, which the compiler implements by also draining every vector-memory load and
// store in flight (so no copy or store can stay outstanding across it).  Wait explicitly
// (s_waitcnt) for the vector-memory operations a barrier publishes.  The memory clobber keeps the
// compiler from moving memory accesses across the barrier.
__device__ inline void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Workgroup barrier with no wait at all: it only brings the waves to the same point of their
// instruction streams (loads and stores in flight stay in flight).  Store-bound loops use it to
// keep the waves of a workgroup writing neighbouring addresses at the same time, which HBM
// serves better than the scattered stream of waves that drifted apart.
__device__ inline void wave_lockstep() { asm volatile("s_barrier" ::: "memory"); }

}  // namespace dev
}  // namespace scd
