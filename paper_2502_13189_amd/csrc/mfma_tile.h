// Building blocks of the bf16 attention kernels on the gfx950 matrix cores
// (v_mfma_f32_32x32x16_bf16), shared by the forward and backward kernels:
// operand types, the LDS DMA of 64-key K / V tiles and packed V^T-style tiles,
// and the 16-MFMA operand pipelines.
//
// The accumulator layout of a 32x32 MFMA gives lane l the column l % 32 and
// rows 8*(i/4) + 4*(l/32) + i%4 for its 16 values i; so the 8 keys a lane
// feeds into one k=16 step of a product that reduces over keys are keys
// {0-3, 8-11} (+4 for the upper half-wave) of a 16-key group, which is the
// order the packed ("transposed") tiles store them in.
//
// LDS rows are padded by one 16-byte chunk (row-major K/V tiles: 64 rows of
// 17 chunks; packed tiles: 128 rows of 9 chunks; the pad chunk receives a
// copy of the row's last chunk), so an operand read, 16 lanes on 16
// consecutive rows at one chunk, hits 16 distinct bank groups, and each
// global_load_lds_dwordx4 (lane L to 16-byte chunk L, 1 KiB per instruction)
// writes whole padded rows.
#pragma once

#include "moba_internal.h"

namespace moba {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));  // one 16-byte chunk

constexpr int kChunksV = kHeadDim * kKeyTile / 8;  // 16-byte chunks per V^T tile (1024)
constexpr int kRowK = kHeadDim / 8 + 1;            // LDS K row: 16 chunks + 1 pad
constexpr int kRowV = kKeyTile / 8 + 1;            // LDS V^T row: 8 chunks + 1 pad
constexpr int kBufK = kKeyTile * kRowK;            // 1088 chunks
constexpr int kBufV = kHeadDim * kRowV;            // 1152 chunks
constexpr int kDmaK = kBufK / 64;                  // DMA instructions per K tile (17)
constexpr int kDmaV = kBufV / 64;                  // DMA instructions per V^T tile (18)
static_assert(kBufK % 64 == 0 && kBufV % 64 == 0, "DMA windows cover whole buffers");

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 u) { return __builtin_bit_cast(bf16x8, u); }

// Two fp32 values to a packed bf16 pair, round-to-nearest-even.
__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  const f32x2 v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

__device__ __forceinline__ float xor32(float v) { return __shfl_xor(v, 32, 64); }

__device__ __forceinline__ int64_t uniform64(int64_t v) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)v >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

__device__ __forceinline__ f32x16 mfma(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Global sources of this thread's lane in the LDS DMA of a tile.  DMA
// instruction j writes buffer chunks 64j .. 64j+63; wave w issues j = w + 8x
// (x = 0..2, while j < kDmaK or kDmaV).  Lane L of instruction j fills chunk
// p = 64j + L: K row p / 17, chunk min(p % 17, 15); V^T row p / 9, chunk
// min(p % 9, 7).  Addresses are a wave-uniform base plus a 32-bit per-lane
// byte offset.
struct Dma {
  const char* kbase;  // K of this kv-head at the sequence start (uniform)
  int64_t k_tile;     // bytes between consecutive key tiles (uniform)
  int64_t len;        // sequence length
  const char* klast;  // the sequence's last key row (uniform)
  uint32_t koff[3];   // per-lane byte offset of the chunk within a tile
  uint32_t kcol[3];   // per-lane byte offset of the chunk within its row
  int krow[3];        // tile row of the lane's chunk
  const char* vbase;  // packed V^T tile 0 (uniform)
  uint32_t voff[3];
  int wave;           // wave-uniform
};

// One LDS DMA instruction: 16 bytes per lane from global memory into LDS,
// lane L to 16-byte chunk L of the 1 KiB at ldst (global_load_lds_dwordx4,
// the LDS address in M0).  Issued as inline assembly, so the compiler does not
// count it as an LDS write: it would otherwise wait for every DMA in flight
// before any later LDS read it cannot prove disjoint from the DMA's target
// (which it cannot for buffers chosen at run time), defeating the prefetch.
// Every caller therefore waits for its DMA explicitly (dma_wait) before the
// barrier that publishes the data.
__device__ __forceinline__ uint32_t lds_addr(const u32x4* p) {
  return __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p);
}

// A per-lane 64-bit source address (gathered rows).
__device__ __forceinline__ void dma16(const void* gsrc, u32x4* ldst) {
  asm volatile("global_load_lds_dwordx4 %0, off" : : "v"(gsrc), "{m0}"(lds_addr(ldst)) : "memory");
}

// A wave-uniform base (scalar registers) plus a 32-bit per-lane byte offset:
// one vector register per address instead of two, which keeps the attention
// kernels' register allocation free of spills.
__device__ __forceinline__ void dma16_at(const char* base, uint32_t off, u32x4* ldst) {
  asm volatile("global_load_lds_dwordx4 %0, %1"
               : : "v"(off), "s"(base), "{m0}"(lds_addr(ldst)) : "memory");
}

__device__ __forceinline__ void dma_k1(const Dma& D, const char* tile, bool tail, int64_t base,
                                       u32x4* buf, int x) {
  uint32_t off = D.koff[x];
  // rows past the sequence end repeat its last key; they are always masked
  // (the tile starts at or before the last key, so the offset stays >= 0)
  if (tail && base + D.krow[x] >= D.len) off = (uint32_t)(D.klast - tile) + D.kcol[x];
  dma16_at(tile, off, buf + 64 * (D.wave + 8 * x));
}

__device__ __forceinline__ void dma_k(const Dma& D, int i, u32x4* buf) {
  const int64_t base = (int64_t)i * kKeyTile;
  const char* tile = D.kbase + (int64_t)i * D.k_tile;
  if (base + kKeyTile <= D.len) {
    dma_k1(D, tile, false, base, buf, 0);
    dma_k1(D, tile, false, base, buf, 1);
    if (D.wave + 16 < kDmaK) dma_k1(D, tile, false, base, buf, 2);
  } else {
    dma_k1(D, tile, true, base, buf, 0);
    dma_k1(D, tile, true, base, buf, 1);
    if (D.wave + 16 < kDmaK) dma_k1(D, tile, true, base, buf, 2);
  }
}

__device__ __forceinline__ void dma_v1(const Dma& D, const char* tile, u32x4* buf, int x) {
  dma16_at(tile, D.voff[x], buf + 64 * (D.wave + 8 * x));
}

__device__ __forceinline__ void dma_v(const Dma& D, int i, u32x4* buf) {
  const char* tile = D.vbase + (int64_t)i * (kChunksV * 16);
  dma_v1(D, tile, buf, 0);
  dma_v1(D, tile, buf, 1);
  if (D.wave + 16 < kDmaV) dma_v1(D, tile, buf, 2);
}

// Wait for this wave's LDS DMA (and everything else) before a barrier.
__device__ __forceinline__ void dma_wait() { __builtin_amdgcn_s_waitcnt(0); }

// Lane read bases (chunks) into a K and a V^T buffer: K row 32*th + qc,
// chunk 2kk + hh is kq + 32*kRowK*th + 2kk; V^T row 32*dt + qc, chunk
// 2st + hh is vq + 32*kRowV*dt + 2st.
struct ReadOff {
  int kq;
  int vq;
};

// Operand reads run kPre MFMAs ahead of their use: the first kPre LDS reads,
// then one MFMA and one read alternately, then the last kPre MFMAs (pinned
// with scheduling groups, so the LDS latency hides behind the matrix core).
constexpr int kPre = 6;

__device__ __forceinline__ void pin_pipeline() {
  __builtin_amdgcn_sched_group_barrier(0x100, kPre, 0);
#pragma unroll
  for (int j = 0; j < 16 - kPre; j++) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, kPre, 0);
}

// S^T: 16 MFMAs from the K buffer at kb.
__device__ __forceinline__ void qk(f32x16 (&s)[2], const u32x4* kb, const ReadOff& ro,
                                   const bf16x8 (&qf)[8]) {
#pragma unroll
  for (int th = 0; th < 2; th++)
#pragma unroll
    for (int r = 0; r < 16; r++) s[th][r] = 0.0f;
  const u32x4* k = kb + ro.kq;
  u32x4 op[16];
#pragma unroll
  for (int j = 0; j < 16; j++) op[j] = k[32 * kRowK * (j & 1) + 2 * (j >> 1)];
#pragma unroll
  for (int j = 0; j < 16; j++) s[j & 1] = mfma(as_bf16x8(op[j]), qf[j >> 1], s[j & 1]);
  pin_pipeline();
}

// O^T += V^T . P^T: 16 MFMAs from the V^T buffer at vb.
__device__ __forceinline__ void pv(f32x16 (&o)[4], const u32x4* vb, const ReadOff& ro,
                                   const bf16x8 (&pb)[4]) {
  const u32x4* v = vb + ro.vq;
  u32x4 op[16];
#pragma unroll
  for (int j = 0; j < 16; j++) op[j] = v[32 * kRowV * (j & 3) + 2 * (j >> 2)];
#pragma unroll
  for (int j = 0; j < 16; j++) o[j & 3] = mfma(as_bf16x8(op[j]), pb[j >> 2], o[j & 3]);
  pin_pipeline();
}

// Query row of one lane in a query-side tile.
struct RowInfo {
  int64_t t;
  int h;
  bool valid;
  int64_t dst;  // partial index (history) or chunk-relative row (current block)
};

// Edge tiles of S^T (keys x queries) keep only keys k of the 64-key tile with
// lo <= k < hi (others become -inf); lo and hi come relative to this lane's
// key offset 4*hh, so each element compares a compile-time constant with a
// lane value.
__device__ __forceinline__ void mask_keys(f32x16 (&s)[2], int lo, int hi) {
#pragma unroll
  for (int th = 0; th < 2; th++)
#pragma unroll
    for (int r = 0; r < 16; r++) {
      const int k = 32 * th + 8 * (r >> 2) + (r & 3);
      s[th][r] = (k >= lo && k < hi) ? s[th][r] : -INFINITY;
    }
}

}  // namespace moba
