// Internal declarations shared by the host library and the gfx950 kernels.
#pragma once

#include <hip/hip_bf16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace moba {

constexpr int kHeadDim = 128;     // D; every kernel is specialised for it
constexpr int kKeyTile = 64;      // keys per LDS tile in the attention kernels
constexpr int kTileRowsMfma = 256;  // query rows per bf16 (matrix-core) attention work-group
constexpr int kTileRowsF32 = 128;   // query rows per fp32 attention work-group
constexpr int kMaxGroup = 128;      // largest Hq / Hkv
constexpr int kMaxBlocksPerSeq = 4096;  // limit of the routing kernels' LDS tables
constexpr int kRouteRows = 1024;  // rows (tokens x query heads of a group) per routing chunk

// Per-sequence bookkeeping, built on the host and uploaded once per shape.
struct SeqInfo {
  int32_t tok_start;   // cu[s]
  int32_t len;         // cu[s+1] - cu[s]
  int32_t blk_off;     // global index of the sequence's block 0
  int32_t nblk;        // ceil(len / B)
  int32_t vt_tile_off; // first 64-key tile of the sequence in the packed V^T layout
  int32_t gate_off;    // first gate work-group of the sequence
  int32_t rc_off;      // first routing chunk of the sequence (per kv-head)
  int32_t pad0;
  int64_t hist_off;    // first routing-histogram word of the sequence (per kv-head)
};

// A causal tile: tokens [t0, t1) of sequence s attend keys [kbeg, token].
struct CausalTile {
  int32_t s;
  int32_t t0;
  int32_t t1;
  int32_t kbeg;
};

struct Problem {
  int64_t T;
  int Hq, Hkv, G, S;
  int B, topk;
  int nblk_total, nblk_max;
  int64_t vt_tiles;       // 64-key tiles per kv-head in the packed V^T layout
  int64_t gate_groups;    // gate work-groups per kv-head
  int gate_tw;            // tokens per gate work-group
  int64_t route_chunks;   // routing chunks per kv-head
  int route_rt;           // tokens per routing chunk
  int64_t hist_words;     // routing-histogram words per kv-head
  int64_t hist_entries;   // history selections over all rows and heads
  int tile_rows;          // query rows per attention work-group (history and causal tiles)
  // the selection's layout: row (t, kv-head g, head hl of the group) of sel
  // starts at (t * sel_st + g * sel_sg + hl) * topk.  [T, Hq, topk] for the
  // callers' arrays (sel_st = Hq, sel_sg = G); kv-head-major [Hkv, T, G, topk]
  // inside moba_forward and moba_backward (sel_st = G, sel_sg = T * G), so
  // a kv-head's rows are contiguous for the gate's writes and the routing.
  int64_t sel_st, sel_sg;
};

// ---------------------------------------------------------------- launches
// Every launcher enqueues on `st` and returns the launch status.
// kterm (nullable): also the three exact bf16 planes of kbar (hi, mid, lo;
// each [nblk_total, Hkv, D]) that the bf16 gate reads.
hipError_t launch_pool(const void* k, bool bf16, int64_t k_st, int64_t k_sh, const SeqInfo* seqs,
                       const Problem& p, float* kbar, __hip_bfloat16* kterm, hipStream_t st);

hipError_t launch_vt_pack(const __hip_bfloat16* v, int64_t v_st, int64_t v_sh, const SeqInfo* seqs,
                          const Problem& p, __hip_bfloat16* vt, hipStream_t st);

// bf16 queries read kterm (from launch_pool), fp32 queries kbar.
hipError_t launch_gate(const void* q, bool bf16, int64_t q_st, int64_t q_sh, const float* kbar,
                       const __hip_bfloat16* kterm, const SeqInfo* seqs, const Problem& p,
                       int32_t* sel, float* scores, int nmax, hipStream_t st);

struct RouteBuffers {
  int32_t* hist;            // [Hkv * hist_words]: per sequence, per block a column over the
                            // sequence's chunks: counts, then exclusive offsets
  int32_t* bin_count;       // [Hkv * nblk_total]
  int64_t* bin_start;       // [Hkv * nblk_total + 1]
  int32_t* bin_tile_start;  // [Hkv * nblk_total + 1] tiles of tile_rows entries
  uint32_t* entries;        // [hist_entries]
  int32_t* tile_bin;        // nullable: [tiles] the bin of every attention tile
};

// Attention tiles of the routing lists, at most: one per tile_rows entries
// plus one partial tile per bin.
inline int64_t route_tiles_bound(int64_t entries, int64_t nbins, int tile_rows) {
  return (entries + tile_rows - 1) / tile_rows + nbins;
}

hipError_t launch_route(const int32_t* sel, const SeqInfo* seqs, const Problem& p,
                        const RouteBuffers& rb, hipStream_t st);

struct AttnArgs {
  const void* q; int64_t q_st, q_sh;
  const void* k; int64_t k_st, k_sh;
  const void* v; int64_t v_st, v_sh;    // f32 path
  const __hip_bfloat16* vt;             // bf16 path: packed V^T tiles
  const SeqInfo* seqs;
  // history tiles
  const int32_t* bin_tile_start;
  const int64_t* bin_start;
  const int32_t* bin_count;
  const uint32_t* entries;
  const int32_t* tile_bin;  // the bin of every history tile
  void* o_part;     // [rows_chunk * (topk-1), D], normalised; bf16 on the bf16
                    // path, fp32 on the fp32 path
  float* lse_part;  // [rows_chunk * (topk-1)]
  // causal tiles
  const CausalTile* tiles;
  int64_t ntiles;
  // final output (current-block and dense tiles)
  void* out; int64_t o_st, o_sh;
  float* lse;
  int g0, g1;     // kv-heads of this chunk
  float scale_log2;
};

// History tiles: `grid` work-groups, an upper bound on the chunk's tiles
// (extra work-groups exit).  Causal tiles: a.ntiles x (g1 - g0) work-groups.
hipError_t launch_attn_hist_bf16(const AttnArgs& a, const Problem& p, int64_t grid, hipStream_t st);
hipError_t launch_attn_causal_bf16(bool dense, const AttnArgs& a, const Problem& p, hipStream_t st);
hipError_t launch_attn_hist_f32(const AttnArgs& a, const Problem& p, int64_t grid, hipStream_t st);
hipError_t launch_attn_causal_f32(bool dense, const AttnArgs& a, const Problem& p, hipStream_t st);
// bf16 path: folds the history partials of chunk rows into out / lse in place.
hipError_t launch_merge_bf16(const AttnArgs& a, const Problem& p, hipStream_t st);

// ------------------------------------------------------------ device helpers
// Largest s with key[s] <= x among sequences, skipping empty ones that share
// the same start.  `field` selects the per-sequence prefix being searched.
template <typename F>
__device__ __forceinline__ int find_seq(const SeqInfo* seqs, int S, int64_t x, F field) {
  int lo = 0, hi = S - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if ((int64_t)field(seqs[mid]) <= x) lo = mid; else hi = mid - 1;
  }
  return lo;
}

}  // namespace moba
