// Internal declarations of the backward pass (gradients of MoBA attention
// w.r.t. q, k and v), shared by the host library and the gfx950 kernels.
#pragma once

#include "moba_internal.h"

namespace moba {

constexpr int kDkdvWaves = 8;                       // waves per dK/dV work-group (two per SIMD)
constexpr int kKeysPerDkdv = 32 * (kDkdvWaves / 2);  // keys per dK/dV work-group (32 per SIMD)

// Keys [k0, k1) of global block b; the block's tokens end at bend.  One dK/dV
// work-group per key tile and kv-head.
struct KeyTile {
  int32_t b;
  int32_t k0;
  int32_t k1;
  int32_t bend;
};

struct BwdArgs {
  const void* q; int64_t q_st, q_sh;
  const void* k; int64_t k_st, k_sh;
  const void* v; int64_t v_st, v_sh;
  const void* o; int64_t o_st, o_sh;
  const void* dout; int64_t do_st, do_sh;
  const float* lse;  // [Hq, T] natural-log lse of the forward
  void* dq; int64_t dq_st, dq_sh;
  void* dk; int64_t dk_st, dk_sh;
  void* dv; int64_t dv_st, dv_sh;
  const __hip_bfloat16* kt;  // packed K^T tiles (the V^T pack applied to K)
  const SeqInfo* seqs;
  // routing lists (null when no row has a history block)
  const int32_t* bin_tile_start;
  const int32_t* tile_bin;  // the bin of every history tile
  const int64_t* bin_start;
  const int32_t* bin_count;
  const uint32_t* entries;
  float2* ld;        // [Hq, T]: (lse * log2 e, Delta = <dO, O>)
  int4* rec;         // [hist_entries]: (t, h, lse * log2 e, Delta) of each routed entry
  float* dq_part;    // [rows_chunk * (topk-1), D] fp32, scaled history-slot dQ
  const CausalTile* tiles;
  int64_t ntiles;
  const KeyTile* ktiles;
  int64_t nktiles;
  int g0, g1;        // kv-heads of this chunk (dQ kernels)
  float scale_log2;  // log2(e) / sqrt(D)
  float scale;       // 1 / sqrt(D)
  // dK/dV hand-over wait: polls before a wave gives up, and an offset added
  // to the awaited flag value (0; a test sets it out of reach so that every
  // wait gives up).  Each give-up adds one to *wait_timeouts.
  int spin_limit;
  int wait_bias;
  uint32_t* wait_timeouts;
};

// Every launcher enqueues on `st` and returns the launch status.
hipError_t launch_bwd_delta(const BwdArgs& a, const Problem& p, hipStream_t st);
hipError_t launch_bwd_rec(const BwdArgs& a, const Problem& p, hipStream_t st);
// History dQ partials of the chunk's kv-heads; `grid` bounds the tile count.
hipError_t launch_bwd_dq_hist(const BwdArgs& a, const Problem& p, int64_t grid, hipStream_t st);
// Current-block dQ plus the history partials, written to dq.
hipError_t launch_bwd_dq_cur(const BwdArgs& a, const Problem& p, hipStream_t st);
// dK and dV of every key (all kv-heads).
hipError_t launch_bwd_dkdv(const BwdArgs& a, const Problem& p, hipStream_t st);

}  // namespace moba
