// Internal declarations of the decode path (one new query per sequence
// against its key/value cache), shared by the host library and the kernels.
#pragma once

#include "moba_internal.h"

namespace moba {

constexpr int kDecodeChunk = 256;     // keys per attention work-group
constexpr int kDecodeMaxGroup = 16;   // largest Hq / Hkv the decode kernels take
constexpr int kCombineShare = 64;    // partials one combine work-group folds
constexpr int kCombineMaxSplit = 64; // combine work-groups per row, at most

struct DecodeArgs {
  const __hip_bfloat16* q; int64_t q_ss, q_sh;  // [S, Hq, D]
  const __hip_bfloat16* k; int64_t k_st, k_sh;  // cache [T, Hkv, D]
  const __hip_bfloat16* v; int64_t v_st, v_sh;
  const float* kbar;     // [nblk_total, Hkv, D] block means of the cache (MoBA)
  const SeqInfo* seqs;   // per cached sequence
  int32_t* sel;          // [S, Hq, topk] selection (MoBA)
  float* part_o;         // [S * Hq, nchunk, D] normalised partials
  float* part_lse;       // [S * Hq, nchunk]
  __hip_bfloat16* out; int64_t o_ss, o_sh;  // [S, Hq, D]
  float* lse;            // [Hq, S]
  int nunion;            // MoBA: block slots per (sequence, kv-head): the most distinct
                         // blocks a group's query heads can select
  int nsub;              // chunks per block
  int nchunk;            // chunk slots per row
  int chunk_block;       // block length the chunks are cut at
  int nsplit;            // combine work-groups per row (1: no second pass)
  int split_len;         // partial slots per combine work-group
  float* mid;            // [S * Hq, nsplit, D + 2] per share: unnormalised o, max, weight sum
  int full;              // 1: causal full attention, 0: MoBA
  float scale_log2;
};

// Every launcher enqueues on `st` and returns the launch status.  p.S is the
// number of sequences (= queries), p.T the cache length.
hipError_t launch_decode_gate(const DecodeArgs& a, const Problem& p, hipStream_t st);
hipError_t launch_decode_attend(const DecodeArgs& a, const Problem& p, hipStream_t st);
// Two passes when nsplit > 1: shares of each row's partials, then the shares.
hipError_t launch_decode_combine(const DecodeArgs& a, const Problem& p, hipStream_t st);

}  // namespace moba
