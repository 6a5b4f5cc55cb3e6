// bf16 attention on the gfx950 matrix cores: the history-block attention,
// the causal current-block attention (Algorithm 1, the two
// flash_attention_varlen calls; Sec. 2.2 "Current Block Attention") and dense
// causal attention (Eq. 1), from one kernel template.
//
// Work-group = 8 waves = 256 query rows, one work-group per CU (two waves per
// SIMD); wave w owns rows 32w..32w+31, one query per lane column.  Sharing
// each K/V tile among 256 rows halves the LDS writes and DMA instructions per
// row compared with 128-row work-groups.
// Keys are consumed in tiles of 64.  LDS holds two K buffers and two V^T
// buffers, filled straight from global memory by global_load_lds_dwordx4 (no
// registers, no LDS store instructions).  Each such instruction writes 1 KiB
// contiguously (lane L to 16-byte chunk L).  Rows are padded by one chunk (K:
// 64 rows of 17 chunks, V^T: 128 rows of 9 chunks; the pad chunk receives a
// copy of the row's last chunk), so the DMA writes whole padded rows and an
// operand read, 16 lanes on 16 consecutive rows at one chunk, hits 16
// distinct bank groups (LDS serves a 16-byte-per-lane read to 16 lanes at a
// time across 64 banks of 4 bytes).  Every operand address is then a per-lane
// base plus a compile-time offset.
//
// Iteration i computes S(i) = K(i) . Q^T, its softmax and O += V(i) . P(i)
// while the DMA fills the other K and V^T buffers with tile i+1; one barrier
// per tile.
//
// Per key tile and wave, on v_mfma_f32_32x32x16_bf16:
//   S^T (keys x queries) = K . Q^T         2 halves x 8 k-steps
//   online softmax in fp32 on S^T: a lane holds one query and 32 of the
//   tile's 64 keys, so the row max needs one exchange with the partner lane
//   (lane ^ 32) and the row sum is kept per lane and combined at the end.
//   The weights are formed under the running max without taking the tile's
//   max first; only when some lane's sum of them exceeds 2^8 (so a weight
//   might) is the row max taken, the running max raised and the weights
//   formed again.  Weights stay at most 2^8 and the max and the rescale are
//   skipped on almost every tile.
//   O^T (dims x queries) += V^T . P^T      4 dim tiles x 4 k-steps, P^T
//   straight from the softmax registers (packed to bf16).
// The accumulator layout of a 32x32 MFMA gives lane l the column l % 32 and
// rows 8*(i/4) + 4*(l/32) + i%4 for its 16 values i; so the 8 keys a lane
// feeds into one k=16 step are keys {0-3, 8-11} (+4 for the upper half-wave)
// of a 16-key group, which is the order the V^T pack stores them in.
//
// Logits use scale 1/sqrt(D), folded with log2(e) into one FMA before exp2.
// Outputs: history tiles write normalised partials, rounded once to bf16 (the
// output dtype of the per-block attention calls of Algorithm 1), and their
// natural-log lse in fp32; current-block and dense tiles write the normalised
// result to the output and its lse (the merge kernel then folds the history
// partials into the current-block result).
#include "mfma_tile.h"

#include <math.h>

namespace moba {
namespace {

enum { kHist = 0, kCur = 1, kDense = 2 };

constexpr int kRows = kTileRowsMfma;               // query rows per work-group (256)
constexpr int kLdsChunks = 2 * kBufK + 2 * kBufV;  // 70 KiB: two K and two V^T buffers
constexpr float kSumLimit = 256.0f;  // largest per-lane weight sum kept without a rescale
constexpr int kPersistMaxBlock = 1024;  // blocks this short run on the persistent history kernel
constexpr float kLn2 = 0.69314718055994531f;

// Weights of S under the running max m as bf16 P^T operands pb[2*th + s2]
// (keys 32*th + 16*s2 .. +15); returns this lane's sum of them.
__device__ __forceinline__ float weights(const f32x16 (&s)[2], float m, bf16x8 (&pb)[4], float c2) {
  float ts = 0.0f;
#pragma unroll
  for (int th = 0; th < 2; th++)
#pragma unroll
    for (int s2 = 0; s2 < 2; s2++) {
      uint32_t w[4];
#pragma unroll
      for (int e = 0; e < 4; e++) {
        const float p0 = __builtin_amdgcn_exp2f(fmaf(s[th][8 * s2 + 2 * e], c2, -m));
        const float p1 = __builtin_amdgcn_exp2f(fmaf(s[th][8 * s2 + 2 * e + 1], c2, -m));
        w[e] = pack_bf16(p0, p1);
        ts += p0 + p1;
      }
      pb[2 * th + s2] = as_bf16x8(u32x4{w[0], w[1], w[2], w[3]});
    }
  return ts;
}

// Masking and online softmax of S(i); the weights leave as bf16 P^T operands.
// The weights are first formed under the running max; only if some lane's
// sum of them exceeds 2^8 (so possibly a weight above 2^8), or on the first
// tile, is the tile's row max taken, the accumulators rescaled and the
// weights formed again.  Weights therefore never exceed 2^8.
template <int MODE>
__device__ __forceinline__ void softmax(f32x16 (&s)[2], float& m, float& l, f32x16 (&o)[4],
                                        bf16x8 (&pb)[4], bool edge, int lo, int hi, float c2) {
  if (edge) mask_keys(s, lo, hi);
  float ts = 0.0f;
  bool redo = __builtin_amdgcn_ballot_w64(m == -INFINITY) != 0;
  if (!redo) {
    ts = weights(s, m, pb, c2);
    redo = __builtin_amdgcn_ballot_w64(!(ts <= kSumLimit)) != 0;
  }
  if (redo) {
    float mx = -INFINITY;
#pragma unroll
    for (int th = 0; th < 2; th++)
#pragma unroll
      for (int r = 0; r < 16; r++) mx = fmaxf(mx, s[th][r]);
    mx = fmaxf(mx, xor32(mx)) * c2;
    const float m_new = fmaxf(m, mx);
    const float alpha = m_new == -INFINITY ? 1.0f : __builtin_amdgcn_exp2f(m - m_new);
    l *= alpha;
#pragma unroll
    for (int dt = 0; dt < 4; dt++)
#pragma unroll
      for (int r = 0; r < 16; r++) o[dt][r] *= alpha;
    m = m_new;
    ts = weights(s, m == -INFINITY ? 0.0f : m, pb, c2);
  }
  l += ts;
}

// History epilogues stage the tile's normalised bf16 rows in LDS (rows of 17
// chunks, so the staging writes of 32 lanes on 32 rows spread over the
// banks) and then write each row as 16 lanes x 16 bytes, four whole rows per
// instruction: the scattered partial rows land in full 128-byte lines
// instead of 16-byte pieces spread over 16 instructions.
constexpr int kStageRow = kHeadDim / 8 + 1;  // 16-byte chunks per staged row

// Stages this lane's row (normalised, bf16) and its partial index; the
// caller then synchronizes and calls store_staged.
__device__ __forceinline__ void stage_row(const f32x16 (&o)[4], float inv, u32x4* stage,
                                          int64_t* sdst, int rloc, int hh, bool valid, int64_t dst) {
  uint2* srow = reinterpret_cast<uint2*>(stage + rloc * kStageRow);
#pragma unroll
  for (int dt = 0; dt < 4; dt++)
#pragma unroll
    for (int r4 = 0; r4 < 4; r4++) {
      uint2 w;
      w.x = pack_bf16(o[dt][4 * r4 + 0] * inv, o[dt][4 * r4 + 1] * inv);
      w.y = pack_bf16(o[dt][4 * r4 + 2] * inv, o[dt][4 * r4 + 3] * inv);
      srow[(32 * dt + 8 * r4 + 4 * hh) >> 2] = w;
    }
  if (hh == 0) sdst[rloc] = valid ? dst : -1;
}

// Wave w writes staged rows 32w .. 32w + 31, four per instruction.
__device__ __forceinline__ void store_staged(const AttnArgs& a, const u32x4* stage,
                                             const int64_t* sdst, int wave, int lane) {
  const int rsub = lane >> 4, ch = lane & 15;
#pragma unroll
  for (int j = 0; j < 8; j++) {
    const int rr = 32 * wave + 4 * j + rsub;
    const int64_t d = sdst[rr];
    if (d >= 0)
      reinterpret_cast<u32x4*>(static_cast<__hip_bfloat16*>(a.o_part) + d * kHeadDim)[ch] =
          stage[rr * kStageRow + ch];
  }
}

// The same for the output rows of current-block and dense tiles: staged
// destinations are element offsets into out.
__device__ __forceinline__ void store_staged_out(const AttnArgs& a, const u32x4* stage,
                                                 const int64_t* sdst, int wave, int lane) {
  const int rsub = lane >> 4, ch = lane & 15;
#pragma unroll
  for (int j = 0; j < 8; j++) {
    const int rr = 32 * wave + 4 * j + rsub;
    const int64_t d = sdst[rr];
    if (d >= 0)
      reinterpret_cast<u32x4*>(static_cast<__hip_bfloat16*>(a.out) + d)[ch] =
          stage[rr * kStageRow + ch];
  }
}

template <int MODE>
__global__ __launch_bounds__(512, 1) void attn_mfma_kernel(AttnArgs a, Problem p) {
  __shared__ u32x4 lds[kLdsChunks];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int qc = lane & 31, hh = lane >> 5;

  // ------------------------------------------------------------ tile setup
  int g, s;
  int64_t kbeg, kend, tmin;
  RowInfo ri;
  const int rloc = wave * 32 + qc;  // this lane's query row within the tile
  if constexpr (MODE == kHist) {
    const int64_t nb = p.nblk_total;
    const int64_t tbeg = a.bin_tile_start[a.g0 * nb];
    const int64_t tend = a.bin_tile_start[a.g1 * nb];
    // XCD-aware order: work-groups go round-robin to the 8 XCDs, so give each
    // XCD a contiguous run of tiles (tiles of one bin share its K/V block).
    // The grid is a multiple of 8, so this map is a bijection of [0, grid).
    const int64_t per = gridDim.x / 8;
    const int64_t tile = tbeg + (int64_t)(blockIdx.x % 8) * per + blockIdx.x / 8;
    if (tile >= tend) return;
    const int64_t bin = a.tile_bin[tile];
    g = (int)(bin / nb);
    const int b = (int)(bin % nb);
    const int64_t e0 = a.bin_start[bin] + (tile - a.bin_tile_start[bin]) * kRows;
    const int n = (int)min((int64_t)kRows, a.bin_start[bin] + a.bin_count[bin] - e0);
    s = find_seq(a.seqs, p.S, b, [](const SeqInfo& x) { return x.blk_off; });
    const SeqInfo sq = a.seqs[s];
    kbeg = (int64_t)sq.tok_start + (int64_t)(b - sq.blk_off) * p.B;
    kend = kbeg + p.B;
    tmin = kend;  // every key precedes every routed query
    const uint64_t kh = (uint64_t)(p.topk - 1);
    const uint64_t TG = (uint64_t)p.T * p.G;
    const uint64_t ev = a.entries[e0 + min(rloc, n - 1)];
    const uint64_t rem = ev / kh - (uint64_t)g * TG;
    const bool ok = rem < TG;
    ri.valid = rloc < n && ok;
    ri.t = ok ? (int64_t)(rem / p.G) : kbeg;
    ri.h = g * p.G + (ok ? (int)(rem % p.G) : 0);
    ri.dst = (int64_t)(ev - (uint64_t)a.g0 * TG * kh);
  } else {
    const CausalTile ct = a.tiles[blockIdx.x];
    if (ct.t1 <= ct.t0) return;  // padding of the tile list
    g = a.g0 + blockIdx.y;
    s = ct.s;
    kbeg = ct.kbeg;
    kend = ct.t1;
    tmin = ct.t0;
    const int nrow = (ct.t1 - ct.t0) * p.G;
    ri.valid = rloc < nrow;
    const int rr = ri.valid ? rloc : 0;
    ri.t = ct.t0 + rr / p.G;
    ri.h = g * p.G + rr % p.G;
    ri.dst = (int64_t)(g - a.g0) * p.T * p.G + ri.t * p.G + (rr % p.G);
  }
  // the tile's key range is wave-uniform: keep it in scalar registers
  g = __builtin_amdgcn_readfirstlane(g);
  s = __builtin_amdgcn_readfirstlane(s);
  kbeg = uniform64(kbeg);
  kend = uniform64(kend);
  tmin = uniform64(tmin);
  const SeqInfo sq = a.seqs[s];
  const int64_t tok0 = sq.tok_start;

  // ---------------------------------------------------------- Q^T operands
  bf16x8 qf[8];
  {
    const __hip_bfloat16* qrow = static_cast<const __hip_bfloat16*>(a.q) + ri.t * a.q_st +
                                 (int64_t)ri.h * a.q_sh + 8 * hh;
#pragma unroll
    for (int kk = 0; kk < 8; kk++)
      qf[kk] = as_bf16x8(*reinterpret_cast<const u32x4*>(qrow + 16 * kk));
  }

  // ------------------------------------------------------------ key tiles
  const int64_t rb = kbeg - tok0, re = kend - tok0;
  const int i0 = (int)(rb / kKeyTile), i1 = (int)((re + kKeyTile - 1) / kKeyTile);
  Dma D;
  {
    const int wv = __builtin_amdgcn_readfirstlane(wave);
    D.wave = wv;
    const int64_t kst = a.k_st * 2;  // bytes
    D.kbase = reinterpret_cast<const char*>(static_cast<const __hip_bfloat16*>(a.k) +
                                            (int64_t)g * a.k_sh) + tok0 * kst;
    D.k_tile = kKeyTile * kst;
    D.len = sq.len;
    D.klast = D.kbase + (sq.len - 1) * kst;
#pragma unroll
    for (int x = 0; x < 3; x++) {
      const int pk = 64 * (wv + 8 * x) + lane;
      const int row = min(pk / kRowK, kKeyTile - 1), c = min(pk % kRowK, kRowK - 2);
      D.krow[x] = row;
      D.kcol[x] = (uint32_t)(c * 16);
      D.koff[x] = (uint32_t)(row * kst) + D.kcol[x];
      const int pv_ = 64 * (wv + 8 * x) + lane;
      const int vrow = min(pv_ / kRowV, kHeadDim - 1), vc = min(pv_ % kRowV, kRowV - 2);
      D.voff[x] = (uint32_t)(vrow * (kKeyTile * 2) + vc * 16);
    }
    D.vbase = reinterpret_cast<const char*>(
        a.vt + ((int64_t)g * p.vt_tiles + sq.vt_tile_off) * (kKeyTile * kHeadDim));
  }
  ReadOff ro;
  ro.kq = qc * kRowK + hh;
  ro.vq = qc * kRowV + hh;
  const float c2 = a.scale_log2;
  f32x16 o[4];
  float m = -INFINITY, l = 0.0f;
#pragma unroll
  for (int dt = 0; dt < 4; dt++)
#pragma unroll
    for (int r = 0; r < 16; r++) o[dt][r] = 0.0f;

  // tile i lives in K and V^T buffers (i - i0) % 2
  dma_k(D, i0, lds);
  dma_v(D, i0, lds + 2 * kBufK);
  // Every prologue load (Q included) lands here, so the loop carries no
  // waits on Q.
  dma_wait();
  __syncthreads();

  f32x16 sc[2];
  bf16x8 pb[4];
  for (int i = i0; i < i1; i++) {
    const int cur = (i - i0) & 1;
    if (i + 1 < i1) {
      dma_k(D, i + 1, lds + (cur ^ 1) * kBufK);
      dma_v(D, i + 1, lds + 2 * kBufK + (cur ^ 1) * kBufV);
    }
    qk(sc, lds + cur * kBufK, ro, qf);
    const int64_t u0 = tok0 + (int64_t)i * kKeyTile;
    const bool edge =
        u0 < kbeg || u0 + kKeyTile > kend || (MODE != kHist && u0 + kKeyTile - 1 > tmin);
    int lo = 0, hi = kKeyTile;
    if (edge) {
      lo = (int)max((int64_t)0, kbeg - u0) - 4 * hh;
      const int64_t lim = min((int64_t)kKeyTile, kend - u0);
      hi = (int)(MODE == kHist ? lim : min(lim, ri.t + 1 - u0)) - 4 * hh;
    }
    softmax<MODE>(sc, m, l, o, pb, edge, lo, hi, c2);
    pv(o, lds + 2 * kBufK + cur * kBufV, ro, pb);
    dma_wait();
    __syncthreads();
  }

  // -------------------------------------------------------------- epilogue
  {
    const float l_tot = l + xor32(l);
    const float inv = 1.0f / l_tot;
    const float lse = (m + __builtin_amdgcn_logf(l_tot)) * kLn2;
    f32x16 (&og)[4] = o;
    const RowInfo& r = ri;
    if constexpr (MODE == kHist) {
      // the K/V buffers are free after the last barrier: stage the rows there
      u32x4* stage = lds;
      int64_t* sdst = reinterpret_cast<int64_t*>(lds + kRows * kStageRow);
      stage_row(og, inv, stage, sdst, rloc, hh, r.valid, r.dst);
      if (r.valid && hh == 0) a.lse_part[r.dst] = lse;
      __syncthreads();
      store_staged(a, stage, sdst, wave, lane);
    } else {
      // the output rows leave the same way, as whole rows
      u32x4* stage = lds;
      int64_t* sdst = reinterpret_cast<int64_t*>(lds + kRows * kStageRow);
      stage_row(og, inv, stage, sdst, rloc, hh, r.valid, r.t * a.o_st + (int64_t)r.h * a.o_sh);
      if (r.valid && hh == 0) a.lse[(int64_t)r.h * p.T + r.t] = lse;
      __syncthreads();
      store_staged_out(a, stage, sdst, wave, lane);
    }
  }
}

// ----------------------------------------------------------------------
// History tiles of short blocks, persistent: one work-group per CU walks a
// run of tiles.  With few key tiles per history tile (B / 64), the per-tile
// cost outside the key loop (work-group start, routed query rows, first K/V
// tile, epilogue) would dominate; here the next tile's query rows and first
// K/V tile are fetched during the current tile's last key tile.
struct HistCtx {
  int g, s;
  int64_t kbeg, kend, tok0;
  int i0, i1;
  RowInfo ri;
};

__device__ __forceinline__ bool hist_setup(const AttnArgs& a, const Problem& p, int64_t tile,
                                           int64_t tlim, int rloc, HistCtx& c) {
  if (tile >= tlim) return false;
  const int64_t nb = p.nblk_total;
  const int64_t bin = a.tile_bin[tile];
  const int g = (int)(bin / nb);
  const int b = (int)(bin % nb);
  const int64_t e0 = a.bin_start[bin] + (tile - a.bin_tile_start[bin]) * kRows;
  const int n = (int)min((int64_t)kRows, a.bin_start[bin] + a.bin_count[bin] - e0);
  const int s = find_seq(a.seqs, p.S, b, [](const SeqInfo& x) { return x.blk_off; });
  const SeqInfo sq = a.seqs[s];
  const int64_t kbeg = (int64_t)sq.tok_start + (int64_t)(b - sq.blk_off) * p.B;
  const uint64_t kh = (uint64_t)(p.topk - 1);
  const uint64_t TG = (uint64_t)p.T * p.G;
  const uint64_t ev = a.entries[e0 + min(rloc, n - 1)];
  const uint64_t rem = ev / kh - (uint64_t)g * TG;
  const bool ok = rem < TG;
  c.ri.valid = rloc < n && ok;
  c.ri.t = ok ? (int64_t)(rem / p.G) : kbeg;
  c.ri.h = g * p.G + (ok ? (int)(rem % p.G) : 0);
  c.ri.dst = (int64_t)(ev - (uint64_t)a.g0 * TG * kh);
  c.g = __builtin_amdgcn_readfirstlane(g);
  c.s = __builtin_amdgcn_readfirstlane(s);
  c.kbeg = uniform64(kbeg);
  c.kend = uniform64(kbeg + p.B);
  c.tok0 = uniform64(sq.tok_start);
  c.i0 = (int)((c.kbeg - c.tok0) / kKeyTile);
  c.i1 = (int)((c.kend - c.tok0 + kKeyTile - 1) / kKeyTile);
  return true;
}

// The tile-dependent (wave-uniform) part of the DMA sources.
__device__ __forceinline__ void dma_tile(Dma& D, const AttnArgs& a, const Problem& p,
                                         const HistCtx& c) {
  const SeqInfo sq = a.seqs[c.s];
  const int64_t kst = a.k_st * 2;
  D.kbase = reinterpret_cast<const char*>(static_cast<const __hip_bfloat16*>(a.k) +
                                          (int64_t)c.g * a.k_sh) + c.tok0 * kst;
  D.len = sq.len;
  D.klast = D.kbase + (sq.len - 1) * kst;
  D.vbase = reinterpret_cast<const char*>(
      a.vt + ((int64_t)c.g * p.vt_tiles + sq.vt_tile_off) * (kKeyTile * kHeadDim));
}

__device__ __forceinline__ void load_q(bf16x8 (&qf)[8], const AttnArgs& a, const RowInfo& ri,
                                       int hh) {
  const __hip_bfloat16* qrow = static_cast<const __hip_bfloat16*>(a.q) + ri.t * a.q_st +
                               (int64_t)ri.h * a.q_sh + 8 * hh;
#pragma unroll
  for (int kk = 0; kk < 8; kk++)
    qf[kk] = as_bf16x8(*reinterpret_cast<const u32x4*>(qrow + 16 * kk));
}

__global__ __launch_bounds__(512, 1) void attn_hist_persist_kernel(AttnArgs a, Problem p) {
  __shared__ u32x4 lds[kLdsChunks];
  __shared__ u32x4 stage[kRows * kStageRow];  // the tile's partial rows (bf16)
  __shared__ int64_t sdst[kRows];             // their partial indices (-1: no row)
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int qc = lane & 31, hh = lane >> 5;
  const int rloc = wave * 32 + qc;

  // XCD-aware walk: work-groups go round-robin to the 8 XCDs; XCD x owns
  // the contiguous run [x*per, (x+1)*per) of the tiles (tiles of one bin share
  // its K/V block), and its work-groups take every nx-th tile of it.  Every
  // work-group leaves the loop once its next tile is past the run.
  const int64_t nb = p.nblk_total;
  const int64_t tbeg = a.bin_tile_start[a.g0 * nb];
  const int64_t tend = a.bin_tile_start[a.g1 * nb];
  const int64_t nx = gridDim.x / 8;
  const int64_t per = (tend - tbeg + 7) / 8;
  const int64_t xs = tbeg + (int64_t)(blockIdx.x % 8) * per;
  const int64_t tlim = min(tend, xs + per);
  int64_t tile = xs + blockIdx.x / 8;

  HistCtx c;
  if (!hist_setup(a, p, tile, tlim, rloc, c)) return;
  bf16x8 qf[8];
  load_q(qf, a, c.ri, hh);
  Dma D;
  {
    const int wv = __builtin_amdgcn_readfirstlane(wave);
    D.wave = wv;
    const int64_t kst = a.k_st * 2;
    D.k_tile = kKeyTile * kst;
#pragma unroll
    for (int x = 0; x < 3; x++) {
      const int pk = 64 * (wv + 8 * x) + lane;
      const int row = min(pk / kRowK, kKeyTile - 1), col = min(pk % kRowK, kRowK - 2);
      D.krow[x] = row;
      D.kcol[x] = (uint32_t)(col * 16);
      D.koff[x] = (uint32_t)(row * kst) + D.kcol[x];
      const int vrow = min(pk / kRowV, kHeadDim - 1), vc = min(pk % kRowV, kRowV - 2);
      D.voff[x] = (uint32_t)(vrow * (kKeyTile * 2) + vc * 16);
    }
  }
  dma_tile(D, a, p, c);
  ReadOff ro;
  ro.kq = qc * kRowK + hh;
  ro.vq = qc * kRowV + hh;
  const float c2 = a.scale_log2;

  dma_k(D, c.i0, lds);
  dma_v(D, c.i0, lds + 2 * kBufK);
  dma_wait();
  __syncthreads();

  int par = 0;  // buffer holding the current key tile
  for (;;) {
    HistCtx n;
    const bool more = hist_setup(a, p, tile + nx, tlim, rloc, n);
    Dma Dn = D;
    if (more) dma_tile(Dn, a, p, n);
    f32x16 o[4];
    float m = -INFINITY, l = 0.0f;
#pragma unroll
    for (int dt = 0; dt < 4; dt++)
#pragma unroll
      for (int r = 0; r < 16; r++) o[dt][r] = 0.0f;
    f32x16 sc[2];
    bf16x8 pb[4];
    for (int i = c.i0; i < c.i1; i++) {
      const int cur = par;
      par ^= 1;
      const bool last = i + 1 == c.i1;
      if (!last) {
        dma_k(D, i + 1, lds + (cur ^ 1) * kBufK);
        dma_v(D, i + 1, lds + 2 * kBufK + (cur ^ 1) * kBufV);
      } else if (more) {
        dma_k(Dn, n.i0, lds + (cur ^ 1) * kBufK);
        dma_v(Dn, n.i0, lds + 2 * kBufK + (cur ^ 1) * kBufV);
      }
      qk(sc, lds + cur * kBufK, ro, qf);
      if (last && more) load_q(qf, a, n.ri, hh);  // this tile's products are issued
      const int64_t u0 = c.tok0 + (int64_t)i * kKeyTile;
      const bool edge = u0 < c.kbeg || u0 + kKeyTile > c.kend;
      int lo = 0, hi = kKeyTile;
      if (edge) {
        lo = (int)max((int64_t)0, c.kbeg - u0) - 4 * hh;
        hi = (int)min((int64_t)kKeyTile, c.kend - u0) - 4 * hh;
      }
      softmax<kHist>(sc, m, l, o, pb, edge, lo, hi, c2);
      pv(o, lds + 2 * kBufK + cur * kBufV, ro, pb);
      dma_wait();
      __syncthreads();
    }
    // epilogue: the normalised partial (bf16) and its lse
    const float l_tot = l + xor32(l);  // every lane takes part in the exchange
    stage_row(o, 1.0f / l_tot, stage, sdst, rloc, hh, c.ri.valid, c.ri.dst);
    if (c.ri.valid && hh == 0) a.lse_part[c.ri.dst] = (m + __builtin_amdgcn_logf(l_tot)) * kLn2;
    __syncthreads();
    store_staged(a, stage, sdst, wave, lane);
    // the staging area is rewritten only after the next tile's key loop,
    // whose barriers order these reads before those writes
    if (!more) break;
    c = n;
    D = Dn;
    tile += nx;
  }
}

}  // namespace

hipError_t launch_attn_hist_bf16(const AttnArgs& a, const Problem& p, int64_t grid, hipStream_t st) {
  if (grid <= 0) return hipSuccess;
  if (p.B <= kPersistMaxBlock) {
    // short blocks: one work-group per CU (a multiple of 8), walking the tiles
    static int ncu = 0;
    if (!ncu) {
      int dev = 0;
      if (hipGetDevice(&dev) != hipSuccess ||
          hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return hipErrorInvalidDevice;
    }
    int64_t g = ncu / 8 * 8;
    if (g < 8) g = 8;
    if (g > (grid + 7) / 8 * 8) g = (grid + 7) / 8 * 8;
    attn_hist_persist_kernel<<<(unsigned)g, 512, 0, st>>>(a, p);
    return hipGetLastError();
  }
  grid = (grid + 7) / 8 * 8;
  attn_mfma_kernel<kHist><<<(unsigned)grid, 512, 0, st>>>(a, p);
  return hipGetLastError();
}

hipError_t launch_attn_causal_bf16(bool dense, const AttnArgs& a, const Problem& p, hipStream_t st) {
  if (a.ntiles <= 0 || a.g1 <= a.g0) return hipSuccess;
  dim3 grid((unsigned)a.ntiles, a.g1 - a.g0);
  if (dense) attn_mfma_kernel<kDense><<<grid, 512, 0, st>>>(a, p);
  else attn_mfma_kernel<kCur><<<grid, 512, 0, st>>>(a, p);
  return hipGetLastError();
}

}  // namespace moba
