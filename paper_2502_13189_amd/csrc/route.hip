// Routing inversion: from each query's selected history blocks to, for each
// (kv-head, block) bin, the ordered list of queries that chose it.  This is
// the "arrange the ordering of query tokens based on their assigned KV
// blocks" step of Sec. 2.3 (Algorithm 1, index_select_moba_attn_block),
// done as a stable counting sort with integer arithmetic only, so the result
// is deterministic.
//
// Rows of kv-head g are ordered r = g*T*G + t*G + hl (hl = query head within
// the GQA group).  Rows are cut into chunks of `route_rt` tokens x G heads
// (at most kRouteRows rows) within one sequence.  Per sequence and kv-head
// the histogram holds one column per block over the sequence's chunks.
// Five kernels:
//   count      per chunk: the chunk's selections, read once and coalesced
//              (each token's G * topk entries are contiguous), counted per
//              block in LDS and written to the blocks' columns;
//   scan_cols  one wave per bin: exclusive prefix over its column (in
//              place), and the bin total;
//   scan_bins  one work-group: exclusive scans of bin totals (entry offsets)
//              and of ceil(total / tile_rows) (attention tile offsets);
//   tile_bins  one wave per bin: the bin of each of its attention tiles;
//   scatter    per chunk, one thread per row: every row ORs its bit into an
//              LDS bitmask per selected block; a row's rank among the chunk's
//              rows that chose the same block is the popcount of the lower
//              bits, which keeps the order of rows (a stable sort).  The
//              chunk's entries are gathered in LDS, grouped by block, and
//              each block's run is then written out contiguously.  When that
//              does not fit in LDS, rounds of 256 rows write their entries
//              one by one.
// Entry value: r * (topk - 1) + slot, where slot is the position of the block
// in the row's ascending selection.  A history slot holding no past block of
// its row (outside [0, c), which the gate never writes) is skipped by the
// count and the scatter alike, so every LDS and global index stays within the
// row's sequence.
#include "moba_internal.h"

namespace moba {
namespace {

constexpr size_t kRouteLdsMax = 160 * 1024;  // LDS of one gfx950 work-group

struct ChunkPos {
  int s;
  int r;      // chunk index within the sequence
  int tl0;    // first local token
  int ntok;   // tokens in the chunk
};

__device__ __forceinline__ ChunkPos chunk_pos(const SeqInfo* seqs, const Problem& p, int idx) {
  ChunkPos c;
  c.s = find_seq(seqs, p.S, idx, [](const SeqInfo& x) { return x.rc_off; });
  c.r = idx - seqs[c.s].rc_off;
  c.tl0 = c.r * p.route_rt;
  c.ntok = min(p.route_rt, seqs[c.s].len - c.tl0);
  return c;
}

// Column of block j of sequence sq (kv-head g) in the histogram.
__device__ __forceinline__ int32_t* hist_col(int32_t* hist, const Problem& p, int g,
                                             const SeqInfo& sq, int j) {
  const int nchunks = (sq.len + p.route_rt - 1) / p.route_rt;
  return hist + (int64_t)g * p.hist_words + sq.hist_off + (int64_t)j * nchunks;
}

__global__ __launch_bounds__(256) void route_count_kernel(const int32_t* __restrict__ sel,
                                                          const SeqInfo* __restrict__ seqs,
                                                          Problem p, int32_t* __restrict__ hist) {
  extern __shared__ int32_t cnt[];
  const int g = blockIdx.y;
  const ChunkPos cp = chunk_pos(seqs, p, blockIdx.x);
  const SeqInfo sq = seqs[cp.s];
  const int kh = p.topk - 1;
  for (int j = threadIdx.x; j < sq.nblk; j += 256) cnt[j] = 0;
  __syncthreads();
  // element e of the chunk: token cp.tl0 + e / (G topk), entry e % (G topk)
  // of the token's group of rows (head hl = entry / topk, slot x = entry % topk)
  const int per_tok = p.G * p.topk;
  const int32_t* base = sel + ((int64_t)(sq.tok_start + cp.tl0) * p.sel_st + (int64_t)g * p.sel_sg) * p.topk;
  const int64_t tok_stride = p.sel_st * p.topk;
  if (per_tok <= 256) {
    // thread -> entry w of token tk0 + k * tpb: the divisions once per thread
    const int tpb = 256 / per_tok;
    const int tk0 = threadIdx.x / per_tok, w = threadIdx.x - tk0 * per_tok;
    const int x = w % p.topk;
    if (tk0 < tpb) {
      for (int tk = tk0; tk < cp.ntok; tk += tpb) {
        const int c = (cp.tl0 + tk) / p.B;
        if (x < min(kh, c)) {
          const int j = base[tk * tok_stride + w];
          if ((unsigned)j < (unsigned)c) atomicAdd(&cnt[j], 1);
        }
      }
    }
  } else {
    const int n = cp.ntok * per_tok;  // at most kRouteRows * topk
    for (int e = threadIdx.x; e < n; e += 256) {
      const int tk = e / per_tok, w = e - tk * per_tok;
      const int x = w % p.topk;
      const int c = (cp.tl0 + tk) / p.B;
      if (x < min(kh, c)) {
        const int j = base[tk * tok_stride + w];
        if ((unsigned)j < (unsigned)c) atomicAdd(&cnt[j], 1);
      }
    }
  }
  __syncthreads();
  const int nchunks = (sq.len + p.route_rt - 1) / p.route_rt;
  int32_t* col0 = hist + (int64_t)g * p.hist_words + sq.hist_off + cp.r;
  for (int j = threadIdx.x; j < sq.nblk; j += 256) col0[(int64_t)j * nchunks] = cnt[j];
}

// One wave per bin: exclusive scan of the bin's column, and its total.
__global__ __launch_bounds__(256) void route_scan_cols_kernel(const SeqInfo* __restrict__ seqs,
                                                              Problem p, int32_t* __restrict__ hist,
                                                              int32_t* __restrict__ bin_count) {
  const int lane = threadIdx.x & 63;
  const int64_t bin = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int64_t nbins = (int64_t)p.Hkv * p.nblk_total;
  if (bin >= nbins) return;
  const int g = (int)(bin / p.nblk_total);
  const int b = (int)(bin % p.nblk_total);
  const int s = find_seq(seqs, p.S, b, [](const SeqInfo& x) { return x.blk_off; });
  const SeqInfo sq = seqs[s];
  const int nchunks = (sq.len + p.route_rt - 1) / p.route_rt;
  int32_t* col = hist_col(hist, p, g, sq, b - sq.blk_off);
  int32_t run = 0;
  for (int r0 = 0; r0 < nchunks; r0 += 64) {
    const int r = r0 + lane;
    const int32_t v = r < nchunks ? col[r] : 0;
    int32_t inc = v;  // inclusive prefix over the 64 lanes
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int32_t o = __shfl_up(inc, d, 64);
      if (lane >= d) inc += o;
    }
    if (r < nchunks) col[r] = run + inc - v;
    run += __shfl(inc, 63, 64);
  }
  if (lane == 0) bin_count[bin] = run;
}

__global__ __launch_bounds__(1024) void route_scan_bins_kernel(const int32_t* __restrict__ bin_count,
                                                               int64_t nbins, int tile_rows,
                                                               int64_t* __restrict__ bin_start,
                                                               int32_t* __restrict__ bin_tile_start) {
  __shared__ int64_t se[1024];
  __shared__ int64_t stl[1024];
  const int tid = threadIdx.x;
  const int64_t per = (nbins + 1023) / 1024;
  const int64_t b0 = min(nbins, tid * per), b1 = min(nbins, b0 + per);
  int64_t e = 0, tl = 0;
  for (int64_t b = b0; b < b1; b++) {
    e += bin_count[b];
    tl += (bin_count[b] + tile_rows - 1) / tile_rows;
  }
  se[tid] = e;
  stl[tid] = tl;
  __syncthreads();
  // Hillis-Steele inclusive scan over the 1024 per-thread sums
  for (int off = 1; off < 1024; off <<= 1) {
    const int64_t a = tid >= off ? se[tid - off] : 0;
    const int64_t c = tid >= off ? stl[tid - off] : 0;
    __syncthreads();
    se[tid] += a;
    stl[tid] += c;
    __syncthreads();
  }
  int64_t eo = se[tid] - e, to = stl[tid] - tl;
  for (int64_t b = b0; b < b1; b++) {
    bin_start[b] = eo;
    bin_tile_start[b] = (int32_t)to;
    eo += bin_count[b];
    to += (bin_count[b] + tile_rows - 1) / tile_rows;
  }
  if (tid == 1023) {
    bin_start[nbins] = se[1023];
    bin_tile_start[nbins] = (int32_t)stl[1023];
  }
}

// One wave per bin: the bin index of each of its attention tiles.
__global__ __launch_bounds__(256) void route_tile_bins_kernel(const int32_t* __restrict__ bin_tile_start,
                                                              int64_t nbins,
                                                              int32_t* __restrict__ tile_bin) {
  const int64_t bin = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (bin >= nbins) return;
  const int32_t t1 = bin_tile_start[bin + 1];
  for (int32_t t = bin_tile_start[bin] + (threadIdx.x & 63); t < t1; t += 64) tile_bin[t] = (int32_t)bin;
}

// Entries written one by one (chunks whose entries do not fit in LDS).
__global__ __launch_bounds__(256) void route_scatter_kernel(const int32_t* __restrict__ sel,
                                                            const SeqInfo* __restrict__ seqs,
                                                            Problem p,
                                                            const int32_t* __restrict__ hist,
                                                            const int64_t* __restrict__ bin_start,
                                                            uint32_t* __restrict__ entries,
                                                            bool use_pre) {
  extern __shared__ uint32_t lds[];
  const int g = blockIdx.y;
  const ChunkPos cp = chunk_pos(seqs, p, blockIdx.x);
  const SeqInfo sq = seqs[cp.s];
  const int nb = sq.nblk;
  uint32_t* mask = lds;            // [8][nb], word-major
  uint32_t* running = lds + 8 * nb;  // [nb]
  // with use_pre: [8][nb] bytes, the set bits of each block's words below a word
  uint8_t* pre = reinterpret_cast<uint8_t*>(lds + 9 * nb);
  const int kh = p.topk - 1;
  const int tid = threadIdx.x, word = tid >> 5, bit = tid & 31;
  const int nchunks = (sq.len + p.route_rt - 1) / p.route_rt;
  const int32_t* chunk_off = hist + (int64_t)g * p.hist_words + sq.hist_off + cp.r;
  const int64_t* bstart = bin_start + (int64_t)g * p.nblk_total + sq.blk_off;
  const uint64_t TG = (uint64_t)p.T * p.G;
  for (int j = tid; j < nb; j += 256) running[j] = 0;
  const int nrow = cp.ntok * p.G;
  for (int base = 0; base < nrow; base += 256) {
    for (int x = tid; x < 8 * nb; x += 256) mask[x] = 0;
    __syncthreads();
    const int i = base + tid;
    const bool valid = i < nrow;
    int tl = 0, hl = 0, nh = 0;
    int64_t row = 0;
    if (valid) {
      tl = cp.tl0 + i / p.G;
      hl = i % p.G;
      nh = min(kh, tl / p.B);
      row = ((int64_t)sq.tok_start + tl) * p.sel_st + (int64_t)g * p.sel_sg + hl;
      for (int x = 0; x < nh; x++) {
        const int j = sel[row * p.topk + x];
        if ((unsigned)j < (unsigned)(tl / p.B)) atomicOr(&mask[word * nb + j], 1u << bit);
      }
    }
    __syncthreads();
    if (use_pre) {
      for (int j = tid; j < nb; j += 256) {
        uint32_t acc = 0;  // at most 7 * 32
#pragma unroll
        for (int w = 0; w < 8; w++) {
          pre[w * nb + j] = (uint8_t)acc;
          acc += __popc(mask[w * nb + j]);
        }
      }
      __syncthreads();
    }
    if (valid) {
      const uint64_t r = (uint64_t)g * TG + (uint64_t)(sq.tok_start + tl) * p.G + hl;
      for (int x = 0; x < nh; x++) {
        const int j = sel[row * p.topk + x];
        if ((unsigned)j >= (unsigned)(tl / p.B)) continue;
        uint32_t rank = running[j] + __popc(mask[word * nb + j] & ((1u << bit) - 1u));
        if (use_pre) {
          rank += pre[word * nb + j];
        } else {
          for (int w = 0; w < word; w++) rank += __popc(mask[w * nb + j]);
        }
        const int64_t pos = bstart[j] + chunk_off[(int64_t)j * nchunks] + rank;
        entries[pos] = (uint32_t)(r * (uint64_t)kh + (uint64_t)x);
      }
    }
    __syncthreads();
    for (int j = tid; j < nb; j += 256) {
      uint32_t c = 0;
#pragma unroll
      for (int w = 0; w < 8; w++) c += __popc(mask[w * nb + j]);
      running[j] += c;
    }
    __syncthreads();
  }
}

// LDS of the staged scatter for nb blocks and kh selections per row: masks
// [32][nb] words (one bit per row of the chunk), their prefix counts [32][nb]
// (u16), per-block segment start and chunk count [nb] each, and the chunk's
// entries [kRouteRows * kh] as u16 codes (row within the chunk << 5 | slot;
// the staged path takes kh <= 31): at top-12 two work-groups fit on a CU up
// to ~290 blocks per sequence, one up to ~700.
__host__ __device__ inline size_t staged_lds_bytes(int nb, int kh) {
  return (size_t)nb * (128 + 64 + 8) + (size_t)kRouteRows * kh * 2;
}

// KH: largest number of history selections per row (register array).
template <int KH>
__global__ __launch_bounds__(kRouteRows) void route_scatter_staged_kernel(
    const int32_t* __restrict__ sel, const SeqInfo* __restrict__ seqs, Problem p,
    const int32_t* __restrict__ hist, const int32_t* __restrict__ bin_count,
    const int64_t* __restrict__ bin_start, uint32_t* __restrict__ entries) {
  extern __shared__ uint32_t lds[];
  constexpr int kWords = kRouteRows / 32;
  const int g = blockIdx.y;
  const ChunkPos cp = chunk_pos(seqs, p, blockIdx.x);
  const SeqInfo sq = seqs[cp.s];
  const int nb = sq.nblk;
  const int kh = p.topk - 1;
  uint32_t* mask = lds;                                  // [32][nb] (word-major: no bank
                                                         // conflicts among a word's lanes)
  uint32_t* seg = mask + kWords * nb;                    // [nb] segment start of block j in ent
  uint32_t* ccnt = seg + nb;                             // [nb] entries of block j in this chunk
  uint16_t* ent = reinterpret_cast<uint16_t*>(ccnt + nb);  // [rows * kh] codes
  uint16_t* pre = ent + kRouteRows * kh;                    // [32][nb]
  const int tid = threadIdx.x, word = tid >> 5, bit = tid & 31;
  const int lane = tid & 63, wave = tid >> 6;
  const int nchunks = (sq.len + p.route_rt - 1) / p.route_rt;
  const int32_t* col0 = hist + (int64_t)g * p.hist_words + sq.hist_off;
  const int64_t bin0 = (int64_t)g * p.nblk_total + sq.blk_off;

  for (int j = tid; j < nb; j += kRouteRows) {
    const int32_t* col = col0 + (int64_t)j * nchunks;
    const int32_t a = col[cp.r];
    const int32_t b = cp.r + 1 < nchunks ? col[cp.r + 1] : bin_count[bin0 + j];
    ccnt[j] = (uint32_t)(b - a);
  }
  for (int x = tid; x < kWords * nb; x += kRouteRows) mask[x] = 0;
  // this thread's row and its selections
  const int nrow = cp.ntok * p.G;
  const bool valid = tid < nrow;
  const int tl = cp.tl0 + tid / p.G, hl = tid % p.G;
  const int nh = valid ? min(kh, tl / p.B) : 0;
  // slots with a block outside [0, c) are skipped (-1), as by the count kernel
  int js[KH];
  const int32_t* mine =
      sel + ((int64_t)(sq.tok_start + tl) * p.sel_st + (int64_t)g * p.sel_sg + hl) * p.topk;
#pragma unroll
  for (int x = 0; x < KH; x++) {
    const int j = x < nh ? mine[x] : -1;
    js[x] = (unsigned)j < (unsigned)(tl / p.B) ? j : -1;
  }
  __syncthreads();
  // segment starts: exclusive scan of ccnt (wave 0, 64 blocks per step)
  if (wave == 0) {
    uint32_t run = 0;
    for (int j0 = 0; j0 < nb; j0 += 64) {
      const int j = j0 + lane;
      const uint32_t v = j < nb ? ccnt[j] : 0;
      uint32_t inc = v;
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) {
        const uint32_t o = __shfl_up(inc, d, 64);
        if (lane >= d) inc += o;
      }
      if (j < nb) seg[j] = run + inc - v;
      run += __shfl(inc, 63, 64);
    }
  }
#pragma unroll
  for (int x = 0; x < KH; x++)
    if (js[x] >= 0) atomicOr(&mask[word * nb + js[x]], 1u << bit);
  __syncthreads();
  // per block: rows of the chunk in the words below each word
  for (int j = tid; j < nb; j += kRouteRows) {
    uint32_t acc = 0;
#pragma unroll
    for (int w = 0; w < kWords; w++) {
      pre[w * nb + j] = (uint16_t)acc;
      acc += __popc(mask[w * nb + j]);
    }
  }
  __syncthreads();
  if (valid) {
#pragma unroll
    for (int x = 0; x < KH; x++) {
      if (js[x] >= 0) {
        const int j = js[x];
        const uint32_t rank = pre[word * nb + j] +
                              __popc(mask[word * nb + j] & ((1u << bit) - 1u));
        ent[seg[j] + rank] = (uint16_t)((tid << 5) | x);
      }
    }
  }
  __syncthreads();
  // each block's run, contiguous in LDS and in the bin's list: one wave per
  // block; the chunk's rows are r0 + (row within the chunk)
  const uint64_t r0 = (uint64_t)g * ((uint64_t)p.T * p.G) + (uint64_t)(sq.tok_start + cp.tl0) * p.G;
  for (int j = wave; j < nb; j += kRouteRows / 64) {
    const uint32_t n = ccnt[j];
    if (n == 0) continue;
    uint32_t* dst = entries + bin_start[bin0 + j] + col0[(int64_t)j * nchunks + cp.r];
    const uint16_t* srcj = ent + seg[j];
    for (uint32_t e = lane; e < n; e += 64) {
      const uint32_t code = srcj[e];
      dst[e] = (uint32_t)((r0 + (code >> 5)) * (uint64_t)kh + (code & 31u));
    }
  }
}

template <int KH>
hipError_t launch_staged(dim3 grid, size_t lds, const int32_t* sel, const SeqInfo* seqs,
                         const Problem& p, const RouteBuffers& rb, hipStream_t st) {
  if (lds > 65536) {
    const hipError_t e = hipFuncSetAttribute(
        reinterpret_cast<const void*>(&route_scatter_staged_kernel<KH>),
        hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  route_scatter_staged_kernel<KH><<<grid, kRouteRows, lds, st>>>(sel, seqs, p, rb.hist,
                                                                 rb.bin_count, rb.bin_start,
                                                                 rb.entries);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_route(const int32_t* sel, const SeqInfo* seqs, const Problem& p,
                        const RouteBuffers& rb, hipStream_t st) {
  const int64_t nbins = (int64_t)p.Hkv * p.nblk_total;
  if (nbins == 0) return hipSuccess;
  if (p.route_chunks > 0) {
    dim3 grid((unsigned)p.route_chunks, p.Hkv);
    route_count_kernel<<<grid, 256, p.nblk_max * sizeof(int32_t), st>>>(sel, seqs, p, rb.hist);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  route_scan_cols_kernel<<<(unsigned)((nbins + 3) / 4), 256, 0, st>>>(seqs, p, rb.hist,
                                                                      rb.bin_count);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  route_scan_bins_kernel<<<1, 1024, 0, st>>>(rb.bin_count, nbins, p.tile_rows, rb.bin_start,
                                              rb.bin_tile_start);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (rb.tile_bin) {
    route_tile_bins_kernel<<<(unsigned)((nbins + 3) / 4), 256, 0, st>>>(rb.bin_tile_start, nbins,
                                                                        rb.tile_bin);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (p.route_chunks > 0 && p.hist_entries > 0) {
    dim3 grid((unsigned)p.route_chunks, p.Hkv);
    const int kh = p.topk - 1;
    const size_t staged = staged_lds_bytes(p.nblk_max, kh);
    if (staged <= kRouteLdsMax && kh <= 31) {
      if (kh <= 3) return launch_staged<3>(grid, staged, sel, seqs, p, rb, st);
      if (kh <= 7) return launch_staged<7>(grid, staged, sel, seqs, p, rb, st);
      if (kh <= 11) return launch_staged<11>(grid, staged, sel, seqs, p, rb, st);
      if (kh <= 15) return launch_staged<15>(grid, staged, sel, seqs, p, rb, st);
      return launch_staged<31>(grid, staged, sel, seqs, p, rb, st);
    }
    // the per-block prefix table when it fits beside the masks in LDS
    const size_t base = (size_t)p.nblk_max * 9 * sizeof(uint32_t);
    const bool use_pre = base + (size_t)p.nblk_max * 8 <= kRouteLdsMax;
    const size_t lds = use_pre ? base + (size_t)p.nblk_max * 8 : base;
    if (lds > 65536) {
      e = hipFuncSetAttribute(reinterpret_cast<const void*>(&route_scatter_kernel),
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      if (e != hipSuccess) return e;
    }
    route_scatter_kernel<<<grid, 256, lds, st>>>(
        sel, seqs, p, rb.hist, rb.bin_start, rb.entries, use_pre);
    e = hipGetLastError();
  }
  return e;
}

}  // namespace moba
