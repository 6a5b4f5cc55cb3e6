// Routing inversion: from each query's selected history blocks to, for each
// (kv-head, block) bin, the ordered list of queries that chose it.  This is
// the "arrange the ordering of query tokens based on their assigned KV
// blocks" step of Sec. 2.3 (Algorithm 1, index_select_moba_attn_block),
// done as a stable counting sort with integer arithmetic only, so the result
// is deterministic.
//
// Rows of kv-head g are ordered r = g*T*G + t*G + hl (hl = query head within
// the GQA group).  Rows are cut into chunks of `route_rt` tokens x G heads
// within one sequence.  Four kernels:
//   count      per chunk: LDS histogram of the chunk's history selections
//              over the sequence's blocks;
//   scan_cols  per bin: exclusive prefix over the chunks of its sequence (in
//              place), and the bin total;
//   scan_bins  one work-group: exclusive scans of bin totals (entry offsets)
//              and of ceil(total / tile_rows) (attention tile offsets);
//   scatter    per chunk, 256 rows at a time: every row ORs its bit into an
//              LDS bitmask per selected block; a row's rank among the round's
//              rows that chose the same block is the popcount of the lower
//              bits, which keeps the order of rows (a stable sort).
// Entry value: r * (topk - 1) + slot, where slot is the position of the block
// in the row's ascending selection.
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
  const int nrow = cp.ntok * p.G;
  for (int i = threadIdx.x; i < nrow; i += 256) {
    const int tl = cp.tl0 + i / p.G, hl = i % p.G;
    const int c = tl / p.B;
    const int nh = min(kh, c);
    const int64_t row = ((int64_t)sq.tok_start + tl) * p.Hq + (int64_t)g * p.G + hl;
    for (int x = 0; x < nh; x++) atomicAdd(&cnt[sel[row * p.topk + x]], 1);
  }
  __syncthreads();
  int32_t* dst = hist + (int64_t)g * p.hist_words + sq.hist_off + (int64_t)cp.r * sq.nblk;
  for (int j = threadIdx.x; j < sq.nblk; j += 256) dst[j] = cnt[j];
}

__global__ __launch_bounds__(256) void route_scan_cols_kernel(const SeqInfo* __restrict__ seqs,
                                                              Problem p, int32_t* __restrict__ hist,
                                                              int32_t* __restrict__ bin_count) {
  const int64_t bin = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t nbins = (int64_t)p.Hkv * p.nblk_total;
  if (bin >= nbins) return;
  const int g = (int)(bin / p.nblk_total);
  const int b = (int)(bin % p.nblk_total);
  const int s = find_seq(seqs, p.S, b, [](const SeqInfo& x) { return x.blk_off; });
  const SeqInfo sq = seqs[s];
  const int j = b - sq.blk_off;
  const int nchunks = (sq.len + p.route_rt - 1) / p.route_rt;
  int32_t* col = hist + (int64_t)g * p.hist_words + sq.hist_off + j;
  int32_t run = 0;
  for (int r = 0; r < nchunks; r++) {
    const int32_t v = col[(int64_t)r * sq.nblk];
    col[(int64_t)r * sq.nblk] = run;
    run += v;
  }
  bin_count[bin] = run;
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
  uint32_t* mask = lds;            // [nb][8]
  uint32_t* running = lds + 8 * nb;  // [nb]
  // with use_pre: [nb][8] bytes, the set bits of each block's words below a word
  uint8_t* pre = reinterpret_cast<uint8_t*>(lds + 9 * nb);
  const int kh = p.topk - 1;
  const int tid = threadIdx.x, word = tid >> 5, bit = tid & 31;
  const int32_t* chunk_off = hist + (int64_t)g * p.hist_words + sq.hist_off + (int64_t)cp.r * nb;
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
      row = ((int64_t)sq.tok_start + tl) * p.Hq + (int64_t)g * p.G + hl;
      for (int x = 0; x < nh; x++) atomicOr(&mask[sel[row * p.topk + x] * 8 + word], 1u << bit);
    }
    __syncthreads();
    if (use_pre) {
      for (int j = tid; j < nb; j += 256) {
        uint32_t acc = 0;  // at most 7 * 32
#pragma unroll
        for (int w = 0; w < 8; w++) {
          pre[j * 8 + w] = (uint8_t)acc;
          acc += __popc(mask[j * 8 + w]);
        }
      }
      __syncthreads();
    }
    if (valid) {
      const uint64_t r = (uint64_t)g * TG + (uint64_t)(sq.tok_start + tl) * p.G + hl;
      for (int x = 0; x < nh; x++) {
        const int j = sel[row * p.topk + x];
        const uint32_t* m = mask + j * 8;
        uint32_t rank = running[j] + __popc(m[word] & ((1u << bit) - 1u));
        if (use_pre) {
          rank += pre[j * 8 + word];
        } else {
          for (int w = 0; w < word; w++) rank += __popc(m[w]);
        }
        const int64_t pos = bstart[j] + chunk_off[j] + rank;
        entries[pos] = (uint32_t)(r * (uint64_t)kh + (uint64_t)x);
      }
    }
    __syncthreads();
    for (int j = tid; j < nb; j += 256) {
      uint32_t c = 0;
#pragma unroll
      for (int w = 0; w < 8; w++) c += __popc(mask[j * 8 + w]);
      running[j] += c;
    }
    __syncthreads();
  }
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
  route_scan_cols_kernel<<<(unsigned)((nbins + 255) / 256), 256, 0, st>>>(seqs, p, rb.hist,
                                                                          rb.bin_count);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  route_scan_bins_kernel<<<1, 1024, 0, st>>>(rb.bin_count, nbins, p.tile_rows, rb.bin_start,
                                              rb.bin_tile_start);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (p.route_chunks > 0 && p.hist_entries > 0) {
    dim3 grid((unsigned)p.route_chunks, p.Hkv);
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
