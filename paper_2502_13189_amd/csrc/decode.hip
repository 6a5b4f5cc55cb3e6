// Decode: one new query per sequence against its key/value cache.  Query s
// sits at the last position L_s - 1 of sequence s (its key and value are the
// cache's last entries), so its result is the last row of the prefill over
// the cache: MoBA (the gate of Eq. 5 / Eq. 6 with the causal rules of
// Sec. 2.2, attention of Eq. 2 over the key set of Eq. 4) or causal full
// attention (Eq. 1), which is what the paper uses for generation (Sec. 3.3).
//
// Decode reads each attended key once per kv-head and does ~2 FLOP per byte,
// far below the ridge of either the matrix cores or the vector ALUs, so it is
// bound by HBM: the kernels use the vector ALUs (packed bf16 dot products,
// which halve the instruction count of fp32 FMAs on unpacked operands), read
// K rows one per lane and V rows coalesced, and in MoBA mode touch only the
// selected blocks.
//
//   gate     one work-group per (sequence, query head): fp32 scores of the
//            query against the block means of the sequence's complete past
//            blocks (coalesced loads staged through LDS; four partial sums
//            over dim quarters, added in order), then top-(k-1) (ties:
//            lower block index): up to 1024 candidates by rank, each thread
//            counting the candidates that precede its own; beyond, by k-1
//            rounds of a wave-wide argmax.  The selection is written
//            ascending with the current block last.
//   attend   one work-group per (sequence, kv-head, 256-key chunk; chunks
//            never cross a block boundary; in MoBA mode only the chunks of
//            the blocks the group's query heads selected, which each
//            work-group finds from the selections itself: its slot's block
//            in the ascending union), all query heads of the group:
//            scores with one key per lane (bf16 dot2 against the packed
//            query, fp32 sums), a per-head softmax over the chunk, P V with
//            one dimension pair per lane and 64 keys per wave (dot2 over key
//            pairs: weights rounded once to bf16, as the prefill's P V, fp32
//            sums); the value rows are all requested before the softmax; the
//            normalised partial and its lse go to the workspace; a head that
//            did not select the chunk's block skips it.
//   combine  log-sum-exp merge of each row's partials: nsplit work-groups
//            per row each fold a share of up to kCombineShare consecutive
//            partial slots (16 interleaved groups, eight partial loads in
//            flight per group, then the groups in order); with one share
//            the work-group writes the row, otherwise a second kernel folds
//            the shares in order.  Rounded once to the output dtype.
#include "decode_internal.h"

#include <math.h>

namespace moba {
namespace {

constexpr float kLn2 = 0.69314718055994531f;
constexpr float kLog2e = 1.4426950408889634f;

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ bf16x2_t as_bf16x2(uint32_t w) { return __builtin_bit_cast(bf16x2_t, w); }
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
// Two fp32 values to a packed bf16 pair, round-to-nearest-even.
__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  const f32x2_t v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Key range of chunk x of sequence length L: block j = x / nsub, piece
// i = x % nsub of kDecodeChunk keys, cut at the block end and at L.
__device__ __forceinline__ void chunk_range(int x, int nsub, int B, int64_t L, int64_t& u0,
                                            int64_t& u1) {
  const int64_t j = x / nsub, i = x % nsub;
  u0 = j * B + i * kDecodeChunk;
  u1 = min(min(u0 + kDecodeChunk, (j + 1) * (int64_t)B), L);
}

// ================================================================== gate
// One work-group per (sequence, query head).  The block means are read with
// coalesced loads (each half-wave reads one block's 512 bytes), up to 256
// blocks per pass, all of a pass's loads in flight at once; 64 blocks at a
// time go through an LDS tile (rows padded by one float, so the dot products
// read it without bank conflicts), where thread t forms the partial sum of
// block t % 64 over dims [32 q, 32 q + 32), q = t / 64, and the four partials
// are added in order.  Wave 0 then selects.
constexpr int kGatePass = 256;              // blocks per pass
constexpr int kGateChunk = 64;              // blocks per LDS tile
constexpr int kGateRow = kHeadDim + 1;      // padded LDS row (floats)
constexpr int kGateLoads = kGatePass * (kHeadDim / 4) / 256;  // float4 per thread per pass
constexpr int kRankMax = 1024;              // candidates ranked in parallel (4 per thread)

__global__ __launch_bounds__(256) void decode_gate_kernel(DecodeArgs a, Problem p) {
  __shared__ float qs[kHeadDim];
  __shared__ float sc[kMaxBlocksPerSeq];
  __shared__ float kt[kGateChunk * kGateRow];
  __shared__ float ps[4][kGateChunk];
  const int tid = threadIdx.x, lane = tid & 63;
  const int64_t row = blockIdx.x;  // s * Hq + h
  const int s = (int)(row / p.Hq), h = (int)(row % p.Hq);
  const int g = h / p.G;
  const SeqInfo sq = a.seqs[s];
  if (tid < kHeadDim / 2) {
    const __hip_bfloat16* qr = a.q + (int64_t)s * a.q_ss + (int64_t)h * a.q_sh;
    const uint32_t w = reinterpret_cast<const uint32_t*>(qr)[tid];
    qs[2 * tid] = bf16_lo(w);
    qs[2 * tid + 1] = bf16_hi(w);
  }
  const int c = (int)((sq.len - 1) / p.B);  // current block; candidates j < c
  const int jb = tid % kGateChunk, quarter = tid / kGateChunk;
  for (int j0 = 0; j0 < c; j0 += kGatePass) {
    // float4 e = tid + 256 i of the pass: block e / 32, piece e % 32
    float4 kv[kGateLoads];
#pragma unroll
    for (int i = 0; i < kGateLoads; i++) {
      const int e = tid + 256 * i;
      const int j = min(j0 + e / (kHeadDim / 4), c - 1);  // past the candidates: re-read, unused
      kv[i] = reinterpret_cast<const float4*>(
          a.kbar + ((int64_t)(sq.blk_off + j) * p.Hkv + g) * kHeadDim)[e % (kHeadDim / 4)];
    }
#pragma unroll
    for (int ch = 0; ch < kGatePass / kGateChunk; ch++) {
      if (j0 + ch * kGateChunk >= c) break;  // uniform over the work-group
      __syncthreads();  // the previous tile (and qs, first time) is done with
#pragma unroll
      for (int i = 0; i < kGateLoads / (kGatePass / kGateChunk); i++) {
        const int ii = ch * (kGateLoads / (kGatePass / kGateChunk)) + i;
        const int e = tid + 256 * ii - ch * kGateChunk * (kHeadDim / 4);
        float* dst = kt + (e / (kHeadDim / 4)) * kGateRow + 4 * (e % (kHeadDim / 4));
        dst[0] = kv[ii].x;
        dst[1] = kv[ii].y;
        dst[2] = kv[ii].z;
        dst[3] = kv[ii].w;
      }
      __syncthreads();
      float acc = 0.0f;
      const float* kr = kt + jb * kGateRow + 32 * quarter;
#pragma unroll
      for (int d = 0; d < 32; d++) acc = fmaf(qs[32 * quarter + d], kr[d], acc);
      ps[quarter][jb] = acc;
      __syncthreads();
      const int j = j0 + ch * kGateChunk + tid;
      if (tid < kGateChunk && j < c) sc[j] = ((ps[0][tid] + ps[1][tid]) + ps[2][tid]) + ps[3][tid];
    }
  }
  __syncthreads();
  const int kh = p.topk - 1;
  const int nh = min(kh, c);
  if (c <= kRankMax) {
    // top-(k-1) by rank: candidate j is kept iff fewer than nh candidates
    // precede it in (score desc, index asc) order — the same set as the
    // argmax rounds below.  Thread t ranks candidates t + 256 i against all
    // (every lane reads the same score: broadcast), then the kept ones are
    // written ascending: a kept candidate's place is the number of kept ones
    // in the earlier 64-candidate groups plus those below it in its own.
    __shared__ int gcnt[kRankMax / 64];
    const int wave = tid >> 6;
    uint64_t bal[kRankMax / 256];
#pragma unroll
    for (int i = 0; i < kRankMax / 256; i++) {
      const int j = tid + 256 * i;
      bool keep = false;
      if (j < c) {
        const float sj = sc[j];
        int above = 0;
        for (int u = 0; u < c; u++) {
          const float su = sc[u];
          above += (su > sj || (su == sj && u < j)) ? 1 : 0;
        }
        keep = above < nh;
      }
      bal[i] = __ballot(keep);
      if (lane == 0) gcnt[4 * i + wave] = __popcll(bal[i]);
    }
    __syncthreads();
    int32_t* out = a.sel + row * p.topk;
#pragma unroll
    for (int i = 0; i < kRankMax / 256; i++) {
      if ((bal[i] >> lane) & 1) {
        int pos = __popcll(bal[i] & ((uint64_t(1) << lane) - 1));
        for (int x = 0; x < 4 * i + wave; x++) pos += gcnt[x];
        out[pos] = tid + 256 * i;
      }
    }
    if (tid == 0) out[nh] = c;
    for (int x = nh + 1 + tid; x < p.topk; x += 256) out[x] = -1;
    return;
  }
  if (tid >= 64) return;
  // top-(k-1) for longer sequences: rounds of a wave-wide argmax over (score
  // desc, index asc); lane L owns candidates L, L + 64, ... and marks its
  // taken ones in a mask
  uint64_t taken = 0;
  for (int r = 0; r < nh; r++) {
    float best = -INFINITY;
    int bj = INT32_MAX;
    for (int j = lane, x = 0; j < c; j += 64, x++) {
      if ((taken >> x) & 1) continue;
      const float v = sc[j];
      if (v > best || (v == best && j < bj)) { best = v; bj = j; }
    }
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
      const float ob = __shfl_xor(best, m, 64);
      const int oj = __shfl_xor(bj, m, 64);
      if (ob > best || (ob == best && oj < bj)) { best = ob; bj = oj; }
    }
    if (bj < c && bj % 64 == lane) taken |= uint64_t(1) << (bj / 64);
  }
  // ascending: round x covers candidates 64x .. 64x+63, one per lane
  int32_t* out = a.sel + row * p.topk;
  int pos = 0;
  for (int x = 0; 64 * x < c; x++) {
    const bool mine = (taken >> x) & 1;
    const uint64_t bal = __ballot(mine);
    if (mine) out[pos + __popcll(bal & ((uint64_t(1) << lane) - 1))] = 64 * x + lane;
    pos += __popcll(bal);
  }
  if (lane == 0) out[nh] = c;
  for (int x = nh + 1 + lane; x < p.topk; x += 64) out[x] = -1;
}

// ================================================================ attend
// GM: the group size rounded up to a power of two (sizes the LDS arrays, so
// small groups leave room for more resident work-groups).
template <int GM>
__global__ __launch_bounds__(256) void decode_attend_kernel(DecodeArgs a, Problem p) {
  __shared__ uint32_t qw[GM][kHeadDim / 2];  // the group's queries, packed bf16 pairs
  __shared__ float ps[GM][kDecodeChunk];
  __shared__ uint32_t pw[GM][kDecodeChunk / 2];
  __shared__ float red[4][GM][2];
  // per-wave P V sums of each head (dims 2*lane, 2*lane+1)
  __shared__ float2 accs[4][GM][64];
  __shared__ int use_head[GM];
  __shared__ unsigned long long umask[kMaxBlocksPerSeq / 64];
  __shared__ int ublock;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int s = blockIdx.y / p.Hkv, g = blockIdx.y % p.Hkv;
  const int G = p.G;
  int x = blockIdx.x;  // chunk id: block * nsub + piece
  if (!a.full) {
    // MoBA: the grid runs over the group's selected blocks only.  Work-group
    // slot blockIdx.x / nsub takes the slot-th smallest block any head of
    // the group selected: the selections as a bitmask (lane w: blocks
    // 64w .. 64w+63), a prefix count over the lanes, then the block.
    const int slot = blockIdx.x / a.nsub;
    if (tid < 64) umask[tid] = 0;
    __syncthreads();
    const int32_t* gs = a.sel + ((int64_t)s * p.Hq + (int64_t)g * G) * p.topk;
    for (int i = tid; i < G * p.topk; i += 256) {
      const int j = gs[i];
      if (j >= 0) atomicOr(&umask[j >> 6], 1ull << (j & 63));
    }
    __syncthreads();
    if (tid < 64) {
      const unsigned long long w = umask[tid];
      const int n = __popcll(w);
      int incl = n;
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) {
        const int o = __shfl_up(incl, d, 64);
        if (lane >= d) incl += o;
      }
      if (slot >= incl - n && slot < incl) {
        unsigned long long r = w;
        for (int k = slot - (incl - n); k > 0; k--) r &= r - 1;
        ublock = 64 * tid + __ffsll((long long)r) - 1;
      }
      if (tid == 63 && slot >= incl) ublock = -1;  // fewer distinct blocks than slots
    }
    __syncthreads();
    const int j = ublock;
    if (j < 0) return;
    x = j * a.nsub + blockIdx.x % a.nsub;
  }
  const SeqInfo sq = a.seqs[s];
  int64_t u0, u1;
  chunk_range(x, a.nsub, a.chunk_block, sq.len, u0, u1);
  if (u0 >= u1) return;
  // heads of the group that attend this chunk
  if (tid < G) {
    const int h = g * G + tid;
    int use = 1;
    if (!a.full) {
      const int j = (int)(u0 / p.B);
      const int32_t* sl = a.sel + ((int64_t)s * p.Hq + h) * p.topk;
      use = 0;
      for (int y = 0; y < p.topk; y++) use |= sl[y] == j;
    }
    use_head[tid] = use;
  }
  for (int i = tid; i < G * (kHeadDim / 2); i += 256) {
    const int hl = i / (kHeadDim / 2), d2 = i % (kHeadDim / 2);
    qw[hl][d2] = reinterpret_cast<const uint32_t*>(a.q + (int64_t)s * a.q_ss +
                                                   (int64_t)(g * G + hl) * a.q_sh)[d2];
  }
  __syncthreads();
  int any = 0;
  for (int hl = 0; hl < G; hl++) any |= use_head[hl];
  if (!any) return;

  // scores: lane = key u0 + 64 * wave + lane; each lane loads its own key
  // row (16 loads of 16 bytes) into registers.  Rows past the chunk end load
  // the chunk's first row (their scores are discarded).
  const int64_t u = u0 + 64 * wave + lane;
  const bool kv_ok = u < u1;
  const int kend = (int)min((int64_t)64, u1 - (u0 + 64 * wave));  // may be <= 0
  uint32_t kw[kHeadDim / 2];  // the key row, packed bf16 pairs
  {
    const int64_t t = sq.tok_start + (kv_ok ? u : u0);
    const uint4* kp = reinterpret_cast<const uint4*>(a.k + t * a.k_st + (int64_t)g * a.k_sh);
#pragma unroll
    for (int c8 = 0; c8 < kHeadDim / 8; c8++) {
      const uint4 w = kp[c8];
      kw[4 * c8] = w.x;
      kw[4 * c8 + 1] = w.y;
      kw[4 * c8 + 2] = w.z;
      kw[4 * c8 + 3] = w.w;
    }
  }
  const float c2 = a.scale_log2;
  for (int hl = 0; hl < G; hl++) {
    // fp32 sum of exact bf16 products, two dims per instruction
    float acc = 0.0f;
#pragma unroll
    for (int d2 = 0; d2 < kHeadDim / 2; d2++)
      acc = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(qw[hl][d2]), as_bf16x2(kw[d2]), acc, false);
    const float sv = kv_ok ? acc * c2 : -INFINITY;
    float m = sv;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
    ps[hl][64 * wave + lane] = sv;
    if (lane == 0) red[wave][hl][0] = m;
  }
  // this wave's 64 value rows (dims 2*lane, 2*lane+1), all in flight across
  // the softmax below; slots past the chunk end load the chunk's first row,
  // which exists, and get weight 0
  const uint32_t* vrow = reinterpret_cast<const uint32_t*>(
      a.v + (sq.tok_start + u0) * a.v_st + (int64_t)g * a.v_sh) + lane;
  uint32_t wv[64];
#pragma unroll
  for (int e = 0; e < 64; e++) wv[e] = vrow[(int64_t)(e < kend ? 64 * wave + e : 0) * a.v_st / 2];
  __syncthreads();
  // per head: chunk max, weights, sum
  for (int hl = 0; hl < G; hl++) {
    const float m = fmaxf(fmaxf(red[0][hl][0], red[1][hl][0]), fmaxf(red[2][hl][0], red[3][hl][0]));
    const float pv = kv_ok ? __builtin_amdgcn_exp2f(ps[hl][64 * wave + lane] - m) : 0.0f;
    // weights of keys 2i, 2i+1 as one bf16 pair (the operand of the P V dot2)
    const float pn = __shfl_xor(pv, 1, 64);
    if ((lane & 1) == 0) pw[hl][32 * wave + (lane >> 1)] = pack_bf16(pv, pn);
    float l = pv;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) l += __shfl_xor(l, o, 64);
    if (lane == 0) red[wave][hl][1] = l;
  }
  __syncthreads();
  // P V: wave w sums keys 64w .. 64w+63 for dims 2*lane, 2*lane+1, a key
  // pair per dot2 (weights rounded once to bf16, fp32 accumulation); slots
  // past the chunk end carry weight 0
  float2 acc[GM];
#pragma unroll
  for (int hl = 0; hl < GM; hl++) acc[hl] = make_float2(0.0f, 0.0f);
#pragma unroll
  for (int e2 = 0; e2 < 32; e2++) {
    const uint32_t v_lo = wv[2 * e2], v_hi = wv[2 * e2 + 1];
    const uint32_t vx = __builtin_amdgcn_perm(v_hi, v_lo, 0x05040100u);  // dim 2*lane of both keys
    const uint32_t vy = __builtin_amdgcn_perm(v_hi, v_lo, 0x07060302u);  // dim 2*lane+1
#pragma unroll
    for (int hl = 0; hl < GM; hl++) {
      if (hl < G) {
        const bf16x2_t pp = as_bf16x2(pw[hl][32 * wave + e2]);
        acc[hl].x = __builtin_amdgcn_fdot2_f32_bf16(pp, as_bf16x2(vx), acc[hl].x, false);
        acc[hl].y = __builtin_amdgcn_fdot2_f32_bf16(pp, as_bf16x2(vy), acc[hl].y, false);
      }
    }
  }
#pragma unroll
  for (int hl = 0; hl < GM; hl++)
    if (hl < G) accs[wave][hl][lane] = acc[hl];
  __syncthreads();
  // normalised partial and lse per attending head; wave w handles heads w, w+4, ...
  for (int hl = wave; hl < G; hl += 4) {
    if (!use_head[hl]) continue;
    const float m = fmaxf(fmaxf(red[0][hl][0], red[1][hl][0]), fmaxf(red[2][hl][0], red[3][hl][0]));
    const float l = red[0][hl][1] + red[1][hl][1] + red[2][hl][1] + red[3][hl][1];
    const float inv = 1.0f / l;
    float2 o = accs[0][hl][lane];
#pragma unroll
    for (int w = 1; w < 4; w++) {
      o.x += accs[w][hl][lane].x;
      o.y += accs[w][hl][lane].y;
    }
    const int64_t pr = ((int64_t)s * p.Hq + g * G + hl) * a.nchunk + x;
    reinterpret_cast<float2*>(a.part_o + pr * kHeadDim)[lane] = make_float2(o.x * inv, o.y * inv);
    if (lane == 0) a.part_lse[pr] = (m + __builtin_amdgcn_logf(l)) * kLn2;
  }
}

// =============================================================== combine
// One work-group per row: 16 groups of 16 lanes each fold every 16th of the
// row's partials (8 dims per lane, online rescale), then the 16 group results
// are merged in group order.
__global__ __launch_bounds__(256) void decode_combine_kernel(DecodeArgs a, Problem p) {
  __shared__ float gm[16], gw[16];
  __shared__ float go[16][kHeadDim];
  const int64_t row = blockIdx.x / a.nsplit;  // s * Hq + h
  const int share = (int)(blockIdx.x % a.nsplit);
  const int xb = share * a.split_len;  // this work-group's partial slots start here
  const int grp = threadIdx.x / 16, l16 = threadIdx.x % 16;
  const int s = (int)(row / p.Hq), h = (int)(row % p.Hq);
  const SeqInfo sq = a.seqs[s];
  float M = -INFINITY, wsum = 0.0f, acc[8];
#pragma unroll
  for (int d = 0; d < 8; d++) acc[d] = 0.0f;
  auto fold_loaded = [&](float lv, float4 o0, float4 o1) {
    const float Mn = fmaxf(M, lv);
    const float sc = __builtin_amdgcn_exp2f((M - Mn) * kLog2e);
    const float w = __builtin_amdgcn_exp2f((lv - Mn) * kLog2e);
    const float f[8] = {o0.x, o0.y, o0.z, o0.w, o1.x, o1.y, o1.z, o1.w};
#pragma unroll
    for (int d = 0; d < 8; d++) acc[d] = fmaf(w, f[d], acc[d] * sc);
    wsum = wsum * sc + w;
    M = Mn;
  };
  if (a.full) {
    // the group's partials x = grp + 16 i, eight loads in flight per round
    constexpr int kAhead = 8;
    const int n = min((int)((sq.len + kDecodeChunk - 1) / kDecodeChunk), xb + a.split_len);
    for (int x0 = xb + grp; x0 < n; x0 += 16 * kAhead) {
      float lv[kAhead];
      float4 o0[kAhead], o1[kAhead];
#pragma unroll
      for (int e = 0; e < kAhead; e++) {
        const int x = min(x0 + 16 * e, n - 1);
        const int64_t pr = row * a.nchunk + x;
        const float4* op = reinterpret_cast<const float4*>(a.part_o + pr * kHeadDim + 8 * l16);
        lv[e] = a.part_lse[pr];
        o0[e] = op[0];
        o1[e] = op[1];
      }
#pragma unroll
      for (int e = 0; e < kAhead; e++)
        if (x0 + 16 * e < n) fold_loaded(lv[e], o0[e], o1[e]);
    }
  } else {
    // the row's chunks: z = y * nsub + i for selection entry y, piece i;
    // the group's z = grp + 16 i, eight loads in flight per round
    constexpr int kAhead = 8;
    const int32_t* sl = a.sel + row * p.topk;
    const int zend = min(p.topk * a.nsub, xb + a.split_len);
    for (int z0 = xb + grp; z0 < zend; z0 += 16 * kAhead) {
      float lv[kAhead];
      float4 o0[kAhead], o1[kAhead];
      bool ok[kAhead];
#pragma unroll
      for (int e = 0; e < kAhead; e++) {
        const int z = z0 + 16 * e;
        ok[e] = false;
        if (z < zend) {
          const int y = z / a.nsub, i = z % a.nsub;
          const int j = sl[y];
          const int64_t u0 = (int64_t)j * p.B + (int64_t)i * kDecodeChunk;
          if (j >= 0 && u0 < min((int64_t)(j + 1) * p.B, (int64_t)sq.len)) {
            ok[e] = true;
            const int64_t pr = row * a.nchunk + j * a.nsub + i;
            const float4* op = reinterpret_cast<const float4*>(a.part_o + pr * kHeadDim + 8 * l16);
            lv[e] = a.part_lse[pr];
            o0[e] = op[0];
            o1[e] = op[1];
          }
        }
      }
#pragma unroll
      for (int e = 0; e < kAhead; e++)
        if (ok[e]) fold_loaded(lv[e], o0[e], o1[e]);
    }
  }
#pragma unroll
  for (int d = 0; d < 8; d++) go[grp][8 * l16 + d] = acc[d];
  if (l16 == 0) {
    gm[grp] = M;
    gw[grp] = wsum;
  }
  __syncthreads();
  if (threadIdx.x >= kHeadDim) return;
  const int d = threadIdx.x;
  float Mt = -INFINITY;
#pragma unroll
  for (int x = 0; x < 16; x++) Mt = fmaxf(Mt, gm[x]);
  float o = 0.0f, wt = 0.0f;
#pragma unroll
  for (int x = 0; x < 16; x++) {
    if (gw[x] == 0.0f) continue;  // a group without partials
    const float sc = __builtin_amdgcn_exp2f((gm[x] - Mt) * kLog2e);
    o = fmaf(sc, go[x][d], o);
    wt = fmaf(sc, gw[x], wt);
  }
  if (a.nsplit == 1) {
    a.out[(int64_t)s * a.o_ss + (int64_t)h * a.o_sh + d] = __float2bfloat16(o / wt);
    if (d == 0) a.lse[(int64_t)h * p.S + s] = Mt + __builtin_amdgcn_logf(wt) * kLn2;
    return;
  }
  // a share without partials leaves weight sum 0, which the second pass skips
  float* m = a.mid + (int64_t)blockIdx.x * (kHeadDim + 2);
  m[d] = o;
  if (d == 0) {
    m[kHeadDim] = Mt;
    m[kHeadDim + 1] = wt;
  }
}

// Second pass: one work-group per row folds its shares in order (every row
// has at least the partial of the chunk holding its own key).
__global__ __launch_bounds__(kHeadDim) void decode_fold_kernel(DecodeArgs a, Problem p) {
  static_assert(kCombineMaxSplit <= kHeadDim, "one thread per share loads its max and sum");
  __shared__ float sm[kCombineMaxSplit], sw[kCombineMaxSplit];
  const int64_t row = blockIdx.x;
  const int s = (int)(row / p.Hq), h = (int)(row % p.Hq);
  const int d = threadIdx.x;
  const float* m = a.mid + row * a.nsplit * (kHeadDim + 2);
  if (d < a.nsplit) {
    sm[d] = m[(int64_t)d * (kHeadDim + 2) + kHeadDim];
    sw[d] = m[(int64_t)d * (kHeadDim + 2) + kHeadDim + 1];
  }
  __syncthreads();
  float Mt = -INFINITY;
  for (int x = 0; x < a.nsplit; x++)
    if (sw[x] != 0.0f) Mt = fmaxf(Mt, sm[x]);
  // every share's value in flight at once (slots past the last share
  // re-read it and are not used)
  float v[kCombineMaxSplit];
#pragma unroll
  for (int x = 0; x < kCombineMaxSplit; x++)
    v[x] = m[(int64_t)min(x, a.nsplit - 1) * (kHeadDim + 2) + d];
  float o = 0.0f, wt = 0.0f;
#pragma unroll
  for (int x = 0; x < kCombineMaxSplit; x++) {
    if (x >= a.nsplit || sw[x] == 0.0f) continue;
    const float sc = __builtin_amdgcn_exp2f((sm[x] - Mt) * kLog2e);
    o = fmaf(sc, v[x], o);
    wt = fmaf(sc, sw[x], wt);
  }
  a.out[(int64_t)s * a.o_ss + (int64_t)h * a.o_sh + d] = __float2bfloat16(o / wt);
  if (d == 0) a.lse[(int64_t)h * p.S + s] = Mt + __builtin_amdgcn_logf(wt) * kLn2;
}

}  // namespace

hipError_t launch_decode_gate(const DecodeArgs& a, const Problem& p, hipStream_t st) {
  const int64_t rows = (int64_t)p.S * p.Hq;
  if (rows <= 0 || a.full) return hipSuccess;
  decode_gate_kernel<<<(unsigned)rows, 256, 0, st>>>(a, p);
  return hipGetLastError();
}

hipError_t launch_decode_attend(const DecodeArgs& a, const Problem& p, hipStream_t st) {
  if (p.S <= 0 || a.nchunk <= 0) return hipSuccess;
  const int nx = a.full ? a.nchunk : a.nunion * a.nsub;
  dim3 grid((unsigned)nx, (unsigned)(p.S * p.Hkv));
  if (p.G <= 1) decode_attend_kernel<1><<<grid, 256, 0, st>>>(a, p);
  else if (p.G <= 2) decode_attend_kernel<2><<<grid, 256, 0, st>>>(a, p);
  else if (p.G <= 4) decode_attend_kernel<4><<<grid, 256, 0, st>>>(a, p);
  else if (p.G <= 8) decode_attend_kernel<8><<<grid, 256, 0, st>>>(a, p);
  else decode_attend_kernel<kDecodeMaxGroup><<<grid, 256, 0, st>>>(a, p);
  return hipGetLastError();
}

hipError_t launch_decode_combine(const DecodeArgs& a, const Problem& p, hipStream_t st) {
  const int64_t rows = (int64_t)p.S * p.Hq;
  if (rows <= 0) return hipSuccess;
  decode_combine_kernel<<<(unsigned)(rows * a.nsplit), 256, 0, st>>>(a, p);
  if (a.nsplit == 1) return hipGetLastError();
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  decode_fold_kernel<<<(unsigned)rows, kHeadDim, 0, st>>>(a, p);
  return hipGetLastError();
}

}  // namespace moba
