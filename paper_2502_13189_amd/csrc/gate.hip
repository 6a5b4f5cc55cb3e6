// Gate and top-k block selection (Eq. 5 and Eq. 6; the causal rules of
// Sec. 2.2: no future block, current block forced on and counted toward k).
//
// One work-group per (sequence, group of `tw` tokens, kv-head): 256 rows,
// row i is query head i / tw of the GQA group and token i % tw, so every row
// of a work-group scores the same kv-head's block keys.  Each row keeps a
// running top-(k-1) list in registers, sorted by (score desc, block asc):
// candidates arrive in ascending block order, so a newcomer is inserted after
// every entry with a score >= its own, which realises the lowest-index
// tie-break.  Unused places of the fixed-size list are +inf sentinels at the
// top (never displaced) and -inf placeholders at the bottom.
//
// bf16 queries: the scores come from the matrix cores.  Each fp32 block key
// is split exactly into three bf16 terms, kbar = hi + mid + lo (each term
// takes the next 8 significant bits, so the sum carries at least 24 and the
// remainder is below 2^-26 |kbar|; the pool kernel writes the three planes);
// a bf16 query element times a term is exact in fp32, so
// s_j = <q, hi> + <q, mid> + <q, lo> is an fp32-accumulated dot product of
// the exact operands.  Per chunk of 32 blocks a wave computes S^T (blocks x
// queries) for its 64 rows with v_mfma_f32_32x32x16_bf16 (3 terms x 8
// k-steps per 32 rows, each block-key operand feeding both 32-row sets; the
// next chunk's terms are fetched meanwhile), passes the tile through LDS so
// that each lane holds its own row's 32 scores, and inserts them in block
// order (fp32 compares; a list place's new score is one median-of-three).
// Only scores that can still enter the list are inserted: those above its
// last entry, or, in the first chunks, those at or above the last entry the
// list will have after the chunk, found first from the scores alone.
//
// fp32 queries: s_j = <q, kbar_j> on the VALU in fp32 with four interleaved
// partial sums combined pairwise, block keys broadcast from LDS.
#include "moba_internal.h"

#include <math.h>

#include <type_traits>

namespace moba {
namespace {

constexpr int kStage = 64;  // block keys per LDS stage

template <typename T>
__device__ __forceinline__ void load_q(const T* p, float* f);

template <>
__device__ __forceinline__ void load_q<float>(const float* p, float* f) {
#pragma unroll
  for (int c = 0; c < kHeadDim / 4; c++) {
    float4 u = reinterpret_cast<const float4*>(p)[c];
    f[4 * c] = u.x; f[4 * c + 1] = u.y; f[4 * c + 2] = u.z; f[4 * c + 3] = u.w;
  }
}

// Sorted insertion of block j with score sj into (sc, id) (see the header),
// branch-free: the newcomer is carried down the list and swapped with every
// entry it beats strictly, so an equal score stays below the earlier (lower
// index) entry; whatever is carried out of the bottom is dropped.
template <int KM>
__device__ __forceinline__ void insert_top(float (&sc)[KM], int (&id)[KM], float sj, int j) {
  float cs = sj;
  int ci = j;
#pragma unroll
  for (int x = 0; x < KM; x++) {
    const bool gt = cs > sc[x];
    const float hi = fmaxf(cs, sc[x]), lo = fminf(cs, sc[x]);
    const int hid = gt ? ci : id[x], lid = gt ? id[x] : ci;
    sc[x] = hi;
    id[x] = hid;
    cs = lo;
    ci = lid;
  }
}

// Writes the row's selection: kept blocks ascending, then the current block,
// then -1 padding.
template <int KM>
__device__ __forceinline__ void write_sel(int32_t* out, const int* id, int c, int K) {
  int nh = 0;
  if (KM > 0 && c >= K) {
#pragma unroll
    for (int x = 0; x < KM; x++) {
      if (id[x] < c) {
        int rank = 0;
#pragma unroll
        for (int y = 0; y < KM; y++) rank += (id[y] < id[x]) ? 1 : 0;
        out[rank] = id[x];
        nh++;
      }
    }
  } else {
    for (int j = 0; j < c; j++) out[j] = j;
    nh = c;
  }
  out[nh] = c;
  for (int x = nh + 1; x < K; x++) out[x] = -1;
}

// KM: capacity of the register list (>= topk - 1); KM == 0 selects every past
// block (topk - 1 >= every row's number of past blocks).
template <typename T, int KM>
__global__ __launch_bounds__(256) void gate_kernel(const T* __restrict__ q, int64_t q_st,
                                                   int64_t q_sh, const float* __restrict__ kbar,
                                                   const SeqInfo* __restrict__ seqs, Problem p,
                                                   int32_t* __restrict__ sel,
                                                   float* __restrict__ scores, int nmax) {
  __shared__ float4 kb[kStage][kHeadDim / 4];
  const int g = blockIdx.y;
  const int s = find_seq(seqs, p.S, (int64_t)blockIdx.x, [](const SeqInfo& x) { return x.gate_off; });
  const SeqInfo sq = seqs[s];
  const int tw = p.gate_tw;
  const int grp = blockIdx.x - sq.gate_off;
  const int hl = threadIdx.x / tw;
  const int tl = grp * tw + (int)(threadIdx.x % tw);
  const bool valid = hl < p.G && tl < sq.len;
  const int last_tok = min(grp * tw + tw, sq.len) - 1;
  const int cmax = last_tok / p.B;
  const int c = valid ? tl / p.B : 0;
  const int64_t t = (int64_t)sq.tok_start + tl;
  const int h = g * p.G + hl;
  const int K = p.topk;
  const int64_t row = t * p.Hq + h;  // scores: [T, Hq, nmax]
  const int64_t srow = t * p.sel_st + (int64_t)g * p.sel_sg + hl;

  if (valid && scores) {
    for (int j = 0; j < nmax; j++) scores[row * nmax + j] = j < c ? 0.0f : NAN;
  }

  float sc[KM > 0 ? KM : 1];
  int id[KM > 0 ? KM : 1];
  if constexpr (KM > 0) {
#pragma unroll
    for (int x = 0; x < KM; x++) {
      const bool blocked = x < KM - (K - 1);
      sc[x] = blocked ? INFINITY : -INFINITY;
      id[x] = 0x7fffffff;
    }
  }
  const bool need_scores = KM > 0 || scores != nullptr;
  if (need_scores && cmax > 0) {
    float qf[kHeadDim];
    if (valid) load_q<T>(q + t * q_st + (int64_t)hl * q_sh + (int64_t)g * p.G * q_sh, qf);
    else {
#pragma unroll
      for (int d = 0; d < kHeadDim; d++) qf[d] = 0.0f;
    }
    const float4* kbg = reinterpret_cast<const float4*>(kbar);
    for (int jc = 0; jc < cmax; jc += kStage) {
      const int nstage = min(kStage, cmax - jc);
      __syncthreads();
      for (int x = threadIdx.x; x < nstage * (kHeadDim / 4); x += 256) {
        const int jj = x / (kHeadDim / 4), c4 = x % (kHeadDim / 4);
        kb[jj][c4] = kbg[((int64_t)(sq.blk_off + jc + jj) * p.Hkv + g) * (kHeadDim / 4) + c4];
      }
      __syncthreads();
      const int jend = min(nstage, c - jc);
      for (int jj = 0; jj < jend; jj++) {
        float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
#pragma unroll
        for (int c4 = 0; c4 < kHeadDim / 4; c4++) {
          const float4 kv = kb[jj][c4];
          a0 = fmaf(qf[4 * c4 + 0], kv.x, a0);
          a1 = fmaf(qf[4 * c4 + 1], kv.y, a1);
          a2 = fmaf(qf[4 * c4 + 2], kv.z, a2);
          a3 = fmaf(qf[4 * c4 + 3], kv.w, a3);
        }
        const float sj = (a0 + a1) + (a2 + a3);
        const int j = jc + jj;
        if (scores && j < nmax) scores[row * nmax + j] = sj;
        if constexpr (KM > 0) insert_top<KM>(sc, id, sj, j);
      }
    }
  }
  if (!valid) return;
  write_sel<KM>(sel + srow * K, id, c, K);
}

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kChunk = 32;               // blocks per matrix tile
constexpr int kTermRow = kHeadDim + 8;   // bf16 per LDS row of a block-key term (272 B)
constexpr int kScoreRow = kChunk + 4;    // floats per LDS score row (144 B)

// a = median(a, b, c), in place.  Issued as assembly in program order, so a
// list rewritten from the bottom up keeps every value in its own register
// (the compiler would otherwise reorder the medians and copy the list back
// at the end of each insertion).
__device__ __forceinline__ void med3_into(float& a, float b, float c) {
  asm volatile("v_med3_f32 %0, %0, %1, %2" : "+v"(a) : "v"(b), "v"(c));
}

// Sorted insertion of block j with score sj into (lf, li) (see the header).
// The newcomer goes below every entry with a score >= its own (an equal score
// stays below the earlier, lower-index entry): with gt[x] = sj > lf[x] (a
// suffix of the list), place x takes place x-1's entry where gt[x-1], the
// newcomer where only gt[x], and keeps its own entry otherwise; the bottom
// entry drops out.  Places are rewritten from the bottom up, in place.  As
// the list is sorted, the new score of place x is the median of its own, its
// upper neighbour's and sj (one v_med3_f32).  Scores are finite; -0 and +0
// compare equal, as the selection rule treats them.
template <int KM>
__device__ __forceinline__ void insert_f(float (&lf)[KM], int (&li)[KM], float sj, int j) {
  bool gt[KM];
#pragma unroll
  for (int x = 0; x < KM; x++) gt[x] = sj > lf[x];
#pragma unroll
  for (int x = KM - 1; x >= 1; x--) {
    const int ai = gt[x - 1] ? li[x - 1] : j;
    li[x] = gt[x] ? ai : li[x];
    med3_into(lf[x], lf[x - 1], sj);
  }
  lf[0] = gt[0] ? sj : lf[0];
  li[0] = gt[0] ? j : li[0];
}

// The scores of a sorted list of KM places after inserting sj, values only.
template <int KM>
__device__ __forceinline__ void insert_value(float (&lc)[KM], float sj) {
#pragma unroll
  for (int x = KM - 1; x >= 1; x--) med3_into(lc[x], lc[x - 1], sj);
  lc[0] = fmaxf(lc[0], sj);
}

// Lists of up to 31 places run two waves per SIMD (256 registers), so one
// wave's loads and products overlap the other's selection work; at 31 places
// that spills some registers and is still faster (top-31 over 128 blocks:
// 0.45 vs 0.53 ms with one wave per SIMD and no spills).
template <int KM>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(KM <= 31 ? 2 : 1)))
void gate_mfma_kernel(const __hip_bfloat16* __restrict__ q, int64_t q_st, int64_t q_sh,
                      const __hip_bfloat16* __restrict__ kterm, const SeqInfo* __restrict__ seqs,
                      Problem p, int32_t* __restrict__ sel, float* __restrict__ scores, int nmax) {
  __shared__ __attribute__((aligned(16))) __bf16 terms[3][kChunk][kTermRow];
  __shared__ __attribute__((aligned(16))) float st[4][64][kScoreRow];
  const int g = blockIdx.y;
  const int s = find_seq(seqs, p.S, (int64_t)blockIdx.x, [](const SeqInfo& x) { return x.gate_off; });
  const SeqInfo sq = seqs[s];
  const int tw = p.gate_tw;
  const int grp = blockIdx.x - sq.gate_off;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int qc = lane & 31, hh = lane >> 5;
  const int last_tok = min(grp * tw + tw, sq.len) - 1;
  const int cmax = last_tok / p.B;
  const int K = p.topk;
  // chunks whose list bound is found first (where it pays for short lists)
  constexpr int kPreChunks = KM <= 11 ? 2 : (KM <= 15 ? 1 : 0);

  // this lane's own row (insertion and output)
  const int i = 64 * wave + lane;
  const int hl = i / tw;
  const int tl = grp * tw + i % tw;
  const bool valid = hl < p.G && tl < sq.len;
  const int c = valid ? tl / p.B : 0;
  const int64_t row = ((int64_t)sq.tok_start + tl) * p.Hq + (int64_t)g * p.G + hl;  // scores
  const int64_t srow = ((int64_t)sq.tok_start + tl) * p.sel_st + (int64_t)g * p.sel_sg + hl;
  if (valid && scores) {
    for (int j = 0; j < nmax; j++) scores[row * nmax + j] = j < c ? 0.0f : NAN;
  }

  float lf[KM > 0 ? KM : 1];
  int li[KM > 0 ? KM : 1];
  if constexpr (KM > 0) {
#pragma unroll
    for (int x = 0; x < KM; x++) {
      lf[x] = x < KM - (K - 1) ? INFINITY : -INFINITY;
      li[x] = 0x7fffffff;
    }
  }
  const bool need_scores = KM > 0 || scores != nullptr;
  if (need_scores && cmax > 0) {
    // Q^T operands of the two 32-row sets of this wave: lane (qc, hh) holds
    // dims 16 kk + 8 hh .. + 7 of row 64 wave + 32 set + qc.
    bf16x8 qf[2][8];
#pragma unroll
    for (int set = 0; set < 2; set++) {
      const int ib = 64 * wave + 32 * set + qc;
      const int hb = ib / tw, tb = grp * tw + ib % tw;
      const bool vb = hb < p.G && tb < sq.len;
      const __hip_bfloat16* qr = q + ((int64_t)sq.tok_start + (vb ? tb : 0)) * q_st +
                                 (int64_t)(g * p.G + (vb ? hb : 0)) * q_sh + 8 * hh;
#pragma unroll
      for (int kk = 0; kk < 8; kk++)
        qf[set][kk] = vb ? __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(qr + 16 * kk))
                         : bf16x8{};
    }
    // staging: thread -> block jb of the chunk, dims d0 .. d0 + 15 of each of
    // the three terms (two 16-byte pieces per term), fetched one chunk ahead
    const int jb = threadIdx.x >> 3, d0 = 16 * (threadIdx.x & 7);
    const int64_t plane = (int64_t)p.nblk_total * p.Hkv * kHeadDim;
    u32x4 pf[3][2];
    auto fetch = [&](int jc) {
      const int j = jc + jb;
      const bool in = j < sq.nblk;
      const __hip_bfloat16* src =
          kterm + (((int64_t)sq.blk_off + (in ? j : 0)) * p.Hkv + g) * kHeadDim + d0;
#pragma unroll
      for (int m = 0; m < 3; m++)
#pragma unroll
        for (int h2 = 0; h2 < 2; h2++)
          pf[m][h2] = in ? *reinterpret_cast<const u32x4*>(src + m * plane + 8 * h2) : u32x4{};
    };
    fetch(0);
    for (int jc = 0; jc < cmax; jc += kChunk) {
      __syncthreads();  // previous chunk's terms are no longer read
#pragma unroll
      for (int m = 0; m < 3; m++)
#pragma unroll
        for (int h2 = 0; h2 < 2; h2++)
          *reinterpret_cast<u32x4*>(&terms[m][jb][d0 + 8 * h2]) = pf[m][h2];
      if (jc + kChunk < cmax) fetch(jc + kChunk);  // lands during this chunk's products
      __syncthreads();
      // S^T for both 32-row sets, one term at a time (lo, mid, hi), so a
      // score is hi.q + (mid.q + lo.q) with each product summed over its
      // k-steps in ascending order.  Each block-key operand is read once and
      // feeds both sets' products; the reads run six products ahead of their
      // use (scheduling groups), so the LDS latency hides behind the matrix
      // core.
      f32x16 part[2], acc[2];
      u32x4 op[24];  // operand i: term 2 - i / 8, k-step i % 8
#pragma unroll
      for (int i = 0; i < 24; i++)
        op[i] = *reinterpret_cast<const u32x4*>(&terms[2 - i / 8][qc][16 * (i % 8) + 8 * hh]);
#pragma unroll
      for (int mi = 0; mi < 3; mi++) {
#pragma unroll
        for (int set = 0; set < 2; set++)
#pragma unroll
          for (int e = 0; e < 16; e++) acc[set][e] = 0.0f;
#pragma unroll
        for (int kk = 0; kk < 8; kk++) {
          const bf16x8 a = __builtin_bit_cast(bf16x8, op[8 * mi + kk]);
          acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[0][kk], acc[0], 0, 0, 0);
          acc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[1][kk], acc[1], 0, 0, 0);
        }
#pragma unroll
        for (int set = 0; set < 2; set++) part[set] = mi == 0 ? acc[set] : acc[set] + part[set];
      }
      __builtin_amdgcn_sched_group_barrier(0x100, 3, 0);
#pragma unroll
      for (int i = 0; i < 21; i++) {
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 6, 0);
#pragma unroll
      for (int set = 0; set < 2; set++) {
        // lane (qc, hh) holds row 32 set + qc, blocks 8 (e / 4) + 4 hh + e % 4
#pragma unroll
        for (int e4 = 0; e4 < 4; e4++) {
          float4 v;
          v.x = part[set][4 * e4 + 0];
          v.y = part[set][4 * e4 + 1];
          v.z = part[set][4 * e4 + 2];
          v.w = part[set][4 * e4 + 3];
          *reinterpret_cast<float4*>(&st[wave][32 * set + qc][8 * e4 + 4 * hh]) = v;
        }
      }
      __builtin_amdgcn_wave_barrier();
      // this lane's row: 32 scores in block order.  Only scores above the
      // list's last entry at the chunk start can enter it (the last entry
      // only rises, and an equal later score never displaces an earlier one),
      // so those are marked and inserted in block order; the other
      // insertions would leave the list unchanged.  In the first chunks,
      // where that bound is weak, the list's last score after the chunk is
      // found first (the chunk's scores inserted into a value-only copy of
      // the list); scores below it cannot be in the list after the chunk, so
      // only those at or above it are marked.
      const int jend = min(kChunk, c - jc);  // blocks from c on never enter
      const uint32_t live = jend >= kChunk ? ~0u : (jend <= 0 ? 0u : (1u << jend) - 1u);
      uint32_t msk = 0;
      if constexpr (KM > 0) {
        if (jc < kPreChunks * kChunk) {
          float lc[KM];
#pragma unroll
          for (int x = 0; x < KM; x++) lc[x] = lf[x];
#pragma unroll
          for (int b4 = 0; b4 < kChunk / 4; b4++) {
            const float4 v = *reinterpret_cast<const float4*>(&st[wave][lane][4 * b4]);
            const float f[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int e = 0; e < 4; e++) insert_value<KM>(lc, 4 * b4 + e < jend ? f[e] : -INFINITY);
          }
          const float thr = lc[KM - 1];
#pragma unroll
          for (int b4 = 0; b4 < kChunk / 4; b4++) {
            const float4 v = *reinterpret_cast<const float4*>(&st[wave][lane][4 * b4]);
            const float f[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int e = 0; e < 4; e++) msk |= (uint32_t)(f[e] >= thr) << (4 * b4 + e);
          }
        } else {
          const float thr = lf[KM - 1];
#pragma unroll
          for (int b4 = 0; b4 < kChunk / 4; b4++) {
            const float4 v = *reinterpret_cast<const float4*>(&st[wave][lane][4 * b4]);
            const float f[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int e = 0; e < 4; e++) msk |= (uint32_t)(f[e] > thr) << (4 * b4 + e);
          }
        }
      }
      // a row with at most k - 1 past blocks keeps all of them (written
      // without the list)
      msk &= c >= K ? live : 0u;
      if (scores) {  // debugging aid: the fp32 scores of this row's past blocks
        for (int b = 0; b < jend && jc + b < nmax; b++) scores[row * nmax + jc + b] = st[wave][lane][b];
      }
      if constexpr (KM > 0) {
        // the next candidate's score is read before the current insertion
        int b = __builtin_ctz(msk | (1u << 31));
        float sb = st[wave][lane][b];
        while (msk) {
          msk &= msk - 1;
          const int bn = __builtin_ctz(msk | (1u << 31));
          const float sn = st[wave][lane][bn];
          insert_f<KM>(lf, li, sb, jc + b);
          b = bn;
          sb = sn;
        }
      }
      __builtin_amdgcn_wave_barrier();
    }
  }
  if (!valid) return;
  write_sel<KM>(sel + srow * K, li, c, K);
}

template <typename T, int KM>
hipError_t launch_km(const void* q, int64_t q_st, int64_t q_sh, const float* kbar,
                     const __hip_bfloat16* kterm, const SeqInfo* seqs, const Problem& p,
                     int32_t* sel, float* scores, int nmax, hipStream_t st) {
  dim3 grid((unsigned)p.gate_groups, p.Hkv);
  if constexpr (std::is_same<T, __hip_bfloat16>::value)
    gate_mfma_kernel<KM><<<grid, 256, 0, st>>>(static_cast<const T*>(q), q_st, q_sh, kterm, seqs,
                                               p, sel, scores, nmax);
  else
    gate_kernel<T, KM><<<grid, 256, 0, st>>>(static_cast<const T*>(q), q_st, q_sh, kbar, seqs, p,
                                             sel, scores, nmax);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_typed(const void* q, int64_t q_st, int64_t q_sh, const float* kbar,
                        const __hip_bfloat16* kterm, const SeqInfo* seqs, const Problem& p,
                        int32_t* sel, float* scores, int nmax, hipStream_t st) {
  const int kh = p.topk - 1;
#define MOBA_GATE_KM(n) launch_km<T, n>(q, q_st, q_sh, kbar, kterm, seqs, p, sel, scores, nmax, st)
  if (kh >= p.nblk_max - 1) return MOBA_GATE_KM(0);
  if (kh <= 1) return MOBA_GATE_KM(1);
  if (kh <= 3) return MOBA_GATE_KM(3);
  if (kh <= 7) return MOBA_GATE_KM(7);
  if (kh <= 11) return MOBA_GATE_KM(11);
  if (kh <= 15) return MOBA_GATE_KM(15);
  if (kh <= 31) return MOBA_GATE_KM(31);
  return MOBA_GATE_KM(63);
#undef MOBA_GATE_KM
}

}  // namespace

hipError_t launch_gate(const void* q, bool bf16, int64_t q_st, int64_t q_sh, const float* kbar,
                       const __hip_bfloat16* kterm, const SeqInfo* seqs, const Problem& p,
                       int32_t* sel, float* scores, int nmax, hipStream_t st) {
  if (p.gate_groups == 0) return hipSuccess;
  if (bf16)
    return launch_typed<__hip_bfloat16>(q, q_st, q_sh, kbar, kterm, seqs, p, sel, scores, nmax, st);
  return launch_typed<float>(q, q_st, q_sh, kbar, nullptr, seqs, p, sel, scores, nmax, st);
}

}  // namespace moba
