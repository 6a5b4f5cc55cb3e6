// Gate and top-k block selection (Eq. 5 and Eq. 6; the causal rules of
// Sec. 2.2: no future block, current block forced on and counted toward k).
//
// One work-group per (sequence, group of `tw` tokens, kv-head).  Its 256
// threads are (query head of the GQA group) x (token): thread i handles head
// i / tw and token i % tw, so every wave scores the same kv-head's block keys
// and its lanes read the same LDS row (broadcast).  Block keys are staged in
// LDS 64 at a time.  Each lane keeps its query row in 128 fp32 registers and
// a running top-(k-1) list in registers.
//
// Arithmetic: s_j = <q, kbar_j> in fp32 with four interleaved partial sums
// combined pairwise.  The list is kept sorted by (score desc, block asc):
// candidates arrive in ascending block order, so a newcomer is inserted after
// every entry with a score >= its own, which realises the lowest-index
// tie-break.  Unused places of the fixed-size list are +inf sentinels at the
// top (never displaced) and -inf placeholders at the bottom.
#include "moba_internal.h"

#include <math.h>

namespace moba {
namespace {

constexpr int kStage = 64;  // block keys per LDS stage

template <typename T>
__device__ __forceinline__ void load_q(const T* p, float* f);

template <>
__device__ __forceinline__ void load_q<__hip_bfloat16>(const __hip_bfloat16* p, float* f) {
#pragma unroll
  for (int c = 0; c < kHeadDim / 8; c++) {
    uint4 u = reinterpret_cast<const uint4*>(p)[c];
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; i++) {
      f[8 * c + 2 * i] = __uint_as_float(w[i] << 16);
      f[8 * c + 2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  }
}

template <>
__device__ __forceinline__ void load_q<float>(const float* p, float* f) {
#pragma unroll
  for (int c = 0; c < kHeadDim / 4; c++) {
    float4 u = reinterpret_cast<const float4*>(p)[c];
    f[4 * c] = u.x; f[4 * c + 1] = u.y; f[4 * c + 2] = u.z; f[4 * c + 3] = u.w;
  }
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
  const int64_t row = t * p.Hq + h;

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
        if constexpr (KM > 0) {
          if (sj > sc[KM - 1]) {
#pragma unroll
            for (int x = KM - 1; x >= 1; x--) {
              const bool after_prev = sj > sc[x - 1];
              const bool here = sj > sc[x];
              sc[x] = after_prev ? sc[x - 1] : (here ? sj : sc[x]);
              id[x] = after_prev ? id[x - 1] : (here ? j : id[x]);
            }
            if (sj > sc[0]) { sc[0] = sj; id[0] = j; }
          }
        }
      }
    }
  }
  if (!valid) return;
  int32_t* out = sel + row * K;
  int nh = 0;
  if constexpr (KM > 0) {
    // kept entries are those with a real block index; write them ascending
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

template <typename T, int KM>
hipError_t launch_km(const void* q, int64_t q_st, int64_t q_sh, const float* kbar,
                     const SeqInfo* seqs, const Problem& p, int32_t* sel, float* scores, int nmax,
                     hipStream_t st) {
  dim3 grid((unsigned)p.gate_groups, p.Hkv);
  gate_kernel<T, KM><<<grid, 256, 0, st>>>(static_cast<const T*>(q), q_st, q_sh, kbar, seqs, p,
                                           sel, scores, nmax);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_typed(const void* q, int64_t q_st, int64_t q_sh, const float* kbar,
                        const SeqInfo* seqs, const Problem& p, int32_t* sel, float* scores,
                        int nmax, hipStream_t st) {
  const int kh = p.topk - 1;
  if (kh >= p.nblk_max - 1) return launch_km<T, 0>(q, q_st, q_sh, kbar, seqs, p, sel, scores, nmax, st);
  if (kh <= 1) return launch_km<T, 1>(q, q_st, q_sh, kbar, seqs, p, sel, scores, nmax, st);
  if (kh <= 3) return launch_km<T, 3>(q, q_st, q_sh, kbar, seqs, p, sel, scores, nmax, st);
  if (kh <= 7) return launch_km<T, 7>(q, q_st, q_sh, kbar, seqs, p, sel, scores, nmax, st);
  if (kh <= 15) return launch_km<T, 15>(q, q_st, q_sh, kbar, seqs, p, sel, scores, nmax, st);
  if (kh <= 31) return launch_km<T, 31>(q, q_st, q_sh, kbar, seqs, p, sel, scores, nmax, st);
  return launch_km<T, 63>(q, q_st, q_sh, kbar, seqs, p, sel, scores, nmax, st);
}

}  // namespace

hipError_t launch_gate(const void* q, bool bf16, int64_t q_st, int64_t q_sh, const float* kbar,
                       const SeqInfo* seqs, const Problem& p, int32_t* sel, float* scores,
                       int nmax, hipStream_t st) {
  if (p.gate_groups == 0) return hipSuccess;
  if (bf16) return launch_typed<__hip_bfloat16>(q, q_st, q_sh, kbar, seqs, p, sel, scores, nmax, st);
  return launch_typed<float>(q, q_st, q_sh, kbar, seqs, p, sel, scores, nmax, st);
}

}  // namespace moba
