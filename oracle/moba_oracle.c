/*
 * moba_oracle.c -- plain, slow, fp64 CPU reference of MoBA's causal prefill
 * forward pass (Mixture of Block Attention, arXiv 2502.13189).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the checker the GPU library is
 * compared against.  Only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg load it; the product path never does.  It shares no code,
 * header, table or helper with the HIP library.
 *
 * Every step follows the paper's definitions literally, in fp64, with one
 * plain loop nest per step and no blocking, fusion or reordering:
 *
 *   pool    : block key = mean of the keys of each block            (Sec. 2.2, Eq. 3 and Eq. 6;
 *                                                                     Alg. 1, mean_pool)
 *   select  : s_j = <q, block key j>, unscaled                       (Eq. 6; Alg. 1, S = Q Kbar^T)
 *             future blocks masked, current block forced on,         (Sec. 2.2, "Causality" and
 *             current block counts toward top-k                       "Current Block Attention";
 *                                                                     Sec. 3.1 footnote on top-3)
 *             top-k with the lower block index winning ties          (Eq. 5; tie rule is our reading)
 *   attend  : softmax over the union of the selected blocks,         (Eq. 2 and Eq. 4)
 *             causal inside the current block                        (Sec. 2.2, "Current Block Attention")
 *   dense   : causal softmax attention over the whole prefix         (Eq. 1)
 *   backward: gradients of attend w.r.t. q, k, v for a fixed         (chain rule through Eq. 2;
 *             selection (the hard gate passes no gradient)            Eq. 3 and Eq. 5 are 0/1)
 *
 * Readings where the paper is silent (each also listed in the design notes):
 *   - logit scale 1/sqrt(d) in the attention softmax (Eq. 1/2 print none; it
 *     is the default of the FlashAttention calls in Alg. 1); the gate score is
 *     unscaled as Eq. 6 prints it;
 *   - blocks restart at every sequence of a packed batch; a sequence's last
 *     block may be short (mean over its actual tokens) and is only ever a
 *     current block;
 *   - GQA: kv-head g = h / (Hq / Hkv); gating per query head against that
 *     kv-head's block keys;
 *   - lse is the natural-log log-sum-exp of the scaled logits.
 *
 * Inputs are raw element arrays in [T, H, D] row-major order, either fp32
 * (dtype 0) or bf16 bit patterns (dtype 1); bf16 is widened exactly to fp64.
 * Parity of every function here is pinned by the CPU test suite (dense
 * equivalence at top-k >= #blocks, per-block causal attention at top-k = 1,
 * brute-force subset enumeration, constructed ties, invariances, the paper's
 * tail-sparsity figures; for the backward: fp64 autograd of causal attention
 * in the dense and top-1 special cases, finite differences of attend, a closed
 * form, and the sum identities of softmax-attention gradients).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORC_OK 0
#define ORC_EARG 1
#define ORC_ENOMEM 2

/* Exact widening of one input element to fp64. */
static double elem(const void* p, int dtype, int64_t i) {
  if (dtype == 0) return (double)((const float*)p)[i];
  uint32_t bits = ((uint32_t)((const uint16_t*)p)[i]) << 16;
  float f;
  memcpy(&f, &bits, sizeof f);
  return (double)f;
}

/* Sequence that holds token t: the s with cu[s] <= t < cu[s+1]. */
static int seq_of(const int32_t* cu, int S, int64_t t) {
  int lo = 0, hi = S - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) / 2;
    if (cu[mid] <= t) lo = mid; else hi = mid - 1;
  }
  /* skip empty sequences that share the same start */
  while (lo + 1 < S && cu[lo + 1] <= t) lo++;
  return lo;
}

static int64_t nblocks(int64_t L, int B) { return (L + B - 1) / B; }

/* First global block index of each sequence; returns the total block count. */
static int64_t block_offsets(const int32_t* cu, int S, int B, int64_t* off) {
  int64_t acc = 0;
  for (int s = 0; s < S; s++) {
    off[s] = acc;
    acc += nblocks((int64_t)cu[s + 1] - cu[s], B);
  }
  return acc;
}

int moba_oracle_num_blocks(const int32_t* cu, int S, int B) {
  int64_t tot = 0;
  for (int s = 0; s < S; s++) tot += nblocks((int64_t)cu[s + 1] - cu[s], B);
  return (int)tot;
}

static int check_common(int64_t T, int Hq, int Hkv, int D, const int32_t* cu, int S) {
  if (T < 0 || Hq <= 0 || Hkv <= 0 || D <= 0 || S < 0 || Hq % Hkv != 0) return ORC_EARG;
  if (S > 0) {
    if (!cu || cu[0] != 0 || cu[S] != T) return ORC_EARG;
    for (int s = 0; s < S; s++)
      if (cu[s + 1] < cu[s]) return ORC_EARG;
  }
  return ORC_OK;
}

/*
 * Block mean-pool (Eq. 6; Alg. 1 mean_pool).  kbar[b, g, :] is the mean of
 * K[t, g, :] over the tokens t of global block b.  kabs (nullable) receives the
 * mean of |K| over the same tokens, used only by the tests' near-tie
 * tolerance.  Layout of both: [nblk_total, Hkv, D].
 */
int moba_oracle_pool(const void* k, int dtype, int64_t T, int Hkv, int D,
                     const int32_t* cu, int S, int B, double* kbar, double* kabs) {
  if (check_common(T, Hkv, Hkv, D, cu, S) != ORC_OK || B < 1 || !kbar) return ORC_EARG;
  int64_t* off = (int64_t*)malloc(sizeof(int64_t) * (S + 1));
  if (!off) return ORC_ENOMEM;
  block_offsets(cu, S, B, off);
  for (int s = 0; s < S; s++) {
    int64_t L = (int64_t)cu[s + 1] - cu[s];
    int64_t n = nblocks(L, B);
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t j = 0; j < n; j++) {
      int64_t t0 = cu[s] + j * B;
      int64_t t1 = cu[s] + ((j + 1) * B < L ? (j + 1) * B : L);
      for (int g = 0; g < Hkv; g++) {
        double* dst = kbar + ((off[s] + j) * Hkv + g) * D;
        double* dsta = kabs ? kabs + ((off[s] + j) * Hkv + g) * D : NULL;
        for (int d = 0; d < D; d++) {
          double acc = 0.0, acca = 0.0;
          for (int64_t t = t0; t < t1; t++) {
            double x = elem(k, dtype, (t * Hkv + g) * D + d);
            acc += x;
            acca += fabs(x);
          }
          dst[d] = acc / (double)(t1 - t0);
          if (dsta) dsta[d] = acca / (double)(t1 - t0);
        }
      }
    }
  }
  free(off);
  return ORC_OK;
}

typedef struct {
  double s;
  int j;
} scored_block;

/* Order for Topk (Eq. 5): higher score first; on equal scores the lower
 * block index wins. */
static int by_score_then_index(const void* a, const void* b) {
  const scored_block* x = (const scored_block*)a;
  const scored_block* y = (const scored_block*)b;
  if (x->s > y->s) return -1;
  if (x->s < y->s) return 1;
  return (x->j > y->j) - (x->j < y->j);
}

static int cmp_int(const void* a, const void* b) {
  int x = *(const int*)a, y = *(const int*)b;
  return (x > y) - (x < y);
}

/*
 * Gate (Eq. 5 and Eq. 6; Alg. 1 S = Q Kbar^T, causal mask, topk) for the
 * listed rows (row id r = t * Hq + h; rows == NULL means all T * Hq rows in
 * order).  q is [T, Hq, D], or with q_compact the listed rows' query vectors
 * only, [nrows, D] in list order (for problems too large to copy whole).
 * For a query in local block c of its sequence:
 *   - candidates are the past blocks j < c (future blocks get s = -inf and
 *     g = 0, and block c itself is forced on rather than scored);
 *   - the current block occupies one of the k places, so at most k - 1
 *     history blocks are kept: the first min(k - 1, c) of the candidates in
 *     (score desc, index asc) order;
 *   - sel[row, :] = kept history blocks ascending, then c, then -1 padding.
 * scores (nullable) receives the unscaled s_j for j < c, and NaN elsewhere,
 * in a [nrows, nmax] array.
 */
int moba_oracle_select(const void* q, int dtype, int64_t T, int Hq, int Hkv, int D,
                       const int32_t* cu, int S, int B, int topk, const double* kbar,
                       const int64_t* rows, int64_t nrows, int32_t* sel,
                       double* scores, int64_t nmax, int q_compact) {
  if (check_common(T, Hq, Hkv, D, cu, S) != ORC_OK || B < 1 || topk < 1 || !kbar || !sel)
    return ORC_EARG;
  if (q_compact && !rows) return ORC_EARG;
  if (!rows) nrows = T * Hq;
  int64_t* off = (int64_t*)malloc(sizeof(int64_t) * (S + 1));
  if (!off) return ORC_ENOMEM;
  block_offsets(cu, S, B, off);
  int G = Hq / Hkv;
  int fail = 0;
#pragma omp parallel
  {
    int64_t cap = 0;
    scored_block* cand = NULL;
#pragma omp for schedule(dynamic, 256)
    for (int64_t i = 0; i < nrows; i++) {
      int64_t r = rows ? rows[i] : i;
      int64_t t = r / Hq;
      int h = (int)(r % Hq);
      int g = h / G;
      int s = seq_of(cu, S, t);
      int64_t tau = t - cu[s];
      int c = (int)(tau / B);
      int64_t qoff = q_compact ? i * D : (t * Hq + h) * D;
      if (c > cap) {
        free(cand);
        cap = c;
        cand = (scored_block*)malloc(sizeof(scored_block) * (size_t)cap);
        if (!cand) { fail = 1; cap = 0; }
      }
      int32_t* out = sel + i * topk;
      for (int x = 0; x < topk; x++) out[x] = -1;
      if (scores)
        for (int64_t x = 0; x < nmax; x++) scores[i * nmax + x] = NAN;
      if (c > 0 && !cand) continue;
      for (int j = 0; j < c; j++) {
        const double* kb = kbar + ((off[s] + j) * Hkv + g) * D;
        double acc = 0.0;
        for (int d = 0; d < D; d++) acc += elem(q, dtype, qoff + d) * kb[d];
        cand[j].s = acc;
        cand[j].j = j;
        if (scores && j < nmax) scores[i * nmax + j] = acc;
      }
      qsort(cand, (size_t)c, sizeof(scored_block), by_score_then_index);
      int nh = c < topk - 1 ? c : topk - 1;
      for (int x = 0; x < nh; x++) out[x] = cand[x].j;
      qsort(out, (size_t)nh, sizeof(int32_t), cmp_int);
      out[nh] = c;
    }
    free(cand);
  }
  free(off);
  return fail ? ORC_ENOMEM : ORC_OK;
}

/*
 * Softmax attention of one query row over an explicit key list (Eq. 2),
 * two-pass: max, then normalised weights.  out[D] and *lse in fp64.
 */
static void attend_keys(const void* q, const void* k, const void* v, int dtype, int Hkv,
                        int D, int64_t qoff, int g, const int64_t* keys, int64_t nk, double* z,
                        double* out, double* lse) {
  double scale = 1.0 / sqrt((double)D);
  double m = -INFINITY;
  for (int64_t x = 0; x < nk; x++) {
    int64_t u = keys[x];
    double acc = 0.0;
    for (int d = 0; d < D; d++)
      acc += elem(q, dtype, qoff + d) * elem(k, dtype, (u * Hkv + g) * D + d);
    z[x] = scale * acc;
    if (z[x] > m) m = z[x];
  }
  double l = 0.0;
  for (int64_t x = 0; x < nk; x++) l += exp(z[x] - m);
  for (int d = 0; d < D; d++) out[d] = 0.0;
  for (int64_t x = 0; x < nk; x++) {
    double p = exp(z[x] - m) / l;
    int64_t u = keys[x];
    for (int d = 0; d < D; d++) out[d] += p * elem(v, dtype, (u * Hkv + g) * D + d);
  }
  *lse = m + log(l);
}

/*
 * MoBA attention given a block selection (Eq. 2 with the key set of Eq. 4):
 * for each listed row with selection sel[i, :] (local block indices, -1
 * padded), the keys are every token of each selected block j < c, plus the
 * tokens of the current block c up to and including the query itself (the
 * causal mask inside the current block).  Outputs out[nrows, D], lse[nrows].
 * q as in moba_oracle_select (q_compact: the listed rows only).
 */
int moba_oracle_attend(const void* q, const void* k, const void* v, int dtype, int64_t T,
                       int Hq, int Hkv, int D, const int32_t* cu, int S, int B, int topk,
                       const int32_t* sel, const int64_t* rows, int64_t nrows, double* out,
                       double* lse, int q_compact) {
  if (check_common(T, Hq, Hkv, D, cu, S) != ORC_OK || B < 1 || topk < 1 || !sel || !out || !lse)
    return ORC_EARG;
  if (q_compact && !rows) return ORC_EARG;
  if (!rows) nrows = T * Hq;
  int G = Hq / Hkv;
  int fail = 0;
#pragma omp parallel
  {
    int64_t cap = 0;
    int64_t* keys = NULL;
    double* z = NULL;
#pragma omp for schedule(dynamic, 64)
    for (int64_t i = 0; i < nrows; i++) {
      int64_t r = rows ? rows[i] : i;
      int64_t t = r / Hq;
      int h = (int)(r % Hq);
      int g = h / G;
      int s = seq_of(cu, S, t);
      int64_t L = (int64_t)cu[s + 1] - cu[s];
      int64_t tau = t - cu[s];
      int64_t c = tau / B;
      int64_t need = (int64_t)topk * B;
      if (need > cap) {
        free(keys); free(z);
        cap = need;
        keys = (int64_t*)malloc(sizeof(int64_t) * cap);
        z = (double*)malloc(sizeof(double) * cap);
        if (!keys || !z) { fail = 1; cap = 0; free(keys); free(z); keys = NULL; z = NULL; }
      }
      if (!keys) continue;
      int64_t nk = 0;
      for (int x = 0; x < topk; x++) {
        int64_t j = sel[i * topk + x];
        if (j < 0) continue;
        if (j > c) { fail = 1; continue; } /* future block: never valid */
        int64_t u0 = j * B;
        int64_t u1 = (j == c) ? tau + 1 : ((j + 1) * B < L ? (j + 1) * B : L);
        for (int64_t u = u0; u < u1; u++) keys[nk++] = cu[s] + u;
      }
      int64_t qoff = q_compact ? i * D : (t * Hq + h) * D;
      attend_keys(q, k, v, dtype, Hkv, D, qoff, g, keys, nk, z, out + i * D, lse + i);
    }
    free(keys);
    free(z);
  }
  return fail ? ORC_EARG : ORC_OK;
}

/*
 * Gradients of MoBA attention given a block selection: the chain rule
 * through Eq. 2 over the key set of Eq. 4.  The gate is a hard 0/1 choice
 * (Eq. 3 and Eq. 5), so no gradient flows into the block keys or the gate
 * scores; only the attention over the selected keys is differentiated.
 *
 * For each listed row (t, h) with key set U (as in moba_oracle_attend),
 * logits z_u = <q, k_u> / sqrt(D), weights p_u = exp(z_u) / sum_w exp(z_w),
 * output o = sum_u p_u v_u, and upstream gradient go = dout[t, h]:
 *   dp_u = <go, v_u>                      (gradient of o w.r.t. p_u)
 *   dz_u = p_u (dp_u - sum_w p_w dp_w)    (softmax Jacobian)
 *   dq   = sum_u dz_u k_u / sqrt(D)
 *   dk_u += dz_u q / sqrt(D)
 *   dv_u += p_u go
 * q and dout are [T, Hq, D], or with q_compact the listed rows only,
 * [nrows, D] in list order.  dq [nrows, D] (nullable).  dk and dv (nullable,
 * both or neither) receive the listed rows' contributions to the keys of
 * tokens kv_lo <= u < kv_hi, as [(kv_hi - kv_lo), Hkv, D]; the contributions
 * to a kv-head sum over the query heads of its group.  Each thread
 * accumulates into private dk/dv arrays, added up in thread order at the end.
 *
 * cq, ck, cv (nullable; ck and cv need dk) receive, in the layouts of dq, dk
 * and dv, the sums of absolute terms that bound a rounded evaluation (used
 * only by the tests' tolerances), with d_row = sum over dims |go| |o|:
 *   cq = sum_u (|dz_u| + p_u d_row) |k_u| / sqrt(D)
 *   ck_u += (|dz_u| + p_u d_row) |q| / sqrt(D)
 *   cv_u += p_u |go|
 */
static void backward_row(const void* q, const void* k, const void* v, const void* dout,
                         int dtype, int Hkv, int D, int64_t qoff, int g, const int64_t* keys,
                         int64_t nk, double* z, double* dpv, double* dq, int64_t kv_lo,
                         int64_t kv_hi, double* dk, double* dv, double* cq, double* ck,
                         double* cv) {
  double scale = 1.0 / sqrt((double)D);
  double m = -INFINITY;
  for (int64_t x = 0; x < nk; x++) {
    int64_t u = keys[x];
    double acc = 0.0;
    for (int d = 0; d < D; d++)
      acc += elem(q, dtype, qoff + d) * elem(k, dtype, (u * Hkv + g) * D + d);
    z[x] = scale * acc;
    if (z[x] > m) m = z[x];
  }
  double l = 0.0;
  for (int64_t x = 0; x < nk; x++) l += exp(z[x] - m);
  /* z[x] becomes p_u, dpv[x] becomes dp_u; then sum_w p_w dp_w */
  double pdp = 0.0;
  for (int64_t x = 0; x < nk; x++) {
    int64_t u = keys[x];
    z[x] = exp(z[x] - m) / l;
    double acc = 0.0;
    for (int d = 0; d < D; d++)
      acc += elem(dout, dtype, qoff + d) * elem(v, dtype, (u * Hkv + g) * D + d);
    dpv[x] = acc;
    pdp += z[x] * acc;
  }
  /* d_row = sum over dims of |go| |o|, o = sum_u p_u v_u (bounds only) */
  double drow = 0.0;
  if (cq || ck)
    for (int d = 0; d < D; d++) {
      double o = 0.0;
      for (int64_t x = 0; x < nk; x++) o += z[x] * elem(v, dtype, (keys[x] * Hkv + g) * D + d);
      drow += fabs(elem(dout, dtype, qoff + d)) * fabs(o);
    }
  if (dq)
    for (int d = 0; d < D; d++) dq[d] = 0.0;
  if (cq)
    for (int d = 0; d < D; d++) cq[d] = 0.0;
  for (int64_t x = 0; x < nk; x++) {
    int64_t u = keys[x];
    double dz = z[x] * (dpv[x] - pdp);
    double az = fabs(dz) + z[x] * drow;
    if (dq)
      for (int d = 0; d < D; d++) dq[d] += dz * scale * elem(k, dtype, (u * Hkv + g) * D + d);
    if (cq)
      for (int d = 0; d < D; d++) cq[d] += az * scale * fabs(elem(k, dtype, (u * Hkv + g) * D + d));
    if (dk && u >= kv_lo && u < kv_hi) {
      double* dkr = dk + ((u - kv_lo) * Hkv + g) * D;
      double* dvr = dv + ((u - kv_lo) * Hkv + g) * D;
      for (int d = 0; d < D; d++) {
        dkr[d] += dz * scale * elem(q, dtype, qoff + d);
        dvr[d] += z[x] * elem(dout, dtype, qoff + d);
      }
      if (ck) {
        double* ckr = ck + ((u - kv_lo) * Hkv + g) * D;
        double* cvr = cv + ((u - kv_lo) * Hkv + g) * D;
        for (int d = 0; d < D; d++) {
          ckr[d] += az * scale * fabs(elem(q, dtype, qoff + d));
          cvr[d] += z[x] * fabs(elem(dout, dtype, qoff + d));
        }
      }
    }
  }
}

int moba_oracle_attend_backward(const void* q, const void* k, const void* v, const void* dout,
                                int dtype, int64_t T, int Hq, int Hkv, int D, const int32_t* cu,
                                int S, int B, int topk, const int32_t* sel, const int64_t* rows,
                                int64_t nrows, int q_compact, double* dq, int64_t kv_lo,
                                int64_t kv_hi, double* dk, double* dv, double* cq, double* ck,
                                double* cv) {
  if (check_common(T, Hq, Hkv, D, cu, S) != ORC_OK || B < 1 || topk < 1 || !sel || !dout)
    return ORC_EARG;
  if (q_compact && !rows) return ORC_EARG;
  if ((dk == NULL) != (dv == NULL)) return ORC_EARG;
  if ((ck == NULL) != (cv == NULL) || (ck && !dk)) return ORC_EARG;
  if (dk && (kv_lo < 0 || kv_hi > T || kv_lo > kv_hi)) return ORC_EARG;
  if (!rows) nrows = T * Hq;
  int G = Hq / Hkv;
  int64_t nkv = dk ? (kv_hi - kv_lo) * Hkv * D : 0;
  int nacc = ck ? 4 : 2; /* dk, dv (, ck, cv) */
  double* outs[4] = {dk, dv, ck, cv};
  if (dk)
    for (int a = 0; a < nacc; a++) memset(outs[a], 0, sizeof(double) * (size_t)nkv);
  int nthr = 1;
#ifdef _OPENMP
  nthr = omp_get_max_threads();
#endif
  /* private accumulators: priv[th * 4 + a] */
  double** priv = (double**)calloc((size_t)nthr * 4, sizeof(double*));
  if (!priv) return ORC_ENOMEM;
  int fail = 0;
#pragma omp parallel num_threads(nthr)
  {
    int me = 0;
#ifdef _OPENMP
    me = omp_get_thread_num();
#endif
    double* mine[4] = {NULL, NULL, NULL, NULL};
    int ok = 1;
    if (dk)
      for (int a = 0; a < nacc; a++) {
        mine[a] = (double*)calloc((size_t)nkv > 0 ? (size_t)nkv : 1, sizeof(double));
        if (!mine[a]) ok = 0;
      }
    if (!ok) fail = 1;
    for (int a = 0; a < 4; a++) priv[me * 4 + a] = mine[a];
    int64_t cap = 0;
    int64_t* keys = NULL;
    double* z = NULL;
    double* dpv = NULL;
#pragma omp for schedule(dynamic, 16)
    for (int64_t i = 0; i < nrows; i++) {
      if (!ok) continue;
      int64_t r = rows ? rows[i] : i;
      int64_t t = r / Hq;
      int h = (int)(r % Hq);
      int g = h / G;
      int s = seq_of(cu, S, t);
      int64_t L = (int64_t)cu[s + 1] - cu[s];
      int64_t tau = t - cu[s];
      int64_t c = tau / B;
      int64_t need = (int64_t)topk * B;
      if (need > cap) {
        free(keys); free(z); free(dpv);
        cap = need;
        keys = (int64_t*)malloc(sizeof(int64_t) * cap);
        z = (double*)malloc(sizeof(double) * cap);
        dpv = (double*)malloc(sizeof(double) * cap);
        if (!keys || !z || !dpv) {
          fail = 1; cap = 0; free(keys); free(z); free(dpv); keys = NULL; z = NULL; dpv = NULL;
        }
      }
      if (!keys) continue;
      int64_t nk = 0;
      for (int x = 0; x < topk; x++) {
        int64_t j = sel[i * topk + x];
        if (j < 0) continue;
        if (j > c) { fail = 1; continue; } /* future block: never valid */
        int64_t u0 = j * B;
        int64_t u1 = (j == c) ? tau + 1 : ((j + 1) * B < L ? (j + 1) * B : L);
        for (int64_t u = u0; u < u1; u++) keys[nk++] = cu[s] + u;
      }
      int64_t qoff = q_compact ? i * D : (t * Hq + h) * D;
      backward_row(q, k, v, dout, dtype, Hkv, D, qoff, g, keys, nk, z, dpv,
                   dq ? dq + i * D : NULL, kv_lo, kv_hi, mine[0], mine[1],
                   cq ? cq + i * D : NULL, mine[2], mine[3]);
    }
    free(keys);
    free(z);
    free(dpv);
  }
  if (dk && !fail)
    for (int th = 0; th < nthr; th++)
      for (int a = 0; a < nacc; a++) {
        const double* src = priv[th * 4 + a];
        if (!src) continue;
        for (int64_t x = 0; x < nkv; x++) outs[a][x] += src[x];
      }
  for (int x = 0; x < nthr * 4; x++) free(priv[x]);
  free(priv);
  return fail ? ORC_EARG : ORC_OK;
}

/* Dense causal attention (Eq. 1): every key of the query's own sequence up to
 * and including the query. */
int moba_oracle_dense(const void* q, const void* k, const void* v, int dtype, int64_t T,
                      int Hq, int Hkv, int D, const int32_t* cu, int S, const int64_t* rows,
                      int64_t nrows, double* out, double* lse) {
  if (check_common(T, Hq, Hkv, D, cu, S) != ORC_OK || !out || !lse) return ORC_EARG;
  if (!rows) nrows = T * Hq;
  int G = Hq / Hkv;
  int fail = 0;
#pragma omp parallel
  {
    int64_t cap = 0;
    int64_t* keys = NULL;
    double* z = NULL;
#pragma omp for schedule(dynamic, 16)
    for (int64_t i = 0; i < nrows; i++) {
      int64_t r = rows ? rows[i] : i;
      int64_t t = r / Hq;
      int h = (int)(r % Hq);
      int s = seq_of(cu, S, t);
      int64_t nk = t - cu[s] + 1;
      if (nk > cap) {
        free(keys); free(z);
        cap = nk;
        keys = (int64_t*)malloc(sizeof(int64_t) * cap);
        z = (double*)malloc(sizeof(double) * cap);
        if (!keys || !z) { fail = 1; cap = 0; free(keys); free(z); keys = NULL; z = NULL; }
      }
      if (!keys) continue;
      for (int64_t x = 0; x < nk; x++) keys[x] = cu[s] + x;
      attend_keys(q, k, v, dtype, Hkv, D, (t * Hq + h) * D, h / G, keys, nk, z, out + i * D,
                  lse + i);
    }
    free(keys);
    free(z);
  }
  return fail ? ORC_ENOMEM : ORC_OK;
}

int moba_oracle_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

void moba_oracle_set_threads(int n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
#else
  (void)n;
#endif
}
