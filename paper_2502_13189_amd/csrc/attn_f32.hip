// fp32 attention on the vector ALUs, for fp32 inputs (the tolerance of an
// fp32 problem rules out bf16 matrix-core products).  Same tiles, rows and
// outputs as the bf16 MFMA kernel: history-block tiles (partials),
// causal current-block tiles (merged with the partials into the output) and
// dense causal tiles.
//
// Work-group = 128 threads, one query row per thread, with the query and the
// output accumulator in registers (2 x 128 fp32).  Keys arrive in tiles of 32
// rows of K and V staged in LDS; all lanes read the same key row (an LDS
// broadcast).  Per tile: 32 scaled logits, one max, one rescale of the
// accumulator, then 32 exp2 weights folded into the accumulator.
#include "moba_internal.h"

#include <math.h>

namespace moba {
namespace {

enum { kHist = 0, kCur = 1, kDense = 2 };
constexpr int kT = 32;  // keys per tile

template <int MODE>
__global__ __launch_bounds__(128, 1) void attn_f32_kernel(AttnArgs a, Problem p) {
  __shared__ float4 ks[kT][kHeadDim / 4];
  __shared__ float4 vs[kT][kHeadDim / 4];
  const int rloc = threadIdx.x;
  int g, s;
  int64_t kbeg, kend, t, dst;
  int h;
  bool valid;
  if constexpr (MODE == kHist) {
    const int64_t nb = p.nblk_total;
    const int64_t tbeg = a.bin_tile_start[a.g0 * nb];
    const int64_t tend = a.bin_tile_start[a.g1 * nb];
    const int64_t tile = tbeg + blockIdx.x;
    if (tile >= tend) return;
    const int64_t bin = a.tile_bin[tile];
    g = (int)(bin / nb);
    const int b = (int)(bin % nb);
    const int64_t e0 = a.bin_start[bin] + (tile - a.bin_tile_start[bin]) * kTileRowsF32;
    const int n = (int)min((int64_t)kTileRowsF32, a.bin_start[bin] + a.bin_count[bin] - e0);
    s = find_seq(a.seqs, p.S, b, [](const SeqInfo& x) { return x.blk_off; });
    const SeqInfo sq = a.seqs[s];
    kbeg = (int64_t)sq.tok_start + (int64_t)(b - sq.blk_off) * p.B;
    kend = kbeg + p.B;
    const uint64_t kh = (uint64_t)(p.topk - 1);
    const uint64_t ev = a.entries[e0 + min(rloc, n - 1)];
    const uint64_t TG = (uint64_t)p.T * p.G;
    const uint64_t rem = ev / kh - (uint64_t)g * TG;
    valid = rloc < n && rem < TG;
    t = valid ? (int64_t)(rem / p.G) : kbeg;
    h = g * p.G + (valid ? (int)(rem % p.G) : 0);
    dst = (int64_t)(ev - (uint64_t)a.g0 * TG * kh);
  } else {
    const CausalTile ct = a.tiles[blockIdx.x];
    if (ct.t1 <= ct.t0) return;  // padding of the tile list
    g = a.g0 + blockIdx.y;
    s = ct.s;
    kbeg = ct.kbeg;
    kend = ct.t1;
    const int nrow = (ct.t1 - ct.t0) * p.G;
    valid = rloc < nrow;
    const int rr = valid ? rloc : 0;
    t = ct.t0 + rr / p.G;
    h = g * p.G + rr % p.G;
    dst = (int64_t)(g - a.g0) * p.T * p.G + t * p.G + (rr % p.G);
  }
  const SeqInfo sq = a.seqs[s];
  const int64_t seq_end = (int64_t)sq.tok_start + sq.len;

  float qf[kHeadDim], of[kHeadDim];
  const float4* qrow = reinterpret_cast<const float4*>(static_cast<const float*>(a.q) + t * a.q_st +
                                                       (int64_t)h * a.q_sh);
#pragma unroll
  for (int c = 0; c < kHeadDim / 4; c++) {
    const float4 x = qrow[c];
    qf[4 * c] = x.x; qf[4 * c + 1] = x.y; qf[4 * c + 2] = x.z; qf[4 * c + 3] = x.w;
    of[4 * c] = of[4 * c + 1] = of[4 * c + 2] = of[4 * c + 3] = 0.0f;
  }
  const float c2 = a.scale_log2;
  float m_run = -INFINITY, l_run = 0.0f;
  const float* kb = static_cast<const float*>(a.k) + (int64_t)g * a.k_sh;
  const float* vb = static_cast<const float*>(a.v) + (int64_t)g * a.v_sh;
  const int64_t rb = kbeg - sq.tok_start, re = kend - sq.tok_start;
  const int i0 = (int)(rb / kT), i1 = (int)((re + kT - 1) / kT);
  for (int i = i0; i < i1; i++) {
    const int64_t u0 = (int64_t)sq.tok_start + (int64_t)i * kT;
    __syncthreads();
    for (int x = threadIdx.x; x < kT * (kHeadDim / 4); x += 128) {
      const int r = x / (kHeadDim / 4), c4 = x % (kHeadDim / 4);
      const int64_t u = u0 + r;
      float4 kv = make_float4(0.f, 0.f, 0.f, 0.f), vv = kv;
      if (u < seq_end) {
        kv = reinterpret_cast<const float4*>(kb + u * a.k_st)[c4];
        vv = reinterpret_cast<const float4*>(vb + u * a.v_st)[c4];
      }
      ks[r][c4] = kv;
      vs[r][c4] = vv;
    }
    __syncthreads();
    float z[kT];
    float mx = -INFINITY;
#pragma unroll
    for (int r = 0; r < kT; r++) {
      float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
#pragma unroll
      for (int c4 = 0; c4 < kHeadDim / 4; c4++) {
        const float4 kv = ks[r][c4];
        a0 = fmaf(qf[4 * c4], kv.x, a0);
        a1 = fmaf(qf[4 * c4 + 1], kv.y, a1);
        a2 = fmaf(qf[4 * c4 + 2], kv.z, a2);
        a3 = fmaf(qf[4 * c4 + 3], kv.w, a3);
      }
      const int64_t u = u0 + r;
      const bool ok = u >= kbeg && u < kend && (MODE == kHist || u <= t);
      z[r] = ok ? ((a0 + a1) + (a2 + a3)) * c2 : -INFINITY;
      mx = fmaxf(mx, z[r]);
    }
    const float m_new = fmaxf(m_run, mx);
    const float m_use = m_new == -INFINITY ? 0.0f : m_new;
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
    l_run *= alpha;
#pragma unroll
    for (int d = 0; d < kHeadDim; d++) of[d] *= alpha;
#pragma unroll
    for (int r = 0; r < kT; r++) {
      const float pw = __builtin_amdgcn_exp2f(z[r] - m_use);
      l_run += pw;
#pragma unroll
      for (int c4 = 0; c4 < kHeadDim / 4; c4++) {
        const float4 vv = vs[r][c4];
        of[4 * c4] = fmaf(pw, vv.x, of[4 * c4]);
        of[4 * c4 + 1] = fmaf(pw, vv.y, of[4 * c4 + 1]);
        of[4 * c4 + 2] = fmaf(pw, vv.z, of[4 * c4 + 2]);
        of[4 * c4 + 3] = fmaf(pw, vv.w, of[4 * c4 + 3]);
      }
    }
    m_run = m_new;
  }
  float inv = 1.0f / l_run;
  float lse = (m_run + __builtin_amdgcn_logf(l_run)) * 0.69314718055994531f;
  if constexpr (MODE == kHist) {
    if (!valid) return;
    float* orow = static_cast<float*>(a.o_part) + dst * kHeadDim;
    a.lse_part[dst] = lse;
#pragma unroll
    for (int c = 0; c < kHeadDim / 4; c++)
      reinterpret_cast<float4*>(orow)[c] =
          make_float4(of[4 * c] * inv, of[4 * c + 1] * inv, of[4 * c + 2] * inv, of[4 * c + 3] * inv);
    return;
  }
  if constexpr (MODE == kCur) {
    // merge with the row's history partials (same order and formula as the
    // bf16 kernel: current block first, then slots ascending)
    const int kh = p.topk - 1;
    const int nh = min(kh, (int)((kbeg - sq.tok_start) / p.B));
    if (nh > 0) {
      const float* lp = a.lse_part + dst * kh;
      const float* op = static_cast<const float*>(a.o_part) + dst * kh * kHeadDim;
      float M = lse;
      for (int x = 0; x < nh; x++) M = fmaxf(M, lp[x]);
      constexpr float kLog2e = 1.4426950408889634f;
      const float wc = __builtin_amdgcn_exp2f((lse - M) * kLog2e);
      float wsum = wc;
#pragma unroll
      for (int d = 0; d < kHeadDim; d++) of[d] *= wc * inv;
      for (int x = 0; x < nh; x++) {
        const float w = __builtin_amdgcn_exp2f((lp[x] - M) * kLog2e);
        wsum += w;
        const float4* ox = reinterpret_cast<const float4*>(op + x * kHeadDim);
#pragma unroll
        for (int c = 0; c < kHeadDim / 4; c++) {
          const float4 v = ox[c];
          of[4 * c] = fmaf(w, v.x, of[4 * c]);
          of[4 * c + 1] = fmaf(w, v.y, of[4 * c + 1]);
          of[4 * c + 2] = fmaf(w, v.z, of[4 * c + 2]);
          of[4 * c + 3] = fmaf(w, v.w, of[4 * c + 3]);
        }
      }
      inv = 1.0f / wsum;
      lse = M + __builtin_amdgcn_logf(wsum) * 0.69314718055994531f;
    }
  }
  if (!valid) return;
  float* orow = static_cast<float*>(a.out) + t * a.o_st + (int64_t)h * a.o_sh;
  a.lse[(int64_t)h * p.T + t] = lse;
#pragma unroll
  for (int c = 0; c < kHeadDim / 4; c++)
    reinterpret_cast<float4*>(orow)[c] =
        make_float4(of[4 * c] * inv, of[4 * c + 1] * inv, of[4 * c + 2] * inv, of[4 * c + 3] * inv);
}

}  // namespace

hipError_t launch_attn_hist_f32(const AttnArgs& a, const Problem& p, int64_t grid, hipStream_t st) {
  if (grid <= 0) return hipSuccess;
  attn_f32_kernel<kHist><<<(unsigned)grid, 128, 0, st>>>(a, p);
  return hipGetLastError();
}

hipError_t launch_attn_causal_f32(bool dense, const AttnArgs& a, const Problem& p, hipStream_t st) {
  if (a.ntiles <= 0 || a.g1 <= a.g0) return hipSuccess;
  dim3 grid((unsigned)a.ntiles, a.g1 - a.g0);
  if (dense) attn_f32_kernel<kDense><<<grid, 128, 0, st>>>(a, p);
  else attn_f32_kernel<kCur><<<grid, 128, 0, st>>>(a, p);
  return hipGetLastError();
}

}  // namespace moba
