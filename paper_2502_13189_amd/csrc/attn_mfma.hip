// bf16 attention on the gfx950 matrix cores: the history-block attention,
// the causal current-block attention (Algorithm 1, the two
// flash_attention_varlen calls; Sec. 2.2 "Current Block Attention") and dense
// causal attention (Eq. 1), from one kernel template.
//
// Work-group = 4 waves = 128 query rows; wave w owns rows 32w..32w+31, one
// query per lane column.  Keys are consumed in tiles of 64 through a
// double-buffered LDS stage: K as 64 rows of 256 B and V^T as 128 rows of
// 128 B, each row padded by 16 B so that the MFMA operand reads (eight lanes
// on eight consecutive rows at one column) fall on distinct banks, and every
// read address is a per-lane base plus an immediate offset.
//
// Per key tile and wave, on v_mfma_f32_32x32x16_bf16:
//   S^T (keys x queries) = K_tile . Q^T      2 x 8 MFMAs, K from LDS, Q^T in registers
//   online softmax in fp32 on S^T: every lane holds one query and 32 of the
//   tile's 64 keys, so the row max needs one exchange with the partner lane
//   (lane ^ 32) and the row sum is kept per lane and combined at the end.
//   The running max is only raised when a tile's max exceeds it by more than
//   2^8 (in exp2 units): the weights then stay below 2^8, and the accumulator
//   rescale, a multiply of all 64 accumulators, is skipped on most tiles.
//   The row sum adds the fp32 weights, so lse is as accurate as fp32 allows.
//   O^T (dims x queries) += V^T_tile . P^T  4 x 4 MFMAs, P^T straight from the
//   softmax registers (converted to bf16), V^T from LDS
// The accumulator layout of a 32x32 MFMA gives lane l the column l % 32 and
// rows 8*(i/4) + 4*(l/32) + i%4 for its 16 values i; so the 8 keys a lane
// feeds into one k=16 step are keys {0-3, 8-11} (+4 for the upper half-wave)
// of a 16-key group, which is the order the V^T pack stores them in.
//
// Logits use scale 1/sqrt(D), folded with log2(e) into one FMA before exp2.
// Outputs: history tiles write normalised fp32 partials and their natural-log
// lse; current-block tiles merge those partials into the final output (the
// log-sum-exp combine of Algorithm 1); dense tiles write the final output.
#include "moba_internal.h"

#include <math.h>

namespace moba {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));  // one 16-byte chunk

enum { kHist = 0, kCur = 1, kDense = 2 };

constexpr int kChunksV = kHeadDim * kKeyTile / 8;  // per V^T tile (1024)
constexpr int kRowK = kHeadDim / 8 + 1;            // LDS K row: 16 chunks + 1 pad
constexpr int kRowV = kKeyTile / 8 + 1;            // LDS V^T row: 8 chunks + 1 pad
constexpr int kStageK = kKeyTile * kRowK;          // chunks of one K stage
constexpr int kStageChunks = kStageK + kHeadDim * kRowV;
constexpr float kRescaleSlack = 8.0f;              // exp2 units

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 u) { return __builtin_bit_cast(bf16x8, u); }

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Two fp32 values to a packed bf16 pair, round-to-nearest-even.
__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  const f32x2 v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}


__device__ __forceinline__ float xor32(float v) { return __shfl_xor(v, 32, 64); }

// Global -> registers: this thread's four 16-byte chunks of K tile i (64 keys
// x 256 B) and of the packed V^T tile i (contiguous 16 KiB).
__device__ __forceinline__ void load_tile(int i, int tid, const __hip_bfloat16* kbase, int64_t k_st,
                                          int64_t tok0, int64_t seq_end, const u32x4* vtbase,
                                          u32x4 (&kreg)[4], u32x4 (&vreg)[4]) {
#pragma unroll
  for (int x = 0; x < 4; x++) {
    const int c = tid + 256 * x;
    const int r = c >> 4, col = c & 15;
    // rows past the sequence end repeat its last key; they are always masked
    const int64_t u = min(tok0 + (int64_t)i * kKeyTile + r, seq_end - 1);
    kreg[x] = *reinterpret_cast<const u32x4*>(kbase + u * k_st + col * 8);
    vreg[x] = vtbase[(int64_t)i * kChunksV + c];
  }
}

// Registers -> one LDS stage (padded rows).
__device__ __forceinline__ void store_tile(u32x4* kl, int tid, const u32x4 (&kreg)[4],
                                           const u32x4 (&vreg)[4]) {
  u32x4* vl = kl + kStageK;
#pragma unroll
  for (int x = 0; x < 4; x++) {
    const int c = tid + 256 * x;
    kl[(c >> 4) * kRowK + (c & 15)] = kreg[x];
    vl[(c >> 3) * kRowV + (c & 7)] = vreg[x];
  }
}

struct RowInfo {
  int64_t t;
  int h;
  bool valid;
  int64_t dst;  // partial index (history / current) or unused (dense)
};

template <int MODE>
__global__ __launch_bounds__(256, 2) void attn_mfma_kernel(AttnArgs a, Problem p) {
  __shared__ u32x4 lds[2 * kStageChunks];  // 70 KiB
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int qc = lane & 31, hh = lane >> 5;
  const int rloc = wave * 32 + qc;  // this lane's query row within the tile

  // ------------------------------------------------------------ tile setup
  int g, s;
  int64_t kbeg, kend, tmin;
  RowInfo ri;
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
    int64_t lo = a.g0 * nb, hi = a.g1 * nb - 1;
    while (lo < hi) {
      const int64_t mid = (lo + hi + 1) >> 1;
      if (a.bin_tile_start[mid] <= tile) lo = mid; else hi = mid - 1;
    }
    const int64_t bin = lo;
    g = (int)(bin / nb);
    const int b = (int)(bin % nb);
    const int64_t e0 = a.bin_start[bin] + (tile - a.bin_tile_start[bin]) * kTileRows;
    const int n = (int)min((int64_t)kTileRows, a.bin_start[bin] + a.bin_count[bin] - e0);
    s = find_seq(a.seqs, p.S, b, [](const SeqInfo& x) { return x.blk_off; });
    const SeqInfo sq = a.seqs[s];
    kbeg = (int64_t)sq.tok_start + (int64_t)(b - sq.blk_off) * p.B;
    kend = kbeg + p.B;
    tmin = kend;  // every key precedes every routed query
    const uint32_t kh = (uint32_t)(p.topk - 1);
    const uint64_t ev = a.entries[e0 + min(rloc, n - 1)];
    const uint64_t gr = ev / kh;
    const uint64_t TG = (uint64_t)p.T * p.G;
    const uint64_t rem = gr - (uint64_t)g * TG;
    ri.t = (int64_t)(rem / p.G);
    ri.h = g * p.G + (int)(rem % p.G);
    ri.dst = (int64_t)(ev - (uint64_t)a.g0 * TG * kh);
    ri.valid = rloc < n && rem < TG;
    if (!(rem < TG)) { ri.t = kbeg; ri.h = g * p.G; }
  } else {
    const CausalTile ct = a.tiles[blockIdx.x];
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
  const SeqInfo sq = a.seqs[s];
  const int64_t seq_end = (int64_t)sq.tok_start + sq.len;

  // ---------------------------------------------------------- Q^T operand
  const __hip_bfloat16* qbase = static_cast<const __hip_bfloat16*>(a.q);
  const __hip_bfloat16* qrow = qbase + ri.t * a.q_st + (int64_t)ri.h * a.q_sh + 8 * hh;
  bf16x8 qf[8];
#pragma unroll
  for (int kk = 0; kk < 8; kk++) qf[kk] = as_bf16x8(*reinterpret_cast<const u32x4*>(qrow + 16 * kk));

  // ------------------------------------------------------------ key tiles
  const int64_t rb = kbeg - sq.tok_start, re = kend - sq.tok_start;
  const int i0 = (int)(rb / kKeyTile), i1 = (int)((re + kKeyTile - 1) / kKeyTile);
  const __hip_bfloat16* kbase = static_cast<const __hip_bfloat16*>(a.k) + (int64_t)g * a.k_sh;
  const u32x4* vtbase = reinterpret_cast<const u32x4*>(
      a.vt + ((int64_t)g * p.vt_tiles + sq.vt_tile_off) * (kKeyTile * kHeadDim));

  const int64_t tok0 = sq.tok_start;
  const int64_t kst = a.k_st;
  u32x4 kreg[4], vreg[4];

  const float c2 = a.scale_log2;
  float m_run = -INFINITY, l_run = 0.0f;
  f32x16 o[4];
#pragma unroll
  for (int dt = 0; dt < 4; dt++)
#pragma unroll
    for (int r = 0; r < 16; r++) o[dt][r] = 0.0f;

  load_tile(i0, tid, kbase, kst, tok0, seq_end, vtbase, kreg, vreg);
  store_tile(lds, tid, kreg, vreg);
  // Let every load of the prologue (Q included) land here: otherwise the
  // loop would carry waits on Q that, in steady state, stall on the prefetch.
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  for (int i = i0; i < i1; i++) {
    const int stage = (i - i0) & 1;
    if (i + 1 < i1) load_tile(i + 1, tid, kbase, kst, tok0, seq_end, vtbase, kreg, vreg);
    const u32x4* kl = lds + stage * kStageChunks + qc * kRowK + hh;
    const u32x4* vl = lds + stage * kStageChunks + kStageK + qc * kRowV + hh;

    // S^T = K . Q^T
    f32x16 sacc[2];
#pragma unroll
    for (int th = 0; th < 2; th++)
#pragma unroll
      for (int r = 0; r < 16; r++) sacc[th][r] = 0.0f;
#pragma unroll
    for (int kk = 0; kk < 8; kk++) {
#pragma unroll
      for (int th = 0; th < 2; th++) {
        const bf16x8 ka = as_bf16x8(kl[32 * th * kRowK + 2 * kk]);
        sacc[th] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[kk], sacc[th], 0, 0, 0);
      }
    }

    // mask keys outside [kbeg, kend) and, on causal tiles, keys after the query
    const int64_t u0 = (int64_t)sq.tok_start + (int64_t)i * kKeyTile;
    const bool edge = u0 < kbeg || u0 + kKeyTile > kend || (MODE != kHist && u0 + kKeyTile - 1 > tmin);
    if (edge) {
#pragma unroll
      for (int th = 0; th < 2; th++)
#pragma unroll
        for (int r = 0; r < 16; r++) {
          const int64_t u = u0 + 32 * th + 8 * (r >> 2) + 4 * hh + (r & 3);
          const bool ok = u >= kbeg && u < kend && (MODE == kHist || u <= ri.t);
          sacc[th][r] = ok ? sacc[th][r] : -INFINITY;
        }
    }

    // online softmax (exp2 units), lazily rescaled
    float mx = -INFINITY;
#pragma unroll
    for (int th = 0; th < 2; th++)
#pragma unroll
      for (int r = 0; r < 16; r++) mx = fmaxf(mx, sacc[th][r]);
    mx = fmaxf(mx, xor32(mx)) * c2;
    if (__builtin_amdgcn_ballot_w64(mx > m_run + kRescaleSlack) != 0) {
      const float m_new = fmaxf(m_run, mx);
      const float alpha = m_new == -INFINITY ? 1.0f : __builtin_amdgcn_exp2f(m_run - m_new);
      l_run *= alpha;
#pragma unroll
      for (int dt = 0; dt < 4; dt++)
#pragma unroll
        for (int r = 0; r < 16; r++) o[dt][r] *= alpha;
      m_run = m_new;
    }
    const float m_use = m_run == -INFINITY ? 0.0f : m_run;

    // weights, row sums, P^T in bf16, O^T += V^T . P^T
#pragma unroll
    for (int th = 0; th < 2; th++) {
#pragma unroll
      for (int s2 = 0; s2 < 2; s2++) {
        uint32_t w[4];
#pragma unroll
        for (int e = 0; e < 4; e++) {
          const float p0 = __builtin_amdgcn_exp2f(fmaf(sacc[th][8 * s2 + 2 * e], c2, -m_use));
          const float p1 = __builtin_amdgcn_exp2f(fmaf(sacc[th][8 * s2 + 2 * e + 1], c2, -m_use));
          w[e] = pack_bf16(p0, p1);
          l_run += p0 + p1;
        }
        const bf16x8 pb = as_bf16x8(u32x4{w[0], w[1], w[2], w[3]});
#pragma unroll
        for (int dt = 0; dt < 4; dt++) {
          const bf16x8 va = as_bf16x8(vl[32 * dt * kRowV + 4 * th + 2 * s2]);
          o[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb, o[dt], 0, 0, 0);
        }
      }
    }

    if (i + 1 < i1) store_tile(lds + (stage ^ 1) * kStageChunks, tid, kreg, vreg);
    __syncthreads();
  }

  // -------------------------------------------------------------- epilogue
  const float l_tot = l_run + xor32(l_run);
  const float inv = 1.0f / l_tot;
  const float lse = (m_run + __builtin_amdgcn_logf(l_tot)) * 0.69314718055994531f;
  if constexpr (MODE == kHist) {
    if (!ri.valid) return;
    float* orow = a.o_part + ri.dst * kHeadDim;
#pragma unroll
    for (int dt = 0; dt < 4; dt++)
#pragma unroll
      for (int r4 = 0; r4 < 4; r4++) {
        const int d = 32 * dt + 8 * r4 + 4 * hh;
        *reinterpret_cast<float4*>(orow + d) =
            make_float4(o[dt][4 * r4 + 0] * inv, o[dt][4 * r4 + 1] * inv, o[dt][4 * r4 + 2] * inv,
                        o[dt][4 * r4 + 3] * inv);
      }
    if (hh == 0) a.lse_part[ri.dst] = lse;
  } else {
    float scale = inv, lse_out = lse;
    if constexpr (MODE == kCur) {
      // Merge with the row's history partials (all rows of a tile share the
      // current block c, so the slot count is uniform):
      //   lse = M + ln(sum_i e^{lse_i - M}),  out = sum_i e^{lse_i - lse} O_i
      // summed in a fixed order: current block first, then slots ascending.
      const int kh = p.topk - 1;
      const int nh = min(kh, (int)((tmin - sq.tok_start) / p.B));
      if (nh > 0) {
        const float* lp = a.lse_part + ri.dst * kh;
        const float* op = a.o_part + ri.dst * kh * kHeadDim;
        float M = lse;
        for (int x = 0; x < nh; x++) M = fmaxf(M, lp[x]);
        constexpr float kLog2e = 1.4426950408889634f;
        const float wc = __builtin_amdgcn_exp2f((lse - M) * kLog2e);
        float wsum = wc;
#pragma unroll
        for (int dt = 0; dt < 4; dt++)
#pragma unroll
          for (int r = 0; r < 16; r++) o[dt][r] *= wc * inv;
        for (int x = 0; x < nh; x++) {
          const float w = __builtin_amdgcn_exp2f((lp[x] - M) * kLog2e);
          wsum += w;
          const float* ox = op + x * kHeadDim;
#pragma unroll
          for (int dt = 0; dt < 4; dt++)
#pragma unroll
            for (int r4 = 0; r4 < 4; r4++) {
              const float4 v = *reinterpret_cast<const float4*>(ox + 32 * dt + 8 * r4 + 4 * hh);
              o[dt][4 * r4 + 0] = fmaf(w, v.x, o[dt][4 * r4 + 0]);
              o[dt][4 * r4 + 1] = fmaf(w, v.y, o[dt][4 * r4 + 1]);
              o[dt][4 * r4 + 2] = fmaf(w, v.z, o[dt][4 * r4 + 2]);
              o[dt][4 * r4 + 3] = fmaf(w, v.w, o[dt][4 * r4 + 3]);
            }
        }
        scale = 1.0f / wsum;
        lse_out = M + __builtin_amdgcn_logf(wsum) * 0.69314718055994531f;
      }
    }
    if (!ri.valid) return;
    __hip_bfloat16* orow = static_cast<__hip_bfloat16*>(a.out) + ri.t * a.o_st + (int64_t)ri.h * a.o_sh;
#pragma unroll
    for (int dt = 0; dt < 4; dt++)
#pragma unroll
      for (int r4 = 0; r4 < 4; r4++) {
        const int d = 32 * dt + 8 * r4 + 4 * hh;
        uint2 w;
        w.x = pack_bf16(o[dt][4 * r4 + 0] * scale, o[dt][4 * r4 + 1] * scale);
        w.y = pack_bf16(o[dt][4 * r4 + 2] * scale, o[dt][4 * r4 + 3] * scale);
        *reinterpret_cast<uint2*>(orow + d) = w;
      }
    if (hh == 0) a.lse[(int64_t)ri.h * p.T + ri.t] = lse_out;
  }
}

}  // namespace

hipError_t launch_attn_hist_bf16(const AttnArgs& a, const Problem& p, int64_t grid, hipStream_t st) {
  if (grid <= 0) return hipSuccess;
  grid = (grid + 7) / 8 * 8;
  attn_mfma_kernel<kHist><<<(unsigned)grid, 256, 0, st>>>(a, p);
  return hipGetLastError();
}

hipError_t launch_attn_causal_bf16(bool dense, const AttnArgs& a, const Problem& p, hipStream_t st) {
  if (a.ntiles <= 0 || a.g1 <= a.g0) return hipSuccess;
  dim3 grid((unsigned)a.ntiles, a.g1 - a.g0);
  if (dense) attn_mfma_kernel<kDense><<<grid, 256, 0, st>>>(a, p);
  else attn_mfma_kernel<kCur><<<grid, 256, 0, st>>>(a, p);
  return hipGetLastError();
}

}  // namespace moba
