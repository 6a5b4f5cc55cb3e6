// Backward of MoBA attention on the gfx950 matrix cores: the gradients w.r.t.
// q, k and v for the selection the forward made.  The gate is a hard 0/1
// choice (Eq. 3 and Eq. 5) and passes no gradient, so this is the chain rule
// through Eq. 2 over the key set of Eq. 4.  With the forward's lse per row
// and Delta = <dO, O> per row (O the forward's output):
//   P = exp(z - lse), z = <q, k> / sqrt(D);   dP = <dO, v>;   dS = P (dP - Delta)
//   dQ = sum over keys of dS k / sqrt(D)
//   dK = sum over rows of dS q / sqrt(D),     dV = sum over rows of P dO
//
// Kernels, in launch order:
//   delta  LD[h, t] = (lse * log2 e, Delta), 16 lanes per row.
//   rec    (t, h, LD[h, t]) of every routed history entry, in routing order,
//          so that the key-side kernel gets a row's facts with one load.
//   dq     query side, on the forward's tiles.  A history tile (256 routed
//          rows of one (kv-head, block) bin) loops over the block's 64-key
//          tiles and writes each row's dQ for that selection slot in fp32; a
//          current-block tile covers the causal keys of its block, adds the
//          row's history partials in slot order and writes dQ.  Per key
//          tile and wave: S^T = K . Q^T and dP^T = V . dO^T (K and V
//          row-major from LDS, Q^T and dO^T operands in registers), then
//          dQ^T += K^T . dS^T from the packed K^T tile: 48 MFMAs.
//   dkdv   key side: a work-group of 8 waves owns 128 keys of one block and
//          kv-head, 32 per SIMD, and loops over every row that attends them,
//          64 rows at a time: the bin's routed history rows, then the
//          block's own rows (causal).  The rows' Q and dO arrive by LDS DMA,
//          gathered row by row, into a swizzled row-major layout that also
//          serves the transposed operands (ds_read_b64_tr_b16).  The two
//          waves of a SIMD split the work for their 32 keys: per 32-row
//          subtile the P-wave forms S = Q . K^T, P and dV^T += dO^T . P, the
//          D-wave dP = dO . V^T, dS (with P from LDS) and dK^T += Q^T . dS:
//          16 MFMAs each; the D-wave's dK product of a subtile runs one
//          subtile late, beside the P-wave's exponentials of the next.  Each
//          key has one owner, so dK and dV need neither atomics nor a merge.
// P and dS enter the second products as bf16; every product accumulates in
// fp32.  The key side forms dS from the bf16 P its dV product uses (the value
// it receives from the pair's P-wave); the query side from its fp32 P.
#include "bwd_internal.h"
#include "mfma_tile.h"

#include <limits.h>
#include <math.h>

namespace moba {
namespace {

enum { kHist = 0, kCur = 1 };

constexpr int kRows = kTileRowsMfma;  // query rows per dQ work-group (256)
constexpr float kLog2e = 1.4426950408889634f;

// Per-lane DMA sources of one 64-key tile set: lane chunk p = 64j + L of DMA
// instruction j holds row p / 17, chunk min(p % 17, 15) of a row-major tile
// and row p / 9, chunk min(p % 9, 7) of a packed tile.
__device__ __forceinline__ void init_dma(Dma& D, int wave, int lane, const char* base, int64_t st_bytes,
                                         int64_t len, const char* packed) {
  D.wave = wave;
  D.kbase = base;
  D.k_tile = kKeyTile * st_bytes;
  D.len = len;
  D.klast = base + (len - 1) * st_bytes;
#pragma unroll
  for (int x = 0; x < 3; x++) {
    const int pk = 64 * (wave + 8 * x) + lane;
    const int row = min(pk / kRowK, kKeyTile - 1), c = min(pk % kRowK, kRowK - 2);
    D.krow[x] = row;
    D.kcol[x] = (uint32_t)(c * 16);
    D.koff[x] = (uint32_t)(row * st_bytes) + D.kcol[x];
    const int vrow = min(pk / kRowV, kHeadDim - 1), vc = min(pk % kRowV, kRowV - 2);
    D.voff[x] = (uint32_t)(vrow * (kKeyTile * 2) + vc * 16);
  }
  D.vbase = packed;
}

// ============================================================ delta, rec
__global__ __launch_bounds__(256) void bwd_delta_kernel(BwdArgs a, Problem p) {
  const int64_t r = (int64_t)blockIdx.x * 16 + threadIdx.x / 16;  // r = t * Hq + h
  const int l16 = threadIdx.x % 16;
  if (r >= p.T * p.Hq) return;  // the 16 lanes of a row leave together
  const int64_t t = r / p.Hq;
  const int h = (int)(r % p.Hq);
  const uint4 ou = *reinterpret_cast<const uint4*>(static_cast<const __hip_bfloat16*>(a.o) +
                                                   t * a.o_st + (int64_t)h * a.o_sh + 8 * l16);
  const uint4 du = *reinterpret_cast<const uint4*>(static_cast<const __hip_bfloat16*>(a.dout) +
                                                   t * a.do_st + (int64_t)h * a.do_sh + 8 * l16);
  const uint32_t ow[4] = {ou.x, ou.y, ou.z, ou.w}, dw[4] = {du.x, du.y, du.z, du.w};
  float acc = 0.0f;
#pragma unroll
  for (int i = 0; i < 4; i++) {
    acc = fmaf(__uint_as_float(ow[i] << 16), __uint_as_float(dw[i] << 16), acc);
    acc = fmaf(__uint_as_float(ow[i] & 0xffff0000u), __uint_as_float(dw[i] & 0xffff0000u), acc);
  }
#pragma unroll
  for (int m = 8; m >= 1; m >>= 1) acc += __shfl_xor(acc, m, 64);
  if (l16 == 0) {
    const int64_t i = (int64_t)h * p.T + t;
    a.ld[i] = make_float2(a.lse[i] * kLog2e, acc);
  }
}

__global__ __launch_bounds__(256) void bwd_rec_kernel(BwdArgs a, Problem p) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e >= p.hist_entries) return;
  const uint64_t kh = (uint64_t)(p.topk - 1);
  const uint64_t TG = (uint64_t)p.T * p.G;
  const uint64_t r = (uint64_t)a.entries[e] / kh;
  const int g = (int)(r / TG);
  const uint64_t rem = r - (uint64_t)g * TG;
  const int64_t t = (int64_t)(rem / p.G);
  const int h = g * p.G + (int)(rem % p.G);
  const float2 ld = a.ld[(int64_t)h * p.T + t];
  a.rec[e] = make_int4((int)t, h, __float_as_int(ld.x), __float_as_int(ld.y));
}

// ================================================================ dQ
// S^T and dP^T of keys 32*th .. 32*th+31 of a 64-key tile: 8 k-steps each
// from the row-major K and V buffers, the two accumulation chains
// interleaved, operand reads kPre MFMAs ahead.
__device__ __forceinline__ void sdp_half(f32x16& s, f32x16& dp, const u32x4* kb, const u32x4* vb,
                                         const ReadOff& ro, int th, const bf16x8 (&qf)[8],
                                         const bf16x8 (&df)[8]) {
#pragma unroll
  for (int r = 0; r < 16; r++) {
    s[r] = 0.0f;
    dp[r] = 0.0f;
  }
  const u32x4* k = kb + ro.kq + 32 * kRowK * th;
  const u32x4* v = vb + ro.kq + 32 * kRowK * th;
  u32x4 op[16];
#pragma unroll
  for (int j = 0; j < 16; j++) op[j] = (j & 1) ? v[2 * (j >> 1)] : k[2 * (j >> 1)];
#pragma unroll
  for (int j = 0; j < 16; j++) {
    if (j & 1) dp = mfma(as_bf16x8(op[j]), df[j >> 1], dp);
    else s = mfma(as_bf16x8(op[j]), qf[j >> 1], s);
  }
  pin_pipeline();
}

// dS^T = P^T (dP^T - Delta), P^T = exp2(S^T c2 - lse2), for keys 32*th ..
// 32*th+31 of the tile, as the bf16 operands db[2*th + s2] (keys 32*th +
// 16*s2 .. +15, the key order of the packed K^T tile).  On edge tiles only
// keys lo <= k < hi (relative to this lane's key offset 4*hh) are kept.
__device__ __forceinline__ void grad_half(const f32x16& s, const f32x16& dp, bf16x8 (&db)[4], int th,
                                          bool edge, int lo, int hi, float c2, float lse2,
                                          float dlt) {
#pragma unroll
  for (int s2 = 0; s2 < 2; s2++) {
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 4; e++) {
      float d[2];
#pragma unroll
      for (int u = 0; u < 2; u++) {
        const int i = 8 * s2 + 2 * e + u;
        const int kk = 32 * th + 8 * (i >> 2) + (i & 3);
        float p = __builtin_amdgcn_exp2f(fmaf(s[i], c2, -lse2));
        if (edge) p = (kk >= lo && kk < hi) ? p : 0.0f;
        d[u] = p * (dp[i] - dlt);
      }
      w[e] = pack_bf16(d[0], d[1]);
    }
    db[2 * th + s2] = as_bf16x8(u32x4{w[0], w[1], w[2], w[3]});
  }
}

// Row-major V tiles for the DMA: the wave-uniform part; the per-lane
// offsets are recomputed from K's rows and columns (V may have its own
// token stride).
struct VDma {
  const char* base;
  const char* last;
  int64_t tile;
  uint32_t st;  // token stride in bytes
};

__device__ __forceinline__ void dma_vrow(const Dma& D, const VDma& V, int i, u32x4* buf) {
  const int64_t base = (int64_t)i * kKeyTile;
  const char* tile = V.base + (int64_t)i * V.tile;
  const bool tail = base + kKeyTile > D.len;
#pragma unroll
  for (int x = 0; x < 3; x++) {
    if (x < 2 || D.wave + 16 < kDmaK) {
      uint32_t off = D.krow[x] * V.st + D.kcol[x];
      // (the tile starts at or before the last row, so the offset stays >= 0)
      if (tail && base + D.krow[x] >= D.len) off = (uint32_t)(V.last - tile) + D.kcol[x];
      dma16_at(tile, off, buf + 64 * (D.wave + 8 * x));
    }
  }
}

constexpr int kDqStage = 2 * kBufK + kBufV;  // K, V (row-major), K^T (packed)
constexpr int kDqRow = kHeadDim / 4 + 1;  // 16-byte chunks per staged fp32 dQ row (one pad)
constexpr int kDqLds = 2 * kDqStage > kRows * kDqRow + kRows / 2 ? 2 * kDqStage : kRows * kDqRow + kRows / 2;

template <int MODE>
__global__ __launch_bounds__(512, 1) void bwd_dq_kernel(BwdArgs a, Problem p) {
  __shared__ u32x4 lds[kDqLds];
  __shared__ RowInfo rtab[MODE == kHist ? 1 : kRows];  // current-block rows (see below)
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int qc = lane & 31, hh = lane >> 5;

  // ------------------------------------------------------------ tile setup
  int g, s;
  int64_t kbeg, kend, tmin;
  RowInfo ri;
  const int rloc = wave * 32 + qc;
  if constexpr (MODE == kHist) {
    const int64_t nb = p.nblk_total;
    const int64_t tbeg = a.bin_tile_start[a.g0 * nb];
    const int64_t tend = a.bin_tile_start[a.g1 * nb];
    // tiles of one bin share its K/V block: a contiguous run of tiles per XCD
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
    tmin = kend;
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
  g = __builtin_amdgcn_readfirstlane(g);
  s = __builtin_amdgcn_readfirstlane(s);
  kbeg = uniform64(kbeg);
  kend = uniform64(kend);
  tmin = uniform64(tmin);
  const SeqInfo sq = a.seqs[s];
  const int64_t tok0 = sq.tok_start;

  // ------------------------------------------- Q^T, dO^T operands, lse, Delta
  bf16x8 qf[8], df[8];
  {
    const __hip_bfloat16* qrow = static_cast<const __hip_bfloat16*>(a.q) + ri.t * a.q_st +
                                 (int64_t)ri.h * a.q_sh + 8 * hh;
    const __hip_bfloat16* drow = static_cast<const __hip_bfloat16*>(a.dout) + ri.t * a.do_st +
                                 (int64_t)ri.h * a.do_sh + 8 * hh;
#pragma unroll
    for (int kk = 0; kk < 8; kk++) {
      qf[kk] = as_bf16x8(*reinterpret_cast<const u32x4*>(qrow + 16 * kk));
      df[kk] = as_bf16x8(*reinterpret_cast<const u32x4*>(drow + 16 * kk));
    }
  }
  const float2 ld = a.ld[(int64_t)ri.h * p.T + ri.t];
  // current-block tiles: the row's bookkeeping waits in LDS (registers are
  // the loop's; measured: the history variant runs faster keeping it)
  if (MODE != kHist && hh == 0) rtab[rloc] = ri;

  // ------------------------------------------------------------ key tiles
  const int64_t rb = kbeg - tok0, re = kend - tok0;
  const int i0 = (int)(rb / kKeyTile), i1 = (int)((re + kKeyTile - 1) / kKeyTile);
  Dma DK;  // K row-major and the packed K^T
  VDma DV;  // V row-major
  {
    const int wv = __builtin_amdgcn_readfirstlane(wave);
    const char* kb = reinterpret_cast<const char*>(static_cast<const __hip_bfloat16*>(a.k) +
                                                   (int64_t)g * a.k_sh) + tok0 * (a.k_st * 2);
    const char* ktb = reinterpret_cast<const char*>(
        a.kt + ((int64_t)g * p.vt_tiles + sq.vt_tile_off) * (kKeyTile * kHeadDim));
    init_dma(DK, wv, lane, kb, a.k_st * 2, sq.len, ktb);
    DV.st = (uint32_t)(a.v_st * 2);
    DV.base = reinterpret_cast<const char*>(static_cast<const __hip_bfloat16*>(a.v) +
                                            (int64_t)g * a.v_sh) + tok0 * (a.v_st * 2);
    DV.last = DV.base + (sq.len - 1) * (a.v_st * 2);
    DV.tile = kKeyTile * (a.v_st * 2);
  }
  ReadOff ro;
  ro.kq = qc * kRowK + hh;
  ro.vq = qc * kRowV + hh;
  const float c2 = a.scale_log2;
  f32x16 acc[4];
#pragma unroll
  for (int dt = 0; dt < 4; dt++)
#pragma unroll
    for (int r = 0; r < 16; r++) acc[dt][r] = 0.0f;

  // stage x: K at lds + x*kDqStage, V at + kBufK, K^T at + 2*kBufK
  dma_k(DK, i0, lds);
  dma_vrow(DK, DV, i0, lds + kBufK);
  dma_v(DK, i0, lds + 2 * kBufK);
  dma_wait();
  __syncthreads();

  for (int i = i0; i < i1; i++) {
    const int cur = (i - i0) & 1;
    u32x4* st = lds + cur * kDqStage;
    if (i + 1 < i1) {
      u32x4* nx = lds + (cur ^ 1) * kDqStage;
      dma_k(DK, i + 1, nx);
      dma_vrow(DK, DV, i + 1, nx + kBufK);
      dma_v(DK, i + 1, nx + 2 * kBufK);
    }
    const int64_t u0 = tok0 + (int64_t)i * kKeyTile;
    const bool edge = u0 < kbeg || u0 + kKeyTile > kend || (MODE != kHist && u0 + kKeyTile - 1 > tmin);
    int lo = 0, hi = kKeyTile;
    if (edge) {
      lo = (int)max((int64_t)0, kbeg - u0) - 4 * hh;
      const int64_t lim = min((int64_t)kKeyTile, kend - u0);
      hi = (int)(MODE == kHist ? lim : min(lim, rtab[rloc].t + 1 - u0)) - 4 * hh;
    }
    bf16x8 db[4];
#pragma unroll
    for (int th = 0; th < 2; th++) {
      f32x16 sh, dh;
      sdp_half(sh, dh, st, st + kBufK, ro, th, qf, df);
      grad_half(sh, dh, db, th, edge, lo, hi, c2, ld.x, ld.y);
    }
    pv(acc, st + 2 * kBufK, ro, db);
    dma_wait();
    __syncthreads();
  }

  // -------------------------------------------------------------- epilogue
  const RowInfo r = MODE == kHist ? ri : rtab[rloc];
  if (MODE != kHist && !r.valid) return;
  const float scl = a.scale;
  if constexpr (MODE == kHist) {
    // the rows leave whole: staged in LDS (free after the loop's last
    // barrier), then 32 lanes x 16 bytes per row, two rows per instruction
    float4* stg = reinterpret_cast<float4*>(lds);
    int64_t* sdst = reinterpret_cast<int64_t*>(lds + kRows * kDqRow);
#pragma unroll
    for (int dt = 0; dt < 4; dt++)
#pragma unroll
      for (int r4 = 0; r4 < 4; r4++)
        stg[rloc * kDqRow + 8 * dt + 2 * r4 + hh] =
            make_float4(acc[dt][4 * r4] * scl, acc[dt][4 * r4 + 1] * scl,
                        acc[dt][4 * r4 + 2] * scl, acc[dt][4 * r4 + 3] * scl);
    if (hh == 0) sdst[rloc] = r.valid ? r.dst : -1;
    __syncthreads();
    const int ch = lane & 31;
#pragma unroll
    for (int j = 0; j < 16; j++) {
      const int rr = 32 * wave + 2 * j + hh;
      const int64_t d = sdst[rr];
      if (d >= 0) reinterpret_cast<float4*>(a.dq_part + d * kHeadDim)[ch] = stg[rr * kDqRow + ch];
    }
  } else {
#pragma unroll
    for (int dt = 0; dt < 4; dt++)
#pragma unroll
      for (int r = 0; r < 16; r++) acc[dt][r] *= scl;
    // history slots of this row, in slot order
    const int kh = p.topk - 1;
    const int nh = (int)min((int64_t)kh, (r.t - tok0) / p.B);
    const float* part = a.dq_part + r.dst * kh * kHeadDim;
    for (int x = 0; x < nh; x++) {
#pragma unroll
      for (int dt = 0; dt < 4; dt++)
#pragma unroll
        for (int r4 = 0; r4 < 4; r4++) {
          const float4 f =
              *reinterpret_cast<const float4*>(part + x * kHeadDim + 32 * dt + 8 * r4 + 4 * hh);
          acc[dt][4 * r4] += f.x;
          acc[dt][4 * r4 + 1] += f.y;
          acc[dt][4 * r4 + 2] += f.z;
          acc[dt][4 * r4 + 3] += f.w;
        }
    }
    __hip_bfloat16* drow =
        static_cast<__hip_bfloat16*>(a.dq) + r.t * a.dq_st + (int64_t)r.h * a.dq_sh;
#pragma unroll
    for (int dt = 0; dt < 4; dt++)
#pragma unroll
      for (int r4 = 0; r4 < 4; r4++) {
        uint2 w;
        w.x = pack_bf16(acc[dt][4 * r4], acc[dt][4 * r4 + 1]);
        w.y = pack_bf16(acc[dt][4 * r4 + 2], acc[dt][4 * r4 + 3]);
        *reinterpret_cast<uint2*>(drow + 32 * dt + 8 * r4 + 4 * hh) = w;
      }
  }
}

// ============================================================== dK, dV
constexpr int kChunk = 64;          // rows per chunk
constexpr int kBufR = kChunk * 16;  // one row-major Q or dO chunk: 64 rows x 16 16-byte chunks
constexpr int kDmaR = kBufR / 64;   // DMA instructions per chunk and tensor (16)
constexpr int kSlots = 3;           // row tables in flight
// s_waitcnt operand that waits for LDS operations only (lgkmcnt 0, vmcnt and
// expcnt at their maxima)
constexpr int kWaitLds = 0xC07F;

// Swizzled row-major chunk: the logical 16-byte chunk c of row r is stored
// at r*16 + (c ^ swz(r)), swz(r) = 4*(r % 4) + (r / 4) % 4.  Both reads of
// the buffer are then free of LDS bank conflicts:
//  - operand reads of S = Q K^T and dP = dO V^T: 16 lanes on 16 consecutive
//    rows at one logical chunk (swz takes 16 distinct values there);
//  - transposed reads (ds_read_b64_tr_b16) for dV^T += dO^T P and
//    dK^T += Q^T dS: per 32 lanes, 4 consecutive rows (starting at a multiple
//    of 4) by the 4 logical chunks of 32 dims; the rows' swz differ in bits
//    2-3, so their 64-byte windows are disjoint.
// ds_read_b64_tr_b16: within each group of 16 lanes, lane i receives element
// i % 4 of the 8-byte pieces addressed by lanes 4e + i / 4 (e = 0..3).  If
// lane j of the group addresses row r0 + j/4 at dims d0 + 4 (j % 4), lane i
// receives dims d0 + i of rows r0 .. r0+3: four consecutive rows of one
// dimension, the transposed operand.
__device__ __forceinline__ int swz(int r) { return ((r & 3) << 2) | ((r >> 2) & 3); }

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ s16x4 tr_read(const char* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)p);
}

struct __align__(16) RowTab {
  int64_t qoff[kSlots][kChunk];  // byte offset of the row's Q vector (t * q_st + h * q_sh)
  int64_t doff[kSlots][kChunk];  // byte offset of the row's dO vector
  int kmax[kSlots][kChunk];   // last key the row may attend (causal rows), -1 for padding
  float lse2[kSlots][kChunk];
  float dlt[kSlots][kChunk];
};

// What one lane of wave 0 fetches for one row of a chunk.
struct RowFetch {
  int4 rec;
  float2 ld;
  int t, h, kind;  // kind 0: routed history row, 1: row of the block itself, 2: padding
};

struct RowList {
  int64_t nhist, bstart, nrows;
  int k0, nct, g;
};

__device__ __forceinline__ RowFetch row_fetch(const BwdArgs& a, const Problem& p, const RowList& L,
                                              int ci, int lane) {
  RowFetch f;
  const int64_t x = (int64_t)ci * kChunk + lane;
  f.t = L.k0;
  f.h = L.g * p.G;
  if (x < L.nhist) {
    f.kind = 0;
    f.rec = a.rec[L.bstart + x];
  } else if (x < L.nrows) {
    f.kind = 1;
    const int y = (int)(x - L.nhist);
    const int hl = y / L.nct;
    f.t = L.k0 + (y - hl * L.nct);
    f.h = L.g * p.G + hl;
    f.ld = a.ld[(int64_t)f.h * p.T + f.t];
  } else {
    f.kind = 2;
  }
  return f;
}

__device__ __forceinline__ void row_store(const BwdArgs& a, RowTab& R, int slot, int lane,
                                          const RowFetch& f) {
  int t = f.t, h = f.h, km = -1;
  float l2 = INFINITY, dl = 0.0f;
  if (f.kind == 0) {
    t = f.rec.x;
    h = f.rec.y;
    l2 = __int_as_float(f.rec.z);
    dl = __int_as_float(f.rec.w);
    km = INT_MAX;
  } else if (f.kind == 1) {
    l2 = f.ld.x;
    dl = f.ld.y;
    km = t;
  }
  R.qoff[slot][lane] = ((int64_t)t * a.q_st + (int64_t)h * a.q_sh) * 2;
  R.doff[slot][lane] = ((int64_t)t * a.do_st + (int64_t)h * a.do_sh) * 2;
  R.kmax[slot][lane] = km;
  R.lse2[slot][lane] = l2;
  R.dlt[slot][lane] = dl;
}

// P of one 32-row subtile as written by a P-wave for its D-wave, the bf16
// operands the P-wave feeds its own dV product (so dS = P (dP - Delta) uses
// the same rounded P as dV): [parity][pair][half][lane] 16 bytes (lane
// order, so every access is one contiguous 1 KiB per wave).
struct __align__(16) PExchange {
  uint4 p[2][kDkdvWaves / 2][2][64];
};

// S = Q K^T (P-wave) or dP = dO V^T (D-wave) of subtile st: 8 k-steps with
// the A operands from the swizzled chunk buffer and B = this wave's K or V.
__device__ __forceinline__ f32x16 sd_product(const char* buf, int st, const uint32_t (&offa)[8],
                                             const bf16x8 (&kv)[8]) {
  u32x4 op[8];
#pragma unroll
  for (int j = 0; j < 8; j++) op[j] = *reinterpret_cast<const u32x4*>(buf + 8192 * st + offa[j]);
  f32x16 acc;
#pragma unroll
  for (int r = 0; r < 16; r++) acc[r] = 0.0f;
#pragma unroll
  for (int j = 0; j < 8; j++) acc = mfma(as_bf16x8(op[j]), kv[j], acc);
  __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
  for (int j = 0; j < 4; j++) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
  return acc;
}

// acc^T (dims x keys) += X^T (dims x rows) . W (rows x keys) over subtile st,
// X the swizzled chunk buffer read transposed, W the bf16 operands w[s2].
__device__ __forceinline__ void g_product(f32x16 (&acc)[4], const char* buf, int st,
                                          const uint32_t (&offt)[2][4], const bf16x8 (&w)[2]) {
  s16x4 tl[8], th[8];
#pragma unroll
  for (int j = 0; j < 8; j++) {
    const int s2 = j >> 2, dt = j & 3;
    const char* b = buf + (32 * st + 16 * s2) * 256;
    tl[j] = tr_read(b + offt[0][dt]);
    th[j] = tr_read(b + offt[1][dt]);
  }
#pragma unroll
  for (int j = 0; j < 8; j++) {
    const int s2 = j >> 2, dt = j & 3;
    acc[dt] = mfma(__builtin_bit_cast(bf16x8, __builtin_shufflevector(tl[j], th[j], 0, 1, 2, 3, 4, 5,
                                                                       6, 7)),
                   w[s2], acc[dt]);
  }
  __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
#pragma unroll
  for (int j = 0; j < 4; j++) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
}

// P-wave: P = exp2(S c2 - lse2) of subtile st (zero where a row may not
// attend the lane's key, EDGE chunks), into the exchange and as bf16
// operands pb[s2].  A lane's values are rows 32*st + 8*r4 + 4*hh + (0..3).
template <bool EDGE>
__device__ __forceinline__ void p_weights(const f32x16& sv, const RowTab& R, int slot, int st,
                                          int hh, int lane, int key, int k1, float c2,
                                          uint4 (&xo)[2][64], bf16x8 (&pb)[2]) {
  uint32_t w[8];
#pragma unroll
  for (int r4 = 0; r4 < 4; r4++) {
    const int row0 = 32 * st + 8 * r4 + 4 * hh;
    const float4 l2 = *reinterpret_cast<const float4*>(&R.lse2[slot][row0]);
    const float lv[4] = {l2.x, l2.y, l2.z, l2.w};
    float pr[4];
#pragma unroll
    for (int c = 0; c < 4; c++) pr[c] = __builtin_amdgcn_exp2f(fmaf(sv[4 * r4 + c], c2, -lv[c]));
    if (EDGE) {
      const int4 km = *reinterpret_cast<const int4*>(&R.kmax[slot][row0]);
      const int kv[4] = {km.x, km.y, km.z, km.w};
#pragma unroll
      for (int c = 0; c < 4; c++) pr[c] = (key <= kv[c] && key < k1) ? pr[c] : 0.0f;
    }
    w[2 * r4] = pack_bf16(pr[0], pr[1]);
    w[2 * r4 + 1] = pack_bf16(pr[2], pr[3]);
  }
  pb[0] = as_bf16x8(u32x4{w[0], w[1], w[2], w[3]});
  pb[1] = as_bf16x8(u32x4{w[4], w[5], w[6], w[7]});
  xo[0][lane] = make_uint4(w[0], w[1], w[2], w[3]);
  xo[1][lane] = make_uint4(w[4], w[5], w[6], w[7]);
}

// D-wave: dS = P (dP - Delta) of subtile st as bf16 operands sb[s2].
__device__ __forceinline__ void ds_weights(const f32x16& dpv, const RowTab& R, int slot, int st,
                                           int hh, int lane, const uint4 (&xi)[2][64],
                                           bf16x8 (&sb)[2]) {
  uint32_t w[8];
  const uint4 x0 = xi[0][lane], x1 = xi[1][lane];
  const uint32_t pw[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
#pragma unroll
  for (int r4 = 0; r4 < 4; r4++) {
    const int row0 = 32 * st + 8 * r4 + 4 * hh;
    const float4 dl = *reinterpret_cast<const float4*>(&R.dlt[slot][row0]);
    const float4 pp = make_float4(__uint_as_float(pw[2 * r4] << 16), __uint_as_float(pw[2 * r4] & 0xffff0000u),
                                  __uint_as_float(pw[2 * r4 + 1] << 16),
                                  __uint_as_float(pw[2 * r4 + 1] & 0xffff0000u));
    w[2 * r4] = pack_bf16(pp.x * (dpv[4 * r4] - dl.x), pp.y * (dpv[4 * r4 + 1] - dl.y));
    w[2 * r4 + 1] = pack_bf16(pp.z * (dpv[4 * r4 + 2] - dl.z), pp.w * (dpv[4 * r4 + 3] - dl.w));
  }
  sb[0] = as_bf16x8(u32x4{w[0], w[1], w[2], w[3]});
  sb[1] = as_bf16x8(u32x4{w[4], w[5], w[6], w[7]});
}

// Work-group: 4 pairs of waves, each pair owning 32 keys.  The P-wave holds
// K, computes S and P and accumulates dV^T; the D-wave holds V, computes dP
// and dS (with the P-wave's P, passed through LDS with a per-pair flag for
// each 32-row subtile) and accumulates dK^T one subtile late.
// Each wave so holds one 32-key operand set and one 32x128 accumulator, and
// the two waves of a SIMD run matrix and vector work beside each other.
// Waves w and w + 4 share a SIMD; P-wave q (wave q) is paired with D-wave
// 4 + (q + 2) % 4, so the two waves of a SIMD belong to different pairs and
// neither waits on the other's progress (2.7% faster than pairing the two
// waves of one SIMD, whose phases then lock together).
__global__ __launch_bounds__(64 * kDkdvWaves, 1) void bwd_dkdv_kernel(BwdArgs a, Problem p) {
  __shared__ u32x4 lds[5 * kBufR];  // Q chunk x3 (dK runs a subtile late), dO chunk x2
  __shared__ RowTab R;
  __shared__ PExchange X;
  __shared__ int pflag[kDkdvWaves / 2];  // subtiles whose P the pair's P-wave has written
  constexpr int kW = kDkdvWaves;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int qc = lane & 31, hh = lane >> 5;
  // role 0: P-wave, 1: D-wave (wave-uniform: scalar branches)
  const int role = __builtin_amdgcn_readfirstlane(wave >> 2), pair = (wave + 2 * role) & 3;

  // work-group -> (kv-head, key tile): each XCD takes a contiguous run (the
  // key tiles of one bin read the same rows), early blocks (longest row
  // lists) first
  const int64_t total = a.nktiles * p.Hkv;
  const int64_t per = gridDim.x / 8;
  const int64_t wi = (int64_t)(blockIdx.x % 8) * per + blockIdx.x / 8;
  if (wi >= total) return;
  RowList L;
  L.g = (int)(wi / a.nktiles);
  const KeyTile kt = a.ktiles[wi % a.nktiles];
  L.k0 = kt.k0;
  L.nct = kt.bend - kt.k0;
  L.nhist = 0;
  L.bstart = 0;
  if (a.bin_count) {
    const int64_t bin = (int64_t)L.g * p.nblk_total + kt.b;
    L.nhist = a.bin_count[bin];
    L.bstart = a.bin_start[bin];
  }
  L.nhist = uniform64(L.nhist);
  L.bstart = uniform64(L.bstart);
  L.nrows = L.nhist + (int64_t)L.nct * p.G;
  const int nch = (int)((L.nrows + kChunk - 1) / kChunk);

  // the pair's 32 keys; this wave's K (P-wave) or V (D-wave) as B operands
  const int kw0 = kt.k0 + 32 * pair;
  const bool live = kw0 < kt.k1;
  const bool full = kw0 + 32 <= kt.k1;
  const int key = kw0 + qc;
  const int kld = min(key, kt.k1 - 1);
  bf16x8 kv[8];
  {
    const __hip_bfloat16* src =
        role == 0 ? static_cast<const __hip_bfloat16*>(a.k) + (int64_t)kld * a.k_st + (int64_t)L.g * a.k_sh
                  : static_cast<const __hip_bfloat16*>(a.v) + (int64_t)kld * a.v_st + (int64_t)L.g * a.v_sh;
#pragma unroll
    for (int kk = 0; kk < 8; kk++)
      kv[kk] = as_bf16x8(*reinterpret_cast<const u32x4*>(src + 8 * hh + 16 * kk));
  }

  // DMA: instruction j (0..15, per tensor) writes buffer chunks 64j ..
  // 64j+63; wave w issues j = w + 8x; lane L fills row 4j + L/16, stored
  // chunk L % 16, i.e. logical chunk (L % 16) ^ swz(row)
  constexpr int kDx = kDmaR / kW;
  static_assert(kDmaR % kW == 0, "whole DMA instructions per wave");
  int drow[kDx];
  uint32_t dcol[kDx];
#pragma unroll
  for (int x = 0; x < kDx; x++) {
    drow[x] = 4 * (wave + kW * x) + (lane >> 4);
    dcol[x] = (uint32_t)((((lane & 15) ^ swz(drow[x]))) * 16);
  }
  const char* qb = static_cast<const char*>(a.q);
  const char* db = static_cast<const char*>(a.dout);
  auto dma_rows = [&](int slot, u32x4* qbuf, u32x4* dbuf) {
#pragma unroll
    for (int x = 0; x < kDx; x++) {
      dma16(qb + R.qoff[slot][drow[x]] + dcol[x], qbuf + 64 * (wave + kW * x));
      dma16(db + R.doff[slot][drow[x]] + dcol[x], dbuf + 64 * (wave + kW * x));
    }
  };

  // per-lane byte offsets into a chunk buffer
  //  S / dP operands: row qc (+32 st), logical chunk 2kk + hh
  uint32_t offa[8];
  {
    const int sq = swz(qc);
#pragma unroll
    for (int kk = 0; kk < 8; kk++) offa[kk] = (uint32_t)(qc * 256 + (((2 * kk + hh) ^ sq) * 16));
  }
  //  transposed operands: group lane i = qc % 16 addresses row
  //  r0 + i/4 (r0 = 32 st + 16 s2 + 4 hh + 8 x) at dims 32 dt + 16 (qc/16) + 4 (i%4)
  uint32_t offt[2][4];
  {
    const int i = qc & 15, trow = i >> 2;
    const int cl = 2 * (qc >> 4) + ((i & 3) >> 1);
#pragma unroll
    for (int x = 0; x < 2; x++)
#pragma unroll
      for (int dt = 0; dt < 4; dt++)
        offt[x][dt] = (uint32_t)((4 * hh + trow + 8 * x) * 256 +
                                 (4 * (dt ^ trow) + (cl ^ (hh + 2 * x))) * 16 + 8 * (i & 1));
  }

  f32x16 acc[4];  // P-wave: dV^T, D-wave: dK^T (dims x keys)
#pragma unroll
  for (int dt = 0; dt < 4; dt++)
#pragma unroll
    for (int r = 0; r < 16; r++) acc[dt][r] = 0.0f;
  const float c2 = a.scale_log2;

  // prologue: row tables of chunks 0 and 1, chunk 0 landed
  if (tid < kDkdvWaves / 2) pflag[tid] = 0;
  if (wave == 0) {
    row_store(a, R, 0, lane, row_fetch(a, p, L, 0, lane));
    if (nch > 1) row_store(a, R, 1, lane, row_fetch(a, p, L, 1, lane));
  }
  __syncthreads();
  dma_rows(0, lds, lds + 3 * kBufR);
  dma_wait();
  __syncthreads();

  // The two roles run separate copies of the chunk loop (same DMA, row
  // tables and one barrier per chunk), so neither carries the other's
  // registers.  D-wave: dK^T += Q^T dS of a subtile runs one subtile late,
  // beside the P-wave's exponentials of the next one (Q chunks are
  // triple-buffered for it).
  volatile __attribute__((address_space(3))) int* flag =
      (volatile __attribute__((address_space(3))) int*)&pflag[pair];
  if (role == 0) {
    for (int i = 0; i < nch; i++) {
      const int cur = i & 1;
      RowFetch nf;
      const bool fetch = wave == 0 && i + 2 < nch;
      if (fetch) nf = row_fetch(a, p, L, i + 2, lane);
      if (i + 1 < nch)
        dma_rows((i + 1) % kSlots, lds + ((i + 1) % 3) * kBufR, lds + (3 + (cur ^ 1)) * kBufR);
      const char* qr = reinterpret_cast<const char*>(lds + (i % 3) * kBufR);
      const char* dr = reinterpret_cast<const char*>(lds + (3 + cur) * kBufR);
      const int slot = i % kSlots;
      const bool edge = (int64_t)(i + 1) * kChunk > L.nhist || !full;
#pragma unroll 1
      for (int st = 0; st < 2; st++) {
        if (!live) continue;
        bf16x8 wb[2];
        const f32x16 sd = sd_product(qr, st, offa, kv);  // S
        if (edge) p_weights<true>(sd, R, slot, st, hh, lane, key, kt.k1, c2, X.p[st][pair], wb);
        else p_weights<false>(sd, R, slot, st, hh, lane, key, kt.k1, c2, X.p[st][pair], wb);
        // hand P(st) to the pair's D-wave: raise the flag once the exchange
        // writes have completed (lgkmcnt 0; the DMA in flight is not waited for)
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        __builtin_amdgcn_s_waitcnt(kWaitLds);
        *flag = 2 * i + st + 1;
        g_product(acc, dr, st, offt, wb);  // dV^T += dO^T P
      }
      dma_wait();
      if (fetch) row_store(a, R, (i + 2) % kSlots, lane, nf);
      __syncthreads();
    }
  } else {
    bool have_prev = false;
    const char* q_prev = nullptr;
    int st_prev = 0;
    bf16x8 wb_prev[2];
    for (int i = 0; i < nch; i++) {
      const int cur = i & 1;
      if (i + 1 < nch)
        dma_rows((i + 1) % kSlots, lds + ((i + 1) % 3) * kBufR, lds + (3 + (cur ^ 1)) * kBufR);
      const char* qr = reinterpret_cast<const char*>(lds + (i % 3) * kBufR);
      const char* dr = reinterpret_cast<const char*>(lds + (3 + cur) * kBufR);
      const int slot = i % kSlots;
#pragma unroll 1
      for (int st = 0; st < 2; st++) {
        if (!live) continue;
        const f32x16 sd = sd_product(dr, st, offa, kv);  // dP
        if (have_prev) g_product(acc, q_prev, st_prev, offt, wb_prev);  // dK^T += Q^T dS
        // wait (bounded, so it always ends) for the P-wave's P(st); a wait
        // that gives up goes on with a stale P and is counted, so the host
        // can report it (the flag is in LDS: n is wave-uniform)
        const int seq = 2 * i + st + 1 + a.wait_bias;
        int n = 0;
        while (*flag < seq && ++n < a.spin_limit) __builtin_amdgcn_s_sleep(1);
        if (n >= a.spin_limit && lane == 0) atomicAdd(a.wait_timeouts, 1u);
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        ds_weights(sd, R, slot, st, hh, lane, X.p[st][pair], wb_prev);
        have_prev = true;
        q_prev = qr;
        st_prev = st;
      }
      dma_wait();
      __syncthreads();
    }
    if (have_prev) g_product(acc, q_prev, st_prev, offt, wb_prev);
  }

  // -------------------------------------------------------------- epilogue
  if (!live || key >= kt.k1) return;
  const float scl = role == 0 ? 1.0f : a.scale;
  __hip_bfloat16* dst = role == 0 ? static_cast<__hip_bfloat16*>(a.dv) + (int64_t)key * a.dv_st +
                                        (int64_t)L.g * a.dv_sh
                                  : static_cast<__hip_bfloat16*>(a.dk) + (int64_t)key * a.dk_st +
                                        (int64_t)L.g * a.dk_sh;
#pragma unroll
  for (int dt = 0; dt < 4; dt++)
#pragma unroll
    for (int r4 = 0; r4 < 4; r4++) {
      uint2 w;
      w.x = pack_bf16(acc[dt][4 * r4] * scl, acc[dt][4 * r4 + 1] * scl);
      w.y = pack_bf16(acc[dt][4 * r4 + 2] * scl, acc[dt][4 * r4 + 3] * scl);
      *reinterpret_cast<uint2*>(dst + 32 * dt + 8 * r4 + 4 * hh) = w;
    }
}

}  // namespace

hipError_t launch_bwd_delta(const BwdArgs& a, const Problem& p, hipStream_t st) {
  const int64_t rows = p.T * p.Hq;
  if (rows <= 0) return hipSuccess;
  bwd_delta_kernel<<<(unsigned)((rows + 15) / 16), 256, 0, st>>>(a, p);
  return hipGetLastError();
}

hipError_t launch_bwd_rec(const BwdArgs& a, const Problem& p, hipStream_t st) {
  if (p.hist_entries <= 0 || p.topk <= 1) return hipSuccess;
  bwd_rec_kernel<<<(unsigned)((p.hist_entries + 255) / 256), 256, 0, st>>>(a, p);
  return hipGetLastError();
}

hipError_t launch_bwd_dq_hist(const BwdArgs& a, const Problem& p, int64_t grid, hipStream_t st) {
  if (grid <= 0) return hipSuccess;
  grid = (grid + 7) / 8 * 8;
  bwd_dq_kernel<kHist><<<(unsigned)grid, 512, 0, st>>>(a, p);
  return hipGetLastError();
}

hipError_t launch_bwd_dq_cur(const BwdArgs& a, const Problem& p, hipStream_t st) {
  if (a.ntiles <= 0 || a.g1 <= a.g0) return hipSuccess;
  dim3 grid((unsigned)a.ntiles, a.g1 - a.g0);
  bwd_dq_kernel<kCur><<<grid, 512, 0, st>>>(a, p);
  return hipGetLastError();
}

hipError_t launch_bwd_dkdv(const BwdArgs& a, const Problem& p, hipStream_t st) {
  const int64_t total = a.nktiles * p.Hkv;
  if (total <= 0) return hipSuccess;
  const int64_t grid = (total + 7) / 8 * 8;
  bwd_dkdv_kernel<<<(unsigned)grid, 64 * kDkdvWaves, 0, st>>>(a, p);
  return hipGetLastError();
}

}  // namespace moba
