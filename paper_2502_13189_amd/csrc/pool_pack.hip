// Block mean-pool of the keys and the packed V^T layout of the MFMA kernels.
//
// Pool (Eq. 6; Algorithm 1 mean_pool): one work-group per (global block,
// kv-head).  256 threads = 16 token rows x 16 lanes; each lane owns 8
// consecutive dims and walks the block's tokens with stride 16, reading a
// 256-byte key row per 16 lanes (coalesced).  Sums are kept in fp64 and
// reduced across the 16 rows in a fixed order, so the result is the block
// mean rounded once to fp32 and is bit-reproducible.
//
// V^T pack: one work-group per (64-key tile of a sequence, kv-head).  The
// tile's 64 x 128 values are staged in LDS and written back as 128 rows
// (dims) of 64 keys, with the keys of every 16-key group stored in the order
// 0-3, 8-11, 4-7, 12-15.  That order is the k-slot order in which the
// attention kernel's P^T operand holds keys after the QK^T MFMA (see
// attn_mfma.hip), so each lane reads its 8 keys as one 16-byte LDS load.
// Keys past the end of the sequence are stored as zeros.
#include "moba_internal.h"

namespace moba {
namespace {

template <typename T>
struct Load8;

template <>
struct Load8<__hip_bfloat16> {
  static __device__ __forceinline__ void run(const __hip_bfloat16* p, float* f) {
    uint4 u = *reinterpret_cast<const uint4*>(p);
    uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; i++) {
      f[2 * i] = __uint_as_float(w[i] << 16);
      f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  }
};

template <>
struct Load8<float> {
  static __device__ __forceinline__ void run(const float* p, float* f) {
    float4 a = *reinterpret_cast<const float4*>(p);
    float4 b = *reinterpret_cast<const float4*>(p + 4);
    f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w;
    f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
  }
};

// kterm (nullable): the block keys split exactly into three bf16 planes,
// kbar = hi + mid + lo, each plane [nblk_total, Hkv, D] (read by the
// matrix-core gate).
template <typename T>
__global__ __launch_bounds__(256) void pool_kernel(const T* __restrict__ k, int64_t k_st, int64_t k_sh,
                                                   const SeqInfo* __restrict__ seqs, int S, int B,
                                                   int Hkv, int nblk_total, float* __restrict__ kbar,
                                                   __hip_bfloat16* __restrict__ kterm) {
  __shared__ double red[16][kHeadDim];
  const int b = blockIdx.x;
  const int g = blockIdx.y;
  const int s = find_seq(seqs, S, b, [](const SeqInfo& x) { return x.blk_off; });
  const SeqInfo sq = seqs[s];
  const int j = b - sq.blk_off;
  const int64_t t0 = (int64_t)sq.tok_start + (int64_t)j * B;
  const int64_t t1 = (int64_t)sq.tok_start + min((int64_t)(j + 1) * B, (int64_t)sq.len);
  const int row = threadIdx.x >> 4;
  const int d0 = (threadIdx.x & 15) * 8;
  double acc[8];
#pragma unroll
  for (int i = 0; i < 8; i++) acc[i] = 0.0;
  for (int64_t t = t0 + row; t < t1; t += 16) {
    float f[8];
    Load8<T>::run(k + t * k_st + (int64_t)g * k_sh + d0, f);
#pragma unroll
    for (int i = 0; i < 8; i++) acc[i] += (double)f[i];
  }
#pragma unroll
  for (int i = 0; i < 8; i++) red[row][d0 + i] = acc[i];
  __syncthreads();
  if (threadIdx.x < kHeadDim) {
    double sum = 0.0;
#pragma unroll
    for (int r = 0; r < 16; r++) sum += red[r][threadIdx.x];
    const float m = (float)(sum / (double)(t1 - t0));
    const int64_t o = ((int64_t)b * Hkv + g) * kHeadDim + threadIdx.x;
    kbar[o] = m;
    if (kterm) {
      const int64_t plane = (int64_t)nblk_total * Hkv * kHeadDim;
      const __hip_bfloat16 hi = __float2bfloat16(m);
      const float r1 = m - __bfloat162float(hi);
      const __hip_bfloat16 mid = __float2bfloat16(r1);
      kterm[o] = hi;
      kterm[o + plane] = mid;
      kterm[o + 2 * plane] = __float2bfloat16(r1 - __bfloat162float(mid));
    }
  }
}

// Position p (0..63) of a packed tile holds key perm(p) of the tile.
__device__ __forceinline__ int packed_key(int p) {
  const int grp = p & ~15, w = p & 15;
  const int half = w >> 3, jj = w & 7;
  return grp + 8 * (jj >> 2) + 4 * half + (jj & 3);
}

__global__ __launch_bounds__(256) void vt_pack_kernel(const __hip_bfloat16* __restrict__ v,
                                                      int64_t v_st, int64_t v_sh,
                                                      const SeqInfo* __restrict__ seqs, int S,
                                                      int64_t vt_tiles,
                                                      __hip_bfloat16* __restrict__ vt) {
  __shared__ uint16_t tile[kKeyTile][kHeadDim + 2];
  const int64_t idx = blockIdx.x;
  const int g = blockIdx.y;
  const int s = find_seq(seqs, S, idx, [](const SeqInfo& x) { return x.vt_tile_off; });
  const SeqInfo sq = seqs[s];
  const int i = (int)(idx - sq.vt_tile_off);
  // stage 64 keys x 128 dims: 1024 chunks of 8 values, 4 per thread
#pragma unroll
  for (int x = 0; x < 4; x++) {
    const int c = threadIdx.x + 256 * x;
    const int r = c >> 4, col = (c & 15) * 8;
    const int local = i * kKeyTile + r;
    uint4 u = make_uint4(0, 0, 0, 0);
    if (local < sq.len)
      u = *reinterpret_cast<const uint4*>(v + ((int64_t)sq.tok_start + local) * v_st +
                                          (int64_t)g * v_sh + col);
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int e = 0; e < 4; e++) {
      tile[r][col + 2 * e] = (uint16_t)(w[e] & 0xffffu);
      tile[r][col + 2 * e + 1] = (uint16_t)(w[e] >> 16);
    }
  }
  __syncthreads();
  __hip_bfloat16* dst = vt + ((int64_t)g * vt_tiles + idx) * (kKeyTile * kHeadDim);
#pragma unroll
  for (int x = 0; x < 4; x++) {
    const int c = threadIdx.x + 256 * x;
    const int d = c >> 3, p0 = (c & 7) * 8;
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 4; e++) {
      const uint32_t lo = tile[packed_key(p0 + 2 * e)][d];
      const uint32_t hi = tile[packed_key(p0 + 2 * e + 1)][d];
      w[e] = lo | (hi << 16);
    }
    *reinterpret_cast<uint4*>(dst + d * kKeyTile + p0) = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

}  // namespace

hipError_t launch_pool(const void* k, bool bf16, int64_t k_st, int64_t k_sh, const SeqInfo* seqs,
                       const Problem& p, float* kbar, __hip_bfloat16* kterm, hipStream_t st) {
  if (p.nblk_total == 0) return hipSuccess;
  dim3 grid(p.nblk_total, p.Hkv);
  if (bf16)
    pool_kernel<__hip_bfloat16><<<grid, 256, 0, st>>>(
        static_cast<const __hip_bfloat16*>(k), k_st, k_sh, seqs, p.S, p.B, p.Hkv, p.nblk_total,
        kbar, kterm);
  else
    pool_kernel<float><<<grid, 256, 0, st>>>(static_cast<const float*>(k), k_st, k_sh, seqs, p.S,
                                             p.B, p.Hkv, p.nblk_total, kbar, kterm);
  return hipGetLastError();
}

hipError_t launch_vt_pack(const __hip_bfloat16* v, int64_t v_st, int64_t v_sh, const SeqInfo* seqs,
                          const Problem& p, __hip_bfloat16* vt, hipStream_t st) {
  if (p.vt_tiles == 0) return hipSuccess;
  dim3 grid((unsigned)p.vt_tiles, p.Hkv);
  vt_pack_kernel<<<grid, 256, 0, st>>>(v, v_st, v_sh, seqs, p.S, p.vt_tiles, vt);
  return hipGetLastError();
}

}  // namespace moba
