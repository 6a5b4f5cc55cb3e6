// Log-sum-exp merge of the partial attention results (Algorithm 1, combine
// with online softmax; Sec. 2.3 "re-arrange the attention outputs back to
// their original ordering" and combine).
//
// Every row (kv-head g, token t, head hl of the group) has the current-block
// partial and min(topk-1, c) history partials, each a normalised output O_i
// with its natural-log lse_i.  With M = max lse_i:
//   lse = M + ln sum_i exp(lse_i - M),  out = sum_i exp(lse_i - lse) O_i.
// The sum runs in a fixed order (current block, then history slots in
// ascending block order), so the result is deterministic.  32 lanes per row,
// 4 dims per lane; the output is rounded once to the input dtype.
#include "moba_internal.h"

#include <math.h>

namespace moba {
namespace {

template <typename T>
__device__ __forceinline__ void store4(T* dst, float4 v);

template <>
__device__ __forceinline__ void store4<float>(float* dst, float4 v) {
  *reinterpret_cast<float4*>(dst) = v;
}

template <>
__device__ __forceinline__ void store4<__hip_bfloat16>(__hip_bfloat16* dst, float4 v) {
  const __hip_bfloat16 a = __float2bfloat16(v.x), b = __float2bfloat16(v.y),
                       c = __float2bfloat16(v.z), d = __float2bfloat16(v.w);
  uint2 w;
  w.x = (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
  w.y = (uint32_t)__builtin_bit_cast(uint16_t, c) | ((uint32_t)__builtin_bit_cast(uint16_t, d) << 16);
  *reinterpret_cast<uint2*>(dst) = w;
}

template <typename T>
__global__ __launch_bounds__(256) void merge_kernel(AttnArgs a, Problem p, int64_t rows) {
  const int64_t cr = (int64_t)blockIdx.x * 8 + (threadIdx.x >> 5);
  if (cr >= rows) return;
  const int d = (threadIdx.x & 31) * 4;
  const int64_t TG = p.T * p.G;
  const int g = a.g0 + (int)(cr / TG);
  const int64_t rem = cr % TG;
  const int64_t t = rem / p.G;
  const int h = g * p.G + (int)(rem % p.G);
  const int s = find_seq(a.seqs, p.S, t, [](const SeqInfo& x) { return x.tok_start; });
  const int c = (int)((t - a.seqs[s].tok_start) / p.B);
  const int kh = p.topk - 1;
  const int nh = min(kh, c);
  const float* lp = a.lse_part + cr * kh;
  const float lc = a.lse_cur[cr];
  float M = lc;
  for (int x = 0; x < nh; x++) M = fmaxf(M, lp[x]);
  float w = expf(lc - M);
  float sum = w;
  float4 acc = reinterpret_cast<const float4*>(a.o_cur + cr * kHeadDim + d)[0];
  acc.x *= w; acc.y *= w; acc.z *= w; acc.w *= w;
  for (int x = 0; x < nh; x++) {
    w = expf(lp[x] - M);
    sum += w;
    const float4 o = reinterpret_cast<const float4*>(a.o_part + (cr * kh + x) * kHeadDim + d)[0];
    acc.x = fmaf(w, o.x, acc.x);
    acc.y = fmaf(w, o.y, acc.y);
    acc.z = fmaf(w, o.z, acc.z);
    acc.w = fmaf(w, o.w, acc.w);
  }
  const float inv = 1.0f / sum;
  acc.x *= inv; acc.y *= inv; acc.z *= inv; acc.w *= inv;
  store4<T>(static_cast<T*>(a.out) + t * a.o_st + (int64_t)h * a.o_sh + d, acc);
  if (d == 0) a.lse[(int64_t)h * p.T + t] = M + logf(sum);
}

}  // namespace

hipError_t launch_merge(bool bf16, const AttnArgs& a, const Problem& p, hipStream_t st) {
  const int64_t rows = (int64_t)(a.g1 - a.g0) * p.T * p.G;
  if (rows == 0) return hipSuccess;
  const unsigned grid = (unsigned)((rows + 7) / 8);
  if (bf16) merge_kernel<__hip_bfloat16><<<grid, 256, 0, st>>>(a, p, rows);
  else merge_kernel<float><<<grid, 256, 0, st>>>(a, p, rows);
  return hipGetLastError();
}

}  // namespace moba
