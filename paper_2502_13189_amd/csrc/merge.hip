// Log-sum-exp combine of the per-block attention results (the combine step of
// Algorithm 1; Sec. 2.3), bf16 path.  The current-block kernel has already
// written each row's normalised current-block result to out (bf16) and its lse
// to lse; this kernel folds the row's history partials into them in place:
//   lse = M + ln(sum_i e^{lse_i - M}),  out = sum_i e^{lse_i - lse} O_i,
// accumulated in fp32 in a fixed order (current block first, then history
// slots ascending) and rounded once to bf16.
//
// 16 lanes per row, 8 dims (one 16-byte load) per lane and partial; each
// lane loads one slot's lse and the row's lanes share them.  Partials
// are read in groups of kGroup, all loads of a group in flight at once, with
// an online rescale between groups (one group covers top-k up to 13).
#include "moba_internal.h"

#include <math.h>

namespace moba {
namespace {

constexpr int kLanesPerRow = 16;
constexpr int kRowsPerGroup = 256 / kLanesPerRow;
constexpr int kGroup = 12;
constexpr float kLn2 = 0.69314718055994531f;
constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ void unpack8(uint4 u, float (&f)[8]) {
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; i++) {
    f[2 * i] = __uint_as_float(w[i] << 16);
    f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Two fp32 values to a packed bf16 pair, round-to-nearest-even.
__device__ __forceinline__ uint32_t pack2(float a, float b) {
  const f32x2 v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

__global__ __launch_bounds__(256) void merge_kernel(AttnArgs a, Problem p) {
  const int64_t TG = p.T * p.G;
  const int64_t nrow = (int64_t)(a.g1 - a.g0) * TG;
  // r = (g - g0) * T * G + t * G + hl: the chunk-relative row, which is also
  // the row index of the history partials
  const int64_t r = (int64_t)blockIdx.x * kRowsPerGroup + (threadIdx.x / kLanesPerRow);
  const int l16 = threadIdx.x % kLanesPerRow;
  if (r >= nrow) return;
  const int gl = (int)(r / TG);
  const int64_t rem = r - gl * TG;
  const int64_t t = rem / p.G;
  const int h = (a.g0 + gl) * p.G + (int)(rem % p.G);
  const int s = find_seq(a.seqs, p.S, t, [](const SeqInfo& x) { return x.tok_start; });
  const int64_t c = (t - a.seqs[s].tok_start) / p.B;
  const int kh = p.topk - 1;
  const int nh = (int)min((int64_t)kh, c);
  if (nh <= 0) return;

  uint4* orow = reinterpret_cast<uint4*>(static_cast<__hip_bfloat16*>(a.out) + t * a.o_st +
                                         (int64_t)h * a.o_sh + 8 * l16);
  float* lrow = a.lse + (int64_t)h * p.T + t;
  const float* lp = a.lse_part + r * kh;
  const uint4* op = reinterpret_cast<const uint4*>(static_cast<const __hip_bfloat16*>(a.o_part) +
                                                   r * kh * kHeadDim + 8 * l16);

  const float lc = *lrow;
  float oc[8];
  unpack8(*orow, oc);
  float M = lc, wsum = 1.0f;
  float acc[8];
#pragma unroll
  for (int d = 0; d < 8; d++) acc[d] = oc[d];
  for (int x0 = 0; x0 < nh; x0 += kGroup) {
    uint4 v[kGroup];
    float lv[kGroup];
    // the group's lse values: lane l16 of the row loads slot x0 + l16, the
    // others read it from that lane
    const float lmine = x0 + l16 < nh ? lp[x0 + l16] : 0.0f;
#pragma unroll
    for (int j = 0; j < kGroup; j++) {
      lv[j] = __shfl(lmine, j, kLanesPerRow);
      if (x0 + j < nh) v[j] = op[(int64_t)(x0 + j) * (kHeadDim / 8)];
    }
    float Mg = M;
#pragma unroll
    for (int j = 0; j < kGroup; j++)
      if (x0 + j < nh) Mg = fmaxf(Mg, lv[j]);
    const float sc = __builtin_amdgcn_exp2f((M - Mg) * kLog2e);
    wsum *= sc;
#pragma unroll
    for (int d = 0; d < 8; d++) acc[d] *= sc;
    M = Mg;
#pragma unroll
    for (int j = 0; j < kGroup; j++) {
      if (x0 + j < nh) {
        const float w = __builtin_amdgcn_exp2f((lv[j] - M) * kLog2e);
        wsum += w;
        float f[8];
        unpack8(v[j], f);
#pragma unroll
        for (int d = 0; d < 8; d++) acc[d] = fmaf(w, f[d], acc[d]);
      }
    }
  }
  const float inv = 1.0f / wsum;
  uint4 o;
  o.x = pack2(acc[0] * inv, acc[1] * inv);
  o.y = pack2(acc[2] * inv, acc[3] * inv);
  o.z = pack2(acc[4] * inv, acc[5] * inv);
  o.w = pack2(acc[6] * inv, acc[7] * inv);
  *orow = o;
  if (l16 == 0) *lrow = M + __builtin_amdgcn_logf(wsum) * kLn2;
}

}  // namespace

hipError_t launch_merge_bf16(const AttnArgs& a, const Problem& p, hipStream_t st) {
  const int64_t nrow = (int64_t)(a.g1 - a.g0) * p.T * p.G;
  if (nrow <= 0 || p.topk <= 1) return hipSuccess;
  const int64_t grid = (nrow + kRowsPerGroup - 1) / kRowsPerGroup;
  merge_kernel<<<(unsigned)grid, 256, 0, st>>>(a, p);
  return hipGetLastError();
}

}  // namespace moba
