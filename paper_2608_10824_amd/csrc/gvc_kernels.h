// Internal declarations shared by the HIP kernels and the host side of libgvc.
//
// Data layouts used on the device:
//  * packed weights: a [N][K] bf16 matrix is stored as 16-row blocks, each
//    block as K/32 fragments of 64 lanes x 8 bf16 (1 KiB), in the operand
//    order of the gfx950 MFMA v_mfma_f32_16x16x32_bf16: lane l of fragment
//    (blk, kb) holds W[blk*16 + l%16][kb*32 + (l/16)*8 + 0..7].  A wave streams
//    a block as contiguous 1 KiB loads.  Rows >= N and columns >= K are zero.
//  * activations feeding a GEMM ("frag layout"): the same arrangement with
//    token rows in place of weight rows: element (m, k) lives in fragment
//    (m/16, k/32), lane ((k%32)/8)*16 + m%16, slot k%8.
//  * K cache: bf16 [B][H][kv_pad][head_dim] per layer, after RoPE.
//  * V cache: bf16 [B][H][head_dim][kv_pad] per layer (transposed, so a run of
//    keys for one dimension is contiguous).
//  * hidden state H: fp32 [L+1][B][P][d]; row index b*P + pos.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gvc {

typedef uint16_t bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ float bf2f(bf16 h) { return __uint_as_float(((uint32_t)h) << 16); }

// fp32 -> bf16, round to nearest even; NaN stays NaN.
__device__ __forceinline__ bf16 f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (bf16)((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (bf16)(u >> 16);
}

__device__ __forceinline__ floatx4 mfma16(const bf16x8& a, const bf16x8& b, const floatx4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Offset (in bf16 elements) of element (m, k) in frag layout with KB k-fragments per row block.
__device__ __forceinline__ size_t frag_off(int m, int k, int KB) {
  return ((((size_t)(m >> 4) * KB + (k >> 5)) * 64 + ((k & 31) >> 3) * 16 + (m & 15)) << 3) + (k & 7);
}

// Cross-lane reductions on DPP row operations (a few cycles each) instead of
// LDS permutes.  dpp_f<C>: v of the lane that DPP control C selects.
template <int C>
__device__ __forceinline__ float dpp_f(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), C, 0xF, 0xF, false));
}
constexpr int kDppXor1 = 0xB1;        // quad_perm [1, 0, 3, 2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2, 3, 0, 1]
constexpr int kDppHalfMirror = 0x141; // lane i of 8 <- lane 7 - i: the other quad, once quads agree
constexpr int kDppMirror = 0x140;     // lane i of 16 <- lane 15 - i: the other half, once halves agree
// Sum over aligned groups of N lanes (N = 1, 2, 4, 8, 16); every lane of a
// group ends with the same value.
template <int N>
__device__ __forceinline__ float group_sum(float v) {
  static_assert(N == 1 || N == 2 || N == 4 || N == 8 || N == 16, "group size");
  if constexpr (N >= 2) v += dpp_f<kDppXor1>(v);
  if constexpr (N >= 4) v += dpp_f<kDppXor2>(v);
  if constexpr (N >= 8) v += dpp_f<kDppHalfMirror>(v);
  if constexpr (N >= 16) v += dpp_f<kDppMirror>(v);
  return v;
}
__device__ __forceinline__ float lane_f(float v, int l) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), l));
}
// Sum and maximum over the whole wave (all lanes active), wave-uniform.
__device__ __forceinline__ float wave_sum(float v) {
  v = group_sum<16>(v);
  return (lane_f(v, 0) + lane_f(v, 16)) + (lane_f(v, 32) + lane_f(v, 48));
}
__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, dpp_f<kDppXor1>(v));
  v = fmaxf(v, dpp_f<kDppXor2>(v));
  v = fmaxf(v, dpp_f<kDppHalfMirror>(v));
  v = fmaxf(v, dpp_f<kDppMirror>(v));
  return fmaxf(fmaxf(lane_f(v, 0), lane_f(v, 16)), fmaxf(lane_f(v, 32), lane_f(v, 48)));
}

// Maximum over aligned groups of N lanes (N = 2, 4, 8, 16), as group_sum.
template <int N>
__device__ __forceinline__ float group_max(float v) {
  static_assert(N == 2 || N == 4 || N == 8 || N == 16, "group size");
  v = fmaxf(v, dpp_f<kDppXor1>(v));
  if constexpr (N >= 4) v = fmaxf(v, dpp_f<kDppXor2>(v));
  if constexpr (N >= 8) v = fmaxf(v, dpp_f<kDppHalfMirror>(v));
  if constexpr (N >= 16) v = fmaxf(v, dpp_f<kDppMirror>(v));
  return v;
}

// ------------------------------------------------------------------ logits
// Greedy-token and margin helpers (Eq. 1) shared by the logits reduction and
// the decode pass: a total order on (logit, id) -- higher logit first, then
// the lower id -- and a running top-2 and (max, sum of exp) under it.
__device__ __forceinline__ bool better(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

// Adds candidate (v, i) to a running top-2 (v1, i1) >= (v2, i2) under `better`,
// a total order (value, then lower id), so the result does not depend on the
// order of the additions.
__device__ __forceinline__ void top2_add(float& v1, int& i1, float& v2, int& i2, float v, int i) {
  const bool b1 = better(v, i, v1, i1), b2 = better(v, i, v2, i2);
  const float nv2 = b1 ? v1 : (b2 ? v : v2);
  const int ni2 = b1 ? i1 : (b2 ? i : i2);
  v1 = b1 ? v : v1;
  i1 = b1 ? i : i1;
  v2 = nv2;
  i2 = ni2;
}

// Running (max, sum of exp(z - max)) pair; a term at -inf contributes 0.
__device__ __forceinline__ void lse_add(float& mx, float& sum, float v) {
  if (v > mx) {
    sum = sum * __expf(mx - v) + 1.f;
    mx = v;
  } else if (v != -INFINITY) {
    sum += __expf(v - mx);
  }
}

__device__ __forceinline__ void lse_merge(float& mx, float& sum, float mo, float so) {
  const float m = fmaxf(mx, mo);
  if (m == -INFINITY) return;
  sum = (mx == -INFINITY ? 0.f : sum * __expf(mx - m)) + (mo == -INFINITY ? 0.f : so * __expf(mo - m));
  mx = m;
}

}  // namespace gvc

#include "gvc_gemm.h"
#include "gvc_decode.h"
#include "gvc_launch.h"
