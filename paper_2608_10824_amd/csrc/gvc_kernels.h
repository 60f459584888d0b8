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

// ------------------------------------------------------------------ GEMM
// Work units of a GEMM launch.  Pair maps give a workgroup two 16-row weight
// blocks whose epilogue partners share lanes; single maps give it one block.
enum { MAP_PLAIN = 0, MAP_QKV = 1, MAP_GU = 2, MAP_SINGLE = 3, MAP_QKV_SINGLE = 4 };
enum { EPI_QKV = 0, EPI_RESID = 1, EPI_SILU = 2, EPI_STORE = 3, EPI_EMBED = 4, EPI_QKV_RAW = 5 };

struct RowMap {
  const int* idx;   // row index into the residual / output arrays
  const int* ep;    // episode b
  const int* pos;   // absolute position
};

struct EpiArgs {
  RowMap rows;
  // EPI_QKV (and EPI_QKV_RAW: q, k before RoPE as fp32 [M][d] in qraw, kraw)
  float* qraw; float* kraw;
  bf16* q;            // [Mp][d] row-major, after RoPE
  bf16* kc;           // this layer's K cache
  bf16* vc;           // this layer's V cache (transposed)
  const float2* rope; // [kv_pad][head_dim/2] (cos, sin)
  int d, head_dim, n_heads, kv_pad;
  // EPI_RESID: out[row] = resid[row] + acc, rows mapped through rows.idx when *_mapped
  const float* resid; int resid_mapped;
  float* out; int out_mapped;
  // EPI_SILU: frag-layout bf16 activations with kb_act k-fragments per row block
  bf16* act; int kb_act; int n_feat;
  // EPI_STORE
  float* store; int ld_store;
  // EPI_EMBED
  float* h0; const bf16* embed; const int* text_ids; const float* extra;
  int n_patches, n_text, n_extra;
  // Folded RMSNorm (decode): the GEMM input is bf16(x * gain) and the
  // accumulator is scaled by 1/sqrt(sum(x^2)/norm_dim + norm_eps), the sum
  // of squares of row m being the sum of ssq_in[m * ssq_parts + 0..parts-1].
  const float* ssq_in; int ssq_parts; float norm_eps; int norm_dim;
  // EPI_RESID, when xn != nullptr: also writes bf16(out * xn_gain) in frag
  // layout (xn_kb k-fragments) and, per row, this pair's sum of squares of
  // out into ssq_out[m * ssq_out_parts + pair].
  bf16* xn; const float* xn_gain; float* ssq_out; int xn_kb; int ssq_out_parts;
};

struct GemmArgs {
  const bf16x8* w[3];   // packed matrices (fragment units)
  int wblk[3];          // 16-row blocks per matrix
  int map;
  int n_pairs;          // work units (pairs, or single blocks for the single maps)
  int n_out;            // output features of the (first) matrix, for MAP_PLAIN
  int KB;               // k-fragments (K padded / 32)
  int splits, kb_per_split;   // waves per workgroup (token groups x k shares), k-steps per share
  int tgroups;                // token groups per workgroup (KT)
  const bf16x8* x;      // frag-layout activations
  int M, mblocks, mtiles;
  EpiArgs e;
};

// k-steps per pipelined register chunk for a tile of NT blocks of 16 token rows.
constexpr int gemm_pf(int NT) { return NT == 1 ? 8 : (NT <= 3 ? 4 : (NT <= 6 ? 2 : 1)); }

// ------------------------------------------------------------------ persistent decode pass
// One single-token pass over all layers for one episode (k_decode.hip).
constexpr int kDecodeMaxSeg = 8;       // weight blocks per workgroup per step
constexpr int kDecodeAbortWord = 512;  // barrier words: abort flag
constexpr int kDecodeXccWord = 544;    // barrier words: set when a workgroup is not on XCD blockIdx % 8
constexpr int kDecodeHeadWord = 1024;  // barrier words: per-head counters, 32 words apart
constexpr int kDecodeMaxHeads = 64;
constexpr int kDecodeBarWords = kDecodeHeadWord + 32 * kDecodeMaxHeads;   // zeroed before a launch sequence
// grid barriers and per-head barriers of one pass over L layers
constexpr int decode_grid_barriers(int L) { return 1 + 3 * L; }
constexpr int decode_head_barriers(int L) { return L; }

struct DecodeArgs {
  // packed weights of layer 0 (k = q + qkv_stride, v = q + 2 qkv_stride,
  // up = gate + gu_stride); layer l's are l * layer_stride further (bf16x8 units)
  const bf16x8* wq; const bf16x8* wo; const bf16x8* wg; const bf16x8* wd;
  size_t qkv_stride, gu_stride, layer_stride;
  bf16* kc; bf16* vc;          // layer 0 caches (episode 0); layer l at l * kv_layer_elems
  size_t kv_layer_elems;
  const float* gains;          // [L][2][d]: attention norm, FFN norm
  const float2* rope;          // [kv_pad][head_dim/2]
  float* x;                    // [d] layer input / output (in place)
  float* r;                    // [d] residual after attention
  float* qkv;                  // [3d] q, k, v before RoPE
  bf16* act;                   // [F] SwiGLU output
  unsigned* bar;               // kDecodeBarWords barrier words
  unsigned bar_base;           // grid barriers completed by earlier launches since the words were zeroed
  unsigned hbar_base;          // per-head barriers completed by earlier launches
  long long timeout_ticks;     // barrier wait limit in wall-clock ticks (100 MHz)
  int L, d, F, H, head_dim, KBd, KBf, kv_pad, pos, act_bytes;
  float eps;
  int flags;                   // kDecodeNtWeights | kDecodeWarmKv
};
constexpr int kDecodeNtWeights = 1;   // weight loads marked non-temporal
constexpr int kDecodeWarmKv = 2;      // step 1 pulls the head's cached keys and values into L2

}  // namespace gvc

#include "gvc_launch.h"
