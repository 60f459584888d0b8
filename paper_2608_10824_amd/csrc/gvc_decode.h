// Arguments and constants of the single-launch decode pass (k_decode.hip).
// Part of gvc_kernels.h: include that header, not this one.
#pragma once

namespace gvc {

// ------------------------------------------------------------------ persistent decode pass
// One single-token pass over all layers for one episode (k_decode.hip).
constexpr int kDecodeMaxSeg = 8;       // weight blocks per workgroup per step
constexpr int kDecodeAbortWord = 512;  // barrier words: abort flag
constexpr int kDecodeXccWord = 544;    // barrier words: set when a workgroup is not on XCD blockIdx % 8
constexpr int kDecodePoisonWord = 576; // barrier words: set when a head contribution was not finite
constexpr int kDecodeHeadWord = 1024;  // barrier words: per-head counters, 32 words apart
constexpr int kDecodeMaxHeads = 64;
constexpr int kDecodeMaxGrid = 1024;   // workgroups of one pass (per-workgroup head records)
// zeroed before a launch sequence, except the abort word, which stays set
// until the gate that follows has reported it
constexpr int kDecodeBarWords = kDecodeHeadWord + 32 * kDecodeMaxHeads;
// grid barriers and per-head barriers of one pass over L layers (one more
// grid barrier when the pass also runs the LM head and the token choice)
constexpr int decode_grid_barriers(int L, bool head) { return 1 + 3 * L + (head ? 1 : 0); }
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
  unsigned long long* racc;    // [d] sum of the heads' attention-output contributions, int64 in 2^-32 units
  float* qkv;                  // [3d] q, k, v before RoPE
  bf16* act;                   // [F] SwiGLU output
  unsigned* bar;               // kDecodeBarWords barrier words
  unsigned bar_base;           // grid barriers completed by earlier launches since the words were zeroed
  unsigned hbar_base;          // per-head barriers completed by earlier launches
  long long timeout_ticks;     // barrier wait limit in wall-clock ticks (100 MHz)
  int L, d, F, H, head_dim, KBd, KBf, kv_pad, pos, act_bytes;
  float eps;
  int flags;                   // kDecodeNtWeights | kDecodeWarmKv | kDecodeHead
  // with kDecodeHead: final norm, LM head and the greedy token and margin of
  // this pass (Eq. 1) after the last layer
  const bf16x8* wlm;           // packed LM head, nlm blocks of KBd fragments
  const float* final_gain;     // [d]
  float* logits;               // [V] this pass's logits
  float* head_part;            // [gridDim <= kDecodeMaxGrid][8] per workgroup: max, sum, v1, i1, v2, i2
  int* tok_out;                // the token of this pass (one int)
  float* margin_out;           // its margin (one float)
  int nlm, V, bin_lo, full_vocab;
};
constexpr int kDecodeNtWeights = 1;   // weight loads marked non-temporal
constexpr int kDecodeWarmKv = 2;      // step 1 pulls the head's cached keys and values into L2
constexpr int kDecodeHead = 4;        // the pass ends with the LM head and the token choice

}  // namespace gvc
