// Host-side launchers of the HIP kernels of libgvc (declarations only; the
// kernels and device helpers they launch are in gvc_kernels.h).
#pragma once
#include "gvc_kernels.h"

namespace gvc {

// ------------------------------------------------------------------ launchers
// All launchers enqueue on `s` and return hipGetLastError().
hipError_t launch_pack(const bf16* src, int N, int K, bf16* dst, int Nblk, int KB, hipStream_t s);
hipError_t launch_convert_gain(const bf16* src, float* dst, int n, hipStream_t s);
hipError_t launch_rope_table(float2* tab, int kv_pad, int head_dim, float theta, hipStream_t s);
hipError_t launch_fill_u32(uint32_t* p, uint32_t v, size_t n, hipStream_t s);
// Zeroes positions [from, kv_pad) of n_blk key blocks ([kv_pad][dh]) and value
// blocks ([dh][kv_pad]).
hipError_t launch_zero_kv_tail(bf16* k, bf16* v, size_t n_blk, int kv_pad, int dh, int from, hipStream_t s);

hipError_t launch_patch_stats(const uint8_t* ft, const uint8_t* fp, int B, int views, int img, int patch,
                              int* stats, hipStream_t s);
// Stage 1 (+ Stage 2 when tv != nullptr: per patch the sum over LH columns of
// tv [B][LH][N], in order; the topk highest, ties to the lower index, are not static).
hipError_t launch_rank_mask(const int* stats, int B, int N, int L, long long tau_num, long long tau_den,
                            const int* permille_host, uint8_t* mask, int* n_static, const float* tv, int LH,
                            int topk, const float* ent, int H, int n_instr, int* q_out, hipStream_t s);

hipError_t launch_build_rows(const uint8_t* mask, const int* valid, int B, int L, int N, int P,
                             int* rows, int* counts, int* ep_counts, int* ep_offsets, hipStream_t s);
hipError_t launch_im2row(const uint8_t* frame, int views, int img, int patch, const int* idx, const int* pos,
                         int M, int P, int KB, bf16* x, hipStream_t s);
hipError_t launch_layernorm(const float* src, int M, int d, const float* gain, const float* bias, float eps,
                            bf16* x, int KB, hipStream_t s);
hipError_t launch_gather_visual(const bf16* src, const int* idx, const int* pos, int M, int P, int N, int KB,
                                bf16* x, hipStream_t s);
// tiled: one workgroup per block of 16 rows (many-row sessions) instead of
// one per row; the two sum a row's squares in different orders, so a session
// keeps one choice.
hipError_t launch_rmsnorm(const float* src, const int* idx, int M, int d, const float* gain, float eps,
                          bf16* x, int KB, bool tiled, hipStream_t s);
hipError_t launch_gemm_big(const GemmArgs& a, int epi, hipStream_t s);
// Split-k prompt-pass GEMM (k_gemm_sk or k_gemm_dx, then the slice sum and
// epilogue); workgroups own groups of gemm_sk_group_blocks(a.sk_shape)
// weight blocks.
hipError_t launch_gemm_sk(const GemmArgs& a, int epi, hipStream_t s);
int gemm_sk_group_blocks(int sk_shape);
// Whether a split-k launch of M rows takes one tall tile per k slice (the
// wide and narrow shapes at 161-288 rows).
bool gemm_sk_tall_rows(int M);
hipError_t launch_gemm(const GemmArgs& a, int epi, int NT, hipStream_t s);
// Stage 2 signal of one layer: tv[b * tv_bstride + h * N + n] = sum over the
// T1 instruction rows after the image of their softmax probability on visual
// key n (1 <= T1 <= 32, N + T1 < 640).
hipError_t launch_text_vis(const bf16* q, const bf16* kc, const int* ep_counts, const int* ep_offsets, int B, int H,
                           int head_dim, int kv_pad, int N, int P, int T1, float* tv, size_t tv_bstride,
                           float* ent, size_t ent_bstride, hipStream_t s);
hipError_t launch_attn_prefill(const bf16* q, const bf16* kc, const bf16* vc, const int* rows_pos,
                               const int* ep_counts, const int* ep_offsets, int B, int H, int head_dim,
                               int kv_pad, int max_tiles, bf16* o, int KB, int block_first, int block_last,
                               bool grouped, hipStream_t s);
hipError_t launch_attn_decode(const float* qraw, const float* kraw, bf16* kc, const bf16* vc, const float2* rope,
                              int B, int H, int head_dim, int kv_pad, int pos, bf16* o, int KB, hipStream_t s);
hipError_t launch_embed_tokens(const bf16* embed, const int* tokens, int tok_stride, int B, int d, int V,
                               float* x, const float* gain, bf16* xn, int KB, float* ssq, hipStream_t s);
hipError_t launch_logits_reduce(const float* logits, int rows, int V, int bin_lo, int full_vocab,
                                int* tok_out, float* margin_out, int out_stride, int out_col,
                                int rows_per_ep, hipStream_t s);
size_t decode_pass_lds_bytes(int act_bytes);
int decode_pass_threads();
int decode_pass_score_offset();
const void* decode_pass_kernel(int head_dim, int d_model);
hipError_t launch_decode_pass(const DecodeArgs& a, int n_wg, hipStream_t s);   // cooperative launch
// abort_word (or NULL): when set, every episode is invalidated and reported as fired with a NaN margin
// Scratch of the allocation-free selection: per-patch statistics of at most
// kSelectScratchEpisodes x kSelectScratchPatches patches (192 KiB per GPU).
constexpr int kSelectScratchEpisodes = 16;
constexpr int kSelectScratchPatches = 1024;
hipError_t select_scratch(int** out);   // this device's copy (looked up once per device)
hipError_t launch_gate(const float* margins, int B, int D, float theta, int use_min, const int8_t* force,
                       const unsigned* abort_word, int* valid, float* m_out, int* fire_out, hipStream_t s);

}  // namespace gvc
