/*
 * gvc.h - C ABI of the Gated VLA-Cache control-step library for MI355X (gfx950).
 *
 * One control step of a Llama-2-shaped vision-language-action decoder in which
 * visually static image-patch tokens reuse the K/V they had at the previous
 * frame, and a logit-margin gate forces a full recompute when the model's
 * action confidence was low (arxiv 2608.10824, Alg. 1).  A step is:
 *
 *   gvc_margin_gate      Eq. 1 margin of the previous step, compared with theta
 *                        (Alg. 1, first test); invalidates fired episodes.
 *   gvc_select_static    Stage 1 patch cosine similarity of I_t vs I_{t-1}
 *                        (Sec. III-B) with a per-layer reuse proportion (Stage 3).
 *   gvc_step_prefill     the prompt pass over the non-reused tokens only, with
 *                        fresh K/V scattered into the persistent cache
 *                        (Alg. 1, partial or full forward pass).
 *   gvc_decode_actions   autoregressive decode of the D action tokens (Sec. III-A,
 *                        Alg. 1 last step), recording each token's margin.
 *
 * Conventions shared by every call:
 *  - Every function returns GVC_OK (0) or a GVC_E* code; gvc_last_error() gives
 *    a thread-local message for the last failure.  No C++ exception crosses
 *    this boundary.
 *  - "dev" pointers are device memory of the GPU current when gvc_init_cache
 *    ran; "host" pointers are ordinary host memory.  The caller owns all
 *    device memory (weights, arenas, inputs, outputs); the library owns only
 *    the host-side context.  Device pointers must be 256-byte aligned.
 *  - Work is enqueued on the HIP stream given to gvc_init_cache, in call
 *    order.  Calls return before the GPU finishes except gvc_margin_gate,
 *    gvc_step_prefill (it waits for the per-layer row counts, a few bytes,
 *    before enqueuing the layers) and gvc_read_state.
 *  - No call allocates device memory; gvc_init_cache allocates only the
 *    host context.
 *  - A context is not thread-safe; calls on one context must not overlap.
 *
 * Key slots per layer: kv_len = P + D - 1 (autoregressive) or P (parallel),
 * padded to kv_pad = kv_len rounded up to a multiple of 32.
 *
 * Data layout of the model (all row-major, bf16 = IEEE bfloat16 bits):
 *  Token order of one episode's prompt of P = N + n_text + n_proprio + n_action_q
 *  rows, row index = position: [text 0] [N visual tokens, view-major, raster]
 *  [text 1..n_text-1] [proprio rows] [action-query rows].  Only visual tokens
 *  can be reused.
 */
#ifndef GVC_H
#define GVC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum gvc_status {
  GVC_OK = 0,
  GVC_EINVAL = 1,   /* null pointer, bad shape or threshold, NaN theta */
  GVC_ESTATE = 2,   /* call out of order (e.g. decode before any prefill) */
  GVC_ENOMEM = 3,   /* an arena is smaller than gvc_sizes reported */
  GVC_EDEVICE = 4   /* a HIP call failed; see gvc_last_error() */
};

enum gvc_reduce { GVC_REDUCE_MEAN = 0, GVC_REDUCE_MIN = 1 };

enum gvc_state_item {
  GVC_STATE_H = 0,       /* fp32 [B][P][d]  hidden state entering layer `layer` (0..L) */
  GVC_STATE_K = 1,       /* bf16 [B][n_heads][kv_pad][head_dim] keys of layer `layer` (after RoPE) */
  GVC_STATE_V = 2,       /* bf16 [B][n_heads][head_dim][kv_pad] values of layer `layer` (dim-major) */
  GVC_STATE_HEAD_LOGITS = 3, /* fp32 [B][n_head_rows][V] logits of the last prompt pass */
  GVC_STATE_VALID = 4,   /* int32 [B] cache-valid flags */
  GVC_STATE_ROWS = 5,    /* int32 [L]: rows recomputed per layer by the last prompt pass */
  GVC_STATE_MARGINS = 6, /* fp32 [B][D] per-position margins of the last decode */
  GVC_STATE_TV = 7,      /* fp32 [B][L][n_heads][N] Stage 2 attention of the last prompt pass
                            (desc.task_topk > 0; the layer argument is ignored) */
  GVC_STATE_ENTROPY = 8, /* fp32 [B][L][n_heads] Stage 3 signal of the last prompt pass: per head,
                            the sum over the instruction tokens after the image of their attention
                            entropy divided by log(keys seen) (desc.entropy_reuse; layer ignored) */
  GVC_STATE_LAYER_Q = 9  /* int32 [B][L] per-layer reuse proportions (per mille) the last
                            gvc_select_static applied (desc.entropy_reuse; layer ignored) */
};

/* Model and workload shape.  Llama-2 block (Sec. V-A backbone): pre-norm
 * RMSNorm, rotary embedding pairing dim i with i + head_dim/2, multi-head
 * attention, SwiGLU; no biases. */
typedef struct gvc_desc {
  int32_t batch;          /* B independent episodes stepped together, 1 <= B <= 16 */
  int32_t n_layers;       /* L */
  int32_t d_model;        /* d, a multiple of 64 */
  int32_t n_heads;        /* head_dim = d / n_heads must be 64 or 128 */
  int32_t ffn;            /* SwiGLU hidden width F */
  int32_t vocab;          /* V; the last n_bins ids are the action bins */
  int32_t n_bins;         /* 2 <= n_bins <= vocab; vocab a multiple of 16 */
  int32_t img;            /* frame side in pixels (square frames) */
  int32_t patch;          /* patch side p; img % p == 0; N = n_views (img/p)^2 */
  int32_t n_views;        /* camera views per frame */
  int32_t n_text;         /* language tokens, >= 1 */
  int32_t n_proprio;      /* proprio rows (given embeddings) */
  int32_t n_action_q;     /* action-query rows (given embeddings) */
  int32_t n_decode;       /* D action tokens per step */
  int32_t parallel_decode;/* 0: D-1 single-token passes follow the prompt pass;
                             1: the D action-query rows give the D positions */
  int32_t norm_full_vocab;/* 1: softmax normaliser over all V ids; 0: over the bins */
  float rms_eps;          /* RMSNorm epsilon (1e-5 for Llama-2) */
  float rope_theta;       /* rotary base (10000 for Llama-2) */
  int32_t task_topk;      /* Stage 2 (Sec. III-B): 0 = off; else each prompt pass records, per layer
                             and head, the softmax probability that the instruction tokens after the
                             image (1 <= n_text - 1 <= 32) put on each visual key, and the next
                             gvc_select_static takes the task_topk patches of highest total out of
                             the static set.  0 <= task_topk <= N; N + n_text < 640. */
  int32_t entropy_reuse;  /* Stage 3 (Sec. III-B): 0 = the caller's fixed proportions; 1 = each
                             prompt pass also records the normalized attention entropy E_l of those
                             instruction tokens (mean over heads and tokens of the entropy over the
                             keys up to the token, divided by log of their count), and the next
                             gvc_select_static reuses q_l = floor(1000 s_l) per mille in layer l,
                             s_0 = u_0, s_l = s_{l-1} + (u_l - s_{l-1}) / 2, u_l = 1 - E_l, clamped to
                             [0, 1]: low-entropy layers reuse more.  Same limits as Stage 2. */
  int32_t action_bidir;   /* OFT action block (Sec. V-A, parallel action-dimension decoding): 0 = every
                             row causal; 1 = the n_action_q action-query rows (the last rows of the
                             prompt) attend to every prompt key, so they see each other both ways.
                             Needs parallel_decode = 1 and n_action_q >= 1. */
  int32_t vit_layers;     /* vision front end (Sec. III-A, Sec. V-A models): 0 = a visual token's
                             embedding is (patch pixels / 255) . patch_proj^T; else every prompt pass
                             runs, per camera view, a ViT without class token over all the view's
                             patches -- patch embedding (pixels / 255, H,W,C order) with bias plus a
                             learned position embedding, vit_layers pre-norm blocks (LayerNorm with
                             bias; multi-head attention with biases in which every patch sees every
                             patch of its view; MLP fc1 -> GELU (tanh form) -> fc2 with biases), a
                             final LayerNorm -- and the projector Linear(vit_dim, d) -> GELU ->
                             Linear(d, d) with biases gives the embedding.  At most 64. */
  int32_t vit_dim;        /* ViT width, a multiple of 64; vit_dim / vit_heads is 64 or 128 */
  int32_t vit_heads;
  int32_t vit_ffn;        /* ViT MLP width, a multiple of 32 */
  float vit_eps;          /* LayerNorm epsilon of the ViT (> 0) */
} gvc_desc;

/* bf16 weights of one decoder layer, canonical [out_features][in_features]. */
typedef struct gvc_layer_weights {
  const void* wq;         /* dev bf16 [d][d] */
  const void* wk;         /* dev bf16 [d][d] */
  const void* wv;         /* dev bf16 [d][d] */
  const void* wo;         /* dev bf16 [d][d] */
  const void* wg;         /* dev bf16 [F][d]  SwiGLU gate */
  const void* wu;         /* dev bf16 [F][d]  SwiGLU up */
  const void* wd;         /* dev bf16 [d][F]  SwiGLU down */
  const void* attn_norm;  /* dev bf16 [d] RMSNorm gain before attention */
  const void* ffn_norm;   /* dev bf16 [d] RMSNorm gain before the FFN */
} gvc_layer_weights;

/* bf16 weights of one ViT block, matrices [out_features][in_features]
 * (Dv = vit_dim, Fv = vit_ffn); vectors hold Dv values unless noted. */
typedef struct gvc_vit_layer_weights {
  const void* ln1_g; const void* ln1_b;   /* LayerNorm before attention */
  const void* wq; const void* bq;         /* [Dv][Dv], [Dv] */
  const void* wk; const void* bk;
  const void* wv; const void* bv;
  const void* wo; const void* bo;
  const void* ln2_g; const void* ln2_b;   /* LayerNorm before the MLP */
  const void* w1; const void* b1;         /* [Fv][Dv], [Fv] */
  const void* w2; const void* b2;         /* [Dv][Fv], [Dv] */
} gvc_vit_layer_weights;

/* bf16 weights of the vision front end (desc.vit_layers > 0). */
typedef struct gvc_vit_weights {
  const void* patch_w;     /* dev bf16 [Dv][p*p*3], input in a patch's H, W, C order */
  const void* patch_b;     /* dev bf16 [Dv] */
  const void* pos;         /* dev bf16 [(img/p)^2][Dv] position embedding, raster order within a view */
  const void* post_g;      /* dev bf16 [Dv] final LayerNorm */
  const void* post_b;
  const void* proj1;       /* dev bf16 [d][Dv] */
  const void* proj1_b;     /* dev bf16 [d] */
  const void* proj2;       /* dev bf16 [d][d] */
  const void* proj2_b;     /* dev bf16 [d] */
  const gvc_vit_layer_weights* layers; /* host array of vit_layers entries */
} gvc_vit_weights;

typedef struct gvc_weights {
  const void* embed;       /* dev bf16 [V][d] token embedding table */
  const void* patch_proj;  /* dev bf16 [d][p*p*3]: visual row = (pixels/255) . W^T (Sec. III-A);
                              unused (may be NULL) with the vision front end */
  const void* lm_head;     /* dev bf16 [V][d] */
  const void* final_norm;  /* dev bf16 [d] */
  const gvc_layer_weights* layers; /* host array of L entries */
  const gvc_vit_weights* vit;      /* host pointer; NULL unless desc.vit_layers > 0 */
} gvc_weights;

typedef struct gvc_ctx gvc_ctx;

/* Device bytes the caller must provide.  weight_bytes: packed weights (written
 * once by gvc_init_cache); state_bytes: the persistent cache (H, K, V, flags,
 * margins); workspace_bytes: per-step scratch.  Any may be NULL.
 * Errors: GVC_EINVAL for a shape the kernels do not support. */
int32_t gvc_sizes(const gvc_desc* desc, size_t* weight_bytes, size_t* state_bytes,
                  size_t* workspace_bytes);

/* Binds a context to the current GPU and to `stream` (a hipStream_t, NULL =
 * the null stream).  Packs the canonical weights into `weight_arena` (the
 * canonical tensors are not referenced afterwards and may be freed once the
 * stream has run the packing), zeroes the state so every episode starts with
 * an invalid cache (the first step is a full pass, Alg. 1) and zeroes the
 * workspace.  *out receives the context.  Errors: GVC_EINVAL (null pointer,
 * unsupported shape), GVC_ENOMEM (an arena too small), GVC_EDEVICE. */
int32_t gvc_init_cache(const gvc_desc* desc, const gvc_weights* weights,
                       void* weight_arena, size_t weight_bytes,
                       void* state, size_t state_bytes,
                       void* workspace, size_t workspace_bytes,
                       void* stream, gvc_ctx** out);

/* Stage 1 + Stage 2 + applied Stage 3 (Sec. III-B).  frame_t, frame_prev: dev uint8
 * [B][n_views][img][img][3].  A patch (p x p x 3 values, H,W,C order) is static
 * iff its cosine with the same patch of frame_prev exceeds tau_num/tau_den,
 * decided exactly in integer arithmetic (both patches all-zero: static;
 * exactly one all-zero: not static).  With desc.task_topk > 0, once a prompt
 * pass has run, the task_topk patches whose total instruction attention in
 * that pass is highest (fp32 sums in a fixed order, ties to the lower index)
 * are not static (Stage 2).  Static patches are ranked by cosine,
 * highest first, ties to the lower index; layer l reuses the first
 * floor(q_l * |S| / 1000) of them, q_l = reuse_permille[l], or with
 * desc.entropy_reuse, once a prompt pass has run, the per-episode q_l of its
 * attention entropy (Stage 3, computed on the GPU in fp32; readable as
 * GVC_STATE_LAYER_Q; reuse_permille is then still validated but not used).
 * reuse_permille: host int32 [L] in [0, 1000], or NULL for 1000 everywhere.
 * reuse_mask: dev uint8 [B][L][N] out (1 = reuse at that layer).
 * n_static: dev int32 [B] out (|S|, after Stage 2), or NULL.
 * Errors: GVC_EINVAL (null frame/mask, 0 < tau_num <= tau_den violated,
 * permille out of range). */
int32_t gvc_select_static(gvc_ctx* ctx, const uint8_t* frame_t, const uint8_t* frame_prev,
                          int32_t tau_num, int32_t tau_den, const int32_t* reuse_permille,
                          uint8_t* reuse_mask, int32_t* n_static);

/* Allocation-free Stage 1 + applied Stage 3 selection, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation) and hold no context.  Same masks and counts
 * as gvc_select_static with fixed proportions, computed from desc's batch,
 * n_layers, img, patch and n_views only (the other fields are ignored, but
 * task_topk and entropy_reuse must be 0: Stages 2 and 3 need a context's last
 * prompt pass).  frame_t, frame_prev, reuse_permille, reuse_mask and n_static
 * as in gvc_select_static; stream: a hipStream_t (NULL = the null stream) on
 * the current GPU, on which the two kernels are enqueued (asynchronous).
 * Scratch: the per-patch statistics live in a fixed array of 16 x 1024 x 3
 * int32 (192 KiB) that each GPU holds for the life of the process; calls
 * that overlap on one GPU (concurrent streams or threads) race on it.
 * Nothing is allocated.  Errors: GVC_EINVAL (null pointer, bad shape, more
 * than 16 episodes or 1024 patches per frame, tau or permille out of range,
 * Stage 2/3 requested), GVC_EDEVICE. */
int32_t gvc_select_static_noalloc(const gvc_desc* desc, const uint8_t* frame_t, const uint8_t* frame_prev,
                                  int32_t tau_num, int32_t tau_den, const int32_t* reuse_permille,
                                  uint8_t* reuse_mask, int32_t* n_static, void* stream);

/* The prompt pass (Alg. 1, full or partial forward).  frame_t: dev uint8
 * [B][n_views][img][img][3]; text_ids: dev int32 [B][n_text] (ids in [0, V); others are clamped into it);
 * extra_rows: dev fp32 [B][n_proprio + n_action_q][d] given embeddings, or
 * NULL when there are none; reuse_mask: dev uint8 [B][L][N] from
 * gvc_select_static, or NULL for a full pass.  Episodes whose cache is
 * invalid run full whatever the mask says.  A visual token reused at layer l
 * keeps its K/V and its layer-l output from the last pass that computed them;
 * every other row is recomputed and its K/V overwrite the cache.  Afterwards
 * every episode's cache is valid and the head logits are ready for
 * gvc_decode_actions.  Blocks until the per-layer row counts are known.
 * Errors: GVC_EINVAL (null frame or ids, missing extra rows), GVC_EDEVICE. */
int32_t gvc_step_prefill(gvc_ctx* ctx, const uint8_t* frame_t, const int32_t* text_ids,
                         const float* extra_rows, const uint8_t* reuse_mask);

/* Action decode (Sec. III-A; Eq. 1 inputs).  For each of the D positions:
 * greedy token = the highest action-bin logit (ties to the lower id) and
 * margin = p1 - p2 of the two highest bin probabilities under the softmax
 * over the whole vocabulary (over the bins if norm_full_vocab == 0).
 * Autoregressive mode runs D-1 single-token passes feeding back each token
 * (or forced_tokens[b][j] when given); parallel mode reads the action-query
 * rows of the prompt pass.  tokens_out: dev int32 [B][D]; margins_out: dev
 * fp32 [B][D]; logits_out: dev fp32 [B][D][V] or NULL; forced_tokens: dev
 * int32 [B][D] or NULL (a fed-back id outside [0, V) is clamped into it
 * before its embedding row is read).  The margins are also kept in the state for
 * gvc_margin_gate.  Errors: GVC_ESTATE if no prompt pass ran since the last
 * decode, GVC_EINVAL, GVC_EDEVICE. */
int32_t gvc_decode_actions(gvc_ctx* ctx, int32_t* tokens_out, float* margins_out,
                           float* logits_out, const int32_t* forced_tokens);

/* The gate of Alg. 1: m_b = mean (Eq. 1) or min over the last decode's D
 * margins of episode b; fire_b = !(m_b >= theta) (strict <, NaN fires);
 * a fired episode's cache becomes invalid so its next prompt pass is full.
 * force: host int8 [B] (-1: decide, 0: keep, 1: fire) or NULL.
 * margin_out: host fp32 [B]; fire_out: host uint8 [B] (either may be NULL).
 * Synchronizes the stream.  Errors: GVC_ESTATE before any decode, GVC_EINVAL
 * (NaN theta, bad reduce), GVC_EDEVICE. */
int32_t gvc_margin_gate(gvc_ctx* ctx, float theta, int32_t reduce, float* margin_out,
                        uint8_t* fire_out, const int8_t* force);

/* Invalidates episode b's cache (b = -1: all episodes). Errors: GVC_EINVAL. */
int32_t gvc_invalidate(gvc_ctx* ctx, int32_t b);

/* Copies one state item (enum gvc_state_item) of layer `layer` into dst (dev),
 * then synchronizes the stream.  dst_bytes must hold the item.
 * Errors: GVC_EINVAL (bad item/layer, short dst), GVC_EDEVICE. */
int32_t gvc_read_state(gvc_ctx* ctx, int32_t item, int32_t layer, void* dst, size_t dst_bytes);

/* Size in bytes of a state item (see gvc_read_state). */
size_t gvc_state_item_bytes(const gvc_ctx* ctx, int32_t item);

/* Host-side check of the compacted row lists of a prompt pass (Alg. 1,
 * partial forward pass: which rows each layer recomputes).  Row r = b*P + pos
 * is recomputed at layer l unless valid[b] != 0, mask != NULL, 1 <= pos <= N
 * and mask[(b*L + l)*N + pos - 1] != 0.  All pointers are host memory:
 * mask uint8 [B][L][N] or NULL; valid int32 [B]; rows int32 [L][3][B*P]
 * (per layer the row index b*P + pos, the episode b and the position pos of
 * each recomputed row, in increasing row order); counts int32 [L];
 * ep_counts, ep_offsets int32 [L][B] (rows of episode b and the index of its
 * first row in the layer's list).  Returns GVC_OK when every list, count and
 * per-episode entry is exactly what the rule gives; otherwise GVC_EINVAL with
 * the first difference in gvc_last_error.  With GVC_VALIDATE=1 in the
 * environment at gvc_init_cache, gvc_step_prefill copies its lists to the host
 * and runs this check (GVC_EDEVICE on a difference). */
int32_t gvc_check_rows(int32_t B, int32_t L, int32_t N, int32_t P, const uint8_t* mask, const int32_t* valid,
                       const int32_t* rows, const int32_t* counts, const int32_t* ep_counts,
                       const int32_t* ep_offsets);

/* Kernel classes for gvc_profile_begin: the launches of one class are
 * bracketed by HIP events on the context's stream. */
enum gvc_kernel_class {
  GVC_K_DECODE_QKV = 0, GVC_K_DECODE_ATTN = 1, GVC_K_DECODE_O = 2, GVC_K_DECODE_GU = 3,
  GVC_K_DECODE_DOWN = 4, GVC_K_DECODE_HEAD = 5,
  GVC_K_PREFILL_QKV = 6, GVC_K_PREFILL_ATTN = 7, GVC_K_PREFILL_O = 8, GVC_K_PREFILL_GU = 9,
  GVC_K_PREFILL_DOWN = 10, GVC_K_PREFILL_HEAD = 11, GVC_K_EMBED = 12, GVC_K_NORM = 13,
  GVC_K_SELECT = 14, GVC_K_DECODE_PASS = 15, GVC_K_STAGE2 = 16,
  GVC_K_VIT = 17,          /* every launch of the vision front end and the first projector GEMM */
  GVC_K_COUNT = 18
};

/* Starts timing every launch of kernel class `cls` (enum gvc_kernel_class):
 * a start and a stop event are recorded on the context's stream around each
 * such launch, for at most `max_launches` launches.  Creates the events (host
 * call; do not use inside a captured region).  Errors: GVC_EINVAL, GVC_EDEVICE. */
int32_t gvc_profile_begin(gvc_ctx* ctx, int32_t cls, int32_t max_launches);

/* Stops timing, synchronizes the stream and returns the summed elapsed time
 * of the recorded launches (milliseconds) and their count.  Errors:
 * GVC_ESTATE if no profile is running, GVC_EDEVICE. */
int32_t gvc_profile_end(gvc_ctx* ctx, double* total_ms, int32_t* launches);

/* Frees the host context.  Device memory stays with the caller. */
int32_t gvc_destroy(gvc_ctx* ctx);

/* Thread-local text of the last error ("" if none). */
const char* gvc_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* GVC_H */
