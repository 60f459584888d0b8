// GEMM work descriptions (k_gemm.hip and its callers).  Part of
// gvc_kernels.h: include that header, not this one.
#pragma once

namespace gvc {

// ------------------------------------------------------------------ GEMM
// Work units of a GEMM launch.  Pair maps give a workgroup two 16-row weight
// blocks whose epilogue partners share lanes; single maps give it one block.
enum { MAP_PLAIN = 0, MAP_QKV = 1, MAP_GU = 2, MAP_SINGLE = 3, MAP_QKV_SINGLE = 4 };
enum { SK_GU = 0, SK_WIDE = 1, SK_NARROW = 2 };
enum { EPI_QKV = 0, EPI_RESID = 1, EPI_SILU = 2, EPI_STORE = 3, EPI_EMBED = 4, EPI_QKV_RAW = 5, EPI_PATCH = 6,
       EPI_GELU = 7 };

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
  const float2* rope; // [kv_pad][head_dim/2] (cos, sin); nullptr: no rotation
  // fp32 biases added to the accumulators (nullptr: none): per matrix for
  // EPI_QKV, bias[0] for EPI_RESID, EPI_GELU, EPI_PATCH and EPI_EMBED
  const float* bias[3];
  // EPI_EMBED: visual rows are acc * vis_scale (+ bias[0])
  float vis_scale;
  // EPI_PATCH: store[m][f] = acc / 255 + bias[0][f] + pos_tab[rows.pos[m]][f] (ld_store floats per row)
  const float* pos_tab;
  int d, head_dim, n_heads, kv_pad;
  // EPI_RESID: out[row] = resid[row] + acc, rows mapped through rows.idx when *_mapped
  const float* resid; int resid_mapped;
  float* out; int out_mapped;
  // EPI_SILU (gate, up pairs) and EPI_GELU (bias, then GELU): frag-layout
  // bf16 activations with kb_act k-fragments per row block
  bf16* act; int kb_act; int n_feat;
  // EPI_STORE
  float* store; int ld_store;
  // EPI_EMBED
  float* h0; const bf16* embed; const int* text_ids; const float* extra;
  int n_patches, n_text, n_extra, n_vocab;   // text ids are clamped into [0, n_vocab)
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
  // split-k variant (k_gemm_sk + k_gemm_sk_epi): the k range in sk_slices
  // slices of sk_steps k steps, fp32 partial sums part[slice][row][feature]
  // with part_ld features per row (all matrices' blocks, matrix-major) and
  // part_rows rows per slice; sk_groups weight-block groups per slice
  float* part;
  int sk_slices, sk_steps, sk_groups, part_ld, part_rows;
  int big_tw;           // many-row kernel: token blocks per wave (2, 3 or 4), 0 = chosen per launch
  int sk_dx;            // split-k core: 0 = k_gemm_sk, 1 = k_gemm_dx (decoupled weight and token streams)
  int sk_shape;         // k_gemm_dx work split: SK_GU (8 waves x 2 blocks), SK_WIDE (12 x 1),
                        // SK_NARROW (8 x 1); see gemm_sk_group_blocks()
  int sk_tall;          // SK_WIDE / SK_NARROW at 11-18 token blocks: one tile of 18 blocks per
                        // k slice instead of two of 10 (0 = always tiles of 10)
  EpiArgs e;
};

// k-steps per pipelined register chunk for a tile of NT blocks of 16 token rows.
constexpr int gemm_pf(int NT) { return NT == 1 ? 4 : (NT <= 3 ? 4 : (NT <= 6 ? 2 : 1)); }

}  // namespace gvc
