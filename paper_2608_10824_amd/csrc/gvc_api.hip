// Host side of libgvc: shape validation, arena planning, weight packing and
// the per-call launch sequences of the C ABI declared in include/gvc.h.
#include "gvc.h"
#include "gvc_kernels.h"

#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

using namespace gvc;

namespace {

thread_local std::string g_err;

int32_t fail(int32_t code, const std::string& msg) {
  g_err = msg;
  return code;
}

#define HIP_TRY(x)                                                                      \
  do {                                                                                  \
    hipError_t e_ = (x);                                                                \
    if (e_ != hipSuccess) return fail(GVC_EDEVICE, std::string(#x) + ": " + hipGetErrorString(e_)); \
  } while (0)

constexpr size_t kAlign = 256;
constexpr int kMaxNT = 5;   // token blocks per GEMM workgroup (best of 2..16 on the 7B prompt pass)
// Vision front-end launches of up to 256 rows (one view) with at most 64
// weight pairs (the 1024-wide output and fc2 projections): tiles of 2 token
// blocks, twice the workgroups of 4-block tiles (ViT-L: 9.5 -> 6.8 and 16.5
// -> 12.5 us per launch; QKV equal, fc1 slower, 1 or 3 blocks slower).  A
// row's result does not depend on the tile.
constexpr int kVitNT = 2;
constexpr int kBigRows = 1024;  // sessions with at least this many prompt rows use k_gemm_big
// Split-k prompt-pass GEMMs (k_gemm_dx, or k_gemm_sk with GVC_SK_CORE=0) of
// the sessions below kBigRows: k slices fixed per matrix shape.  Gate/up in 2
// slices of 12-block groups, QKV in 4 slices of 12-block groups, the down
// projection in 8 slices of 8-block groups (one weight block per compute
// wave): at the 7B shape 230, 256 and 256 workgroups.  Inside the 7B prompt
// pass at 148 rows this took the pass from 6.48 ms (per-pair kernels for QKV
// and down, 16-block gate/up groups: 172 workgroups) to 5.72 ms; the output
// projection stays on the per-pair kernel (8 slices measured 0.1 ms slower).
constexpr int kSkGuSlices = 2;
constexpr int kSkQkvSlices = 4, kSkDownSlices = 8;

struct Bump {
  size_t off = 0;
  size_t take(size_t bytes) {
    const size_t o = off;
    off += (bytes + kAlign - 1) / kAlign * kAlign;
    return o;
  }
};

struct Packed {
  size_t off = 0;
  int N = 0, K = 0, Nblk = 0, KB = 0;
};

struct Plan {
  gvc_desc d{};
  int B, L, D, H, dh, F, V, N, P, kv_len, kv_pad, head_rows, patch_dim, n_extra, bin_lo;
  int KBd, KBf, KBp, KBx;
  int Mmax, Mp;
  // weight arena
  std::vector<Packed> wq, wk, wv, wo, wg, wu, wd;
  Packed patch, lm;
  size_t embed_off, gains_off, final_gain_off, weight_bytes;
  // state
  size_t H_off, K_off, V_off, valid_off, margins_off, head_logits_off, rowcount_off, tv_off, ent_off, lq_off,
      state_bytes;
  bool stage2;   // task_topk > 0 and at least one instruction token after the image
  bool stage3;   // entropy_reuse and at least one instruction token after the image
  int block_first, block_last;   // bidirectional action block [block_first, P - 1], or empty
  // vision front end (vit_layers > 0): Sv patches per view, E = B * views
  // view passes, Mv = B * N rows; fp32 vectors at vvec_off (see vit_vec_*)
  bool vit = false;
  int Sv = 0, E = 0, Mv = 0, Mvp = 0, Dv = 0, Hv = 0, dhv = 0, Fv = 0, KBv = 0, KBvf = 0, kvpad_v = 0;
  std::vector<Packed> vq, vk, vv, vo, v1, v2;
  Packed vpatch, vproj1, vproj2;
  size_t vvec_off, vrows_off, vepc_off, vepo_off, vx_off, vq_off, vk_off, vv_off, vo_off, vh_off, va_off, vp_off;
  size_t layer_kv_elems;
  // workspace
  size_t rows_off, counts_off, epc_off, epo_off, stats_off, x_off, q_off, o_off, r_off, act_off, xdec_off, xf_off,
      ssq_a_off, ssq_f_off, qraw_off, kraw_off, part_off, part_bytes,
      logits_off, rope_off, decrows_off, headrows_off, tokens_off, gate_m_off, gate_f_off, qkv3_off, bar_off,
      hpart_off, ws_bytes;
};

Packed plan_packed(Bump& a, int N, int K) {
  Packed p;
  p.N = N; p.K = K;
  p.Nblk = (N + 15) / 16;
  p.KB = (K + 31) / 32;
  p.off = a.take((size_t)p.Nblk * 16 * p.KB * 32 * 2);
  return p;
}

// fp32 vectors of the vision front end, in floats from vvec_off: patch bias
// [Dv], position table [Sv][Dv], final LayerNorm gain and bias [Dv], projector
// biases [d] and [d]; then per block ln1 gain, ln1 bias, bq, bk, bv, bo, ln2
// gain, ln2 bias, b2 (each [Dv]) and b1 [Fv].
size_t vit_vec_glob(const Plan& p) { return (size_t)p.Dv * (3 + p.Sv) + 2 * (size_t)p.d.d_model; }
size_t vit_vec_floats(const Plan& p) { return vit_vec_glob(p) + (size_t)p.d.vit_layers * (9 * p.Dv + p.Fv); }
enum { VV_LN1G = 0, VV_LN1B, VV_BQ, VV_BK, VV_BV, VV_BO, VV_LN2G, VV_LN2B, VV_B2, VV_B1 };
// offset (floats) of vector `which` of ViT block l
size_t vit_vec_layer(const Plan& p, int l, int which) {
  return vit_vec_glob(p) + (size_t)l * (9 * p.Dv + p.Fv) + (size_t)which * p.Dv;
}

int32_t make_plan(const gvc_desc* dsc, Plan& p) {
  if (!dsc) return fail(GVC_EINVAL, "null desc");
  const gvc_desc& d = *dsc;
  p.d = d;
  // the batched decode folds each RMSNorm into GEMMs over one 16-row token block
  if (d.batch < 1 || d.batch > 16) return fail(GVC_EINVAL, "batch must be in [1, 16]");
  if (d.n_layers < 1 || d.n_layers > 128) return fail(GVC_EINVAL, "n_layers must be in [1, 128]");
  if (d.d_model < 64 || d.d_model % 64) return fail(GVC_EINVAL, "d_model must be a positive multiple of 64");
  if (d.n_heads < 1 || d.d_model % d.n_heads) return fail(GVC_EINVAL, "n_heads must divide d_model");
  const int dh = d.d_model / d.n_heads;
  if (dh != 64 && dh != 128) return fail(GVC_EINVAL, "head_dim must be 64 or 128");
  if (d.ffn < 16 || d.ffn % 16) return fail(GVC_EINVAL, "ffn must be a positive multiple of 16");
  if (d.n_bins < 2 || d.n_bins > d.vocab || d.vocab % 16) return fail(GVC_EINVAL, "bad vocab / n_bins");
  if (d.patch < 1 || d.img < d.patch || d.img % d.patch) return fail(GVC_EINVAL, "img must be a multiple of patch");
  if (d.n_views < 1) return fail(GVC_EINVAL, "n_views must be >= 1");
  if (d.n_text < 1 || d.n_proprio < 0 || d.n_action_q < 0) return fail(GVC_EINVAL, "bad token counts");
  if (d.n_decode < 1) return fail(GVC_EINVAL, "n_decode must be >= 1");
  if (d.parallel_decode && d.n_action_q != d.n_decode)
    return fail(GVC_EINVAL, "parallel decode needs n_action_q == n_decode");
  if (!(d.rms_eps >= 0.f) || !(d.rope_theta > 0.f)) return fail(GVC_EINVAL, "bad rms_eps / rope_theta");
  p.B = d.batch; p.L = d.n_layers; p.D = d.n_decode; p.H = d.n_heads; p.dh = dh; p.F = d.ffn; p.V = d.vocab;
  const int side = d.img / d.patch;
  p.N = d.n_views * side * side;
  if (p.N > 1024) return fail(GVC_EINVAL, "at most 1024 patches per frame");
  p.n_extra = d.n_proprio + d.n_action_q;
  p.P = p.N + d.n_text + p.n_extra;
  p.kv_len = d.parallel_decode ? p.P : p.P + p.D - 1;
  p.kv_pad = (p.kv_len + 31) / 32 * 32;
  if (p.kv_pad > 8192) return fail(GVC_EINVAL, "sequence too long");
  if (d.task_topk < 0 || d.task_topk > p.N) return fail(GVC_EINVAL, "task_topk must lie in [0, N]");
  if (d.entropy_reuse != 0 && d.entropy_reuse != 1) return fail(GVC_EINVAL, "entropy_reuse must be 0 or 1");
  if (d.action_bidir != 0 && d.action_bidir != 1) return fail(GVC_EINVAL, "action_bidir must be 0 or 1");
  if (d.action_bidir && (!d.parallel_decode || d.n_action_q < 1))
    return fail(GVC_EINVAL, "action_bidir needs parallel_decode and n_action_q >= 1");
  p.block_first = d.action_bidir ? p.P - d.n_action_q : p.P;
  p.block_last = p.P - 1;
  if (d.vit_layers < 0 || d.vit_layers > 64) return fail(GVC_EINVAL, "vit_layers must be in [0, 64]");
  p.vit = d.vit_layers > 0;
  if (p.vit) {
    if (d.vit_dim < 64 || d.vit_dim % 64 || d.vit_dim > 8192)
      return fail(GVC_EINVAL, "vit_dim must be a multiple of 64 in [64, 8192]");
    if (d.vit_heads < 1 || d.vit_dim % d.vit_heads) return fail(GVC_EINVAL, "vit_heads must divide vit_dim");
    p.dhv = d.vit_dim / d.vit_heads;
    if (p.dhv != 64 && p.dhv != 128) return fail(GVC_EINVAL, "vit_dim / vit_heads must be 64 or 128");
    if (d.vit_ffn < 32 || d.vit_ffn % 32 || d.vit_ffn > 32768)
      return fail(GVC_EINVAL, "vit_ffn must be a multiple of 32 in [32, 32768]");
    if (!(d.vit_eps > 0.f)) return fail(GVC_EINVAL, "vit_eps must be > 0");
    p.Sv = side * side;
    p.E = d.batch * d.n_views;
    p.Mv = d.batch * p.N;
    p.Mvp = (p.Mv + 15) / 16 * 16;
    p.Dv = d.vit_dim; p.Hv = d.vit_heads; p.Fv = d.vit_ffn;
    p.KBv = p.Dv / 32; p.KBvf = p.Fv / 32;
    p.kvpad_v = (p.Sv + 31) / 32 * 32;
  }
  p.stage2 = d.task_topk > 0 && d.n_text >= 2;
  p.stage3 = d.entropy_reuse && d.n_text >= 2;
  if ((p.stage2 || p.stage3) && (d.n_text - 1 > 32 || p.N + d.n_text >= 640 || (dh != 64 && dh != 128)))
    return fail(GVC_EINVAL, "Stages 2 and 3 need n_text - 1 <= 32 and N + n_text < 640");
  p.head_rows = d.parallel_decode ? d.n_action_q : 1;
  p.patch_dim = d.patch * d.patch * 3;
  p.bin_lo = d.vocab - d.n_bins;
  p.KBd = d.d_model / 32;
  p.KBf = (d.ffn + 31) / 32;
  p.KBp = (p.patch_dim + 31) / 32;
  p.KBx = std::max(p.KBd, p.KBp);
  p.Mmax = std::max(p.B * p.P, p.B);
  p.Mp = (p.Mmax + 15) / 16 * 16;

  Bump w;
  for (int l = 0; l < p.L; ++l) {
    p.wq.push_back(plan_packed(w, d.d_model, d.d_model));
    p.wk.push_back(plan_packed(w, d.d_model, d.d_model));
    p.wv.push_back(plan_packed(w, d.d_model, d.d_model));
    p.wo.push_back(plan_packed(w, d.d_model, d.d_model));
    p.wg.push_back(plan_packed(w, d.ffn, d.d_model));
    p.wu.push_back(plan_packed(w, d.ffn, d.d_model));
    p.wd.push_back(plan_packed(w, d.d_model, d.ffn));
  }
  p.patch = plan_packed(w, d.d_model, p.patch_dim);
  if (p.vit) {
    for (int l = 0; l < d.vit_layers; ++l) {
      p.vq.push_back(plan_packed(w, p.Dv, p.Dv));
      p.vk.push_back(plan_packed(w, p.Dv, p.Dv));
      p.vv.push_back(plan_packed(w, p.Dv, p.Dv));
      p.vo.push_back(plan_packed(w, p.Dv, p.Dv));
      p.v1.push_back(plan_packed(w, p.Fv, p.Dv));
      p.v2.push_back(plan_packed(w, p.Dv, p.Fv));
    }
    p.vpatch = plan_packed(w, p.Dv, p.patch_dim);
    p.vproj1 = plan_packed(w, d.d_model, p.Dv);
    p.vproj2 = plan_packed(w, d.d_model, d.d_model);
    p.vvec_off = w.take(vit_vec_floats(p) * 4);
  }
  p.lm = plan_packed(w, d.vocab, d.d_model);
  p.embed_off = w.take((size_t)d.vocab * d.d_model * 2);
  p.gains_off = w.take((size_t)p.L * 2 * d.d_model * 4);
  p.final_gain_off = w.take((size_t)d.d_model * 4);
  p.weight_bytes = w.off;

  Bump s;
  p.layer_kv_elems = (size_t)p.B * p.H * p.kv_pad * dh;
  p.H_off = s.take((size_t)(p.L + 1) * p.B * p.P * d.d_model * 4);
  p.K_off = s.take(p.layer_kv_elems * p.L * 2);
  p.V_off = s.take(p.layer_kv_elems * p.L * 2);
  p.valid_off = s.take((size_t)p.B * 4);
  p.margins_off = s.take((size_t)p.B * p.D * 4);
  p.head_logits_off = s.take((size_t)p.B * p.head_rows * p.V * 4);
  p.rowcount_off = s.take((size_t)p.L * 4);
  p.tv_off = s.take(p.stage2 ? (size_t)p.B * p.L * p.H * p.N * 4 : 0);
  p.ent_off = s.take(p.stage3 ? (size_t)p.B * p.L * p.H * 4 : 0);
  p.lq_off = s.take(p.stage3 ? (size_t)p.B * p.L * 4 : 0);
  p.state_bytes = s.off;

  Bump k;
  const size_t tot = (size_t)p.B * p.P;
  p.rows_off = k.take((size_t)p.L * 3 * tot * 4);
  p.counts_off = k.take((size_t)p.L * 4);
  p.epc_off = k.take((size_t)p.L * p.B * 4);
  p.epo_off = k.take((size_t)p.L * p.B * 4);
  p.stats_off = k.take((size_t)p.B * p.N * 3 * 4);
  p.x_off = k.take((size_t)p.Mp * p.KBx * 32 * 2);
  p.q_off = k.take((size_t)p.Mp * d.d_model * 2);
  p.o_off = k.take((size_t)p.Mp * p.KBd * 32 * 2);
  p.r_off = k.take((size_t)p.Mp * d.d_model * 4);
  p.act_off = k.take((size_t)p.Mp * p.KBf * 32 * 2);
  p.xdec_off = k.take((size_t)p.B * d.d_model * 4);
  p.xf_off = k.take((size_t)((p.B + 15) / 16 * 16) * p.KBd * 32 * 2);
  p.qraw_off = k.take((size_t)p.B * d.d_model * 4);
  p.kraw_off = k.take((size_t)p.B * d.d_model * 4);
  p.ssq_a_off = k.take((size_t)p.B * (d.d_model / 16) * 4);
  p.ssq_f_off = k.take((size_t)p.B * (d.d_model / 16) * 4);
  p.logits_off = k.take((size_t)p.B * p.V * 4);
  p.rope_off = k.take((size_t)p.kv_pad * (dh / 2) * 8);
  p.decrows_off = k.take((size_t)p.D * 3 * p.B * 4);
  p.headrows_off = k.take((size_t)3 * p.B * p.head_rows * 4);
  p.tokens_off = k.take((size_t)p.B * p.D * 4);
  p.gate_m_off = k.take((size_t)p.B * 4);
  p.gate_f_off = k.take((size_t)p.B * 4);
  p.qkv3_off = k.take((size_t)3 * p.B * d.d_model * 4);
  p.bar_off = k.take((size_t)kDecodeBarWords * 4);
  p.hpart_off = k.take((size_t)kDecodeMaxGrid * 8 * 4);
  {   // split-k partial sums (slices x rows x features) of the largest user:
      // gate/up, QKV or the down projection
    auto nsl = [](int KB, int want) { const int kps = (KB + want - 1) / want; return (size_t)((KB + kps - 1) / kps); };
    const size_t gu = nsl(p.KBd, kSkGuSlices) * 2 * (size_t)((d.ffn + 15) / 16 * 16);
    const size_t qkv = nsl(p.KBd, kSkQkvSlices) * 3 * (size_t)d.d_model;
    const size_t down = nsl(p.KBf, kSkDownSlices) * (size_t)d.d_model;
    p.part_bytes = (size_t)p.Mp * std::max({gu, qkv, down}) * 4;
    p.part_off = k.take(p.part_bytes);
  }
  if (p.vit) {
    const size_t kvv = (size_t)p.E * p.Hv * p.kvpad_v * p.dhv * 2;
    p.vrows_off = k.take((size_t)4 * p.Mv * 4);
    p.vepc_off = k.take((size_t)p.E * 4);
    p.vepo_off = k.take((size_t)p.E * 4);
    p.vx_off = k.take((size_t)p.Mvp * std::max(p.KBv, p.KBp) * 32 * 2);
    p.vq_off = k.take((size_t)p.Mvp * p.Dv * 2);
    p.vk_off = k.take(kvv);
    p.vv_off = k.take(kvv);
    p.vo_off = k.take((size_t)p.Mvp * p.KBv * 32 * 2);
    p.vh_off = k.take((size_t)p.Mvp * p.Dv * 4);
    p.va_off = k.take((size_t)p.Mvp * p.KBvf * 32 * 2);
    p.vp_off = k.take((size_t)p.Mvp * p.KBd * 32 * 2);
  }
  p.ws_bytes = k.off;
  return GVC_OK;
}

}  // namespace

struct gvc_ctx {
  Plan p;
  hipStream_t stream = nullptr;
  int device = 0;
  char* w = nullptr;
  char* st = nullptr;
  char* ws = nullptr;
  bool prefill_done = false;
  bool decode_done = false;
  int force_splits = 0;   // GVC_FORCE_SPLITS: waves splitting each GEMM's k range (4 or 8; testing)
  int big_tw = 0;         // GVC_BIG_TW: tile height of the many-row kernel, 2, 3 or 4 token blocks per wave (testing)
  bool poison = false;    // GVC_POISON: arenas start as 0xFF bytes instead of zeros (testing)
  int validate = 0;       // GVC_VALIDATE: 1 = every prompt pass checks its row lists on the host, 2 = also
                          // alters the host copy first, so the check must fail (tests that it runs)
  // prompt-pass projections on the many-row kernel: sessions of at least
  // kBigRows prompt rows (B * P), for every pass of the session, so a row's
  // result never depends on how many rows a pass recomputes; GVC_GEMM=big
  // or small overrides (testing)
  bool big_gemm = false;
  // the other sessions' gate/up projection on the split-k kernel (GVC_SK=0
  // turns it off: testing)
  bool sk_gemm = true;
  int sk_dx = 1;          // GVC_SK_CORE: split-k core, 1 = k_gemm_dx (decoupled streams), 0 = k_gemm_sk
  // QKV and down projections of those sessions on the one-block-per-wave
  // split-k shapes of the decoupled core (GVC_SK_QKV=0, GVC_SK_DOWN=0 turn
  // them off)
  bool sk_qkv = true, sk_down = true;
  // those shapes at 161-288 rows in one tile of 18 token blocks per k slice
  // (GVC_SK_TALL=0: two tiles of 10, testing)
  bool sk_tall = true;
  // the output projection on the narrow split-k shape where tall tiles apply
  // (GVC_SK_O=0: the per-pair kernel at every height)
  bool sk_o = true;
  // persistent decode pass (k_decode.hip): eligible shape, its grid and LDS
  bool persist = false;
  int persist_wg = 0;
  DecodeArgs dargs{};
  bool persist_ran = false;       // a launch sequence ran since the last check of the abort word
  bool tv_ready = false;          // a prompt pass has written the Stage 2 / Stage 3 signals
  uint32_t abort_word = 0;        // host copy, read by margin_gate
  // launch timing of one kernel class (gvc_profile_begin / _end)
  int prof_cls = -1;
  std::vector<hipEvent_t> prof_ev;
  int prof_n = 0;
  std::vector<int> counts;

  template <class T> T* W(size_t off) const { return reinterpret_cast<T*>(w + off); }
  template <class T> T* S(size_t off) const { return reinterpret_cast<T*>(st + off); }
  template <class T> T* K(size_t off) const { return reinterpret_cast<T*>(ws + off); }
  const bf16x8* packed(const Packed& m) const { return reinterpret_cast<const bf16x8*>(w + m.off); }
  float* H(int l) const { return S<float>(p.H_off) + (size_t)l * p.B * p.P * p.d.d_model; }
  bf16* Kc(int l) const { return S<bf16>(p.K_off) + (size_t)l * p.layer_kv_elems; }
  bf16* Vc(int l) const { return S<bf16>(p.V_off) + (size_t)l * p.layer_kv_elems; }
  RowMap rows(int l) const {
    const int tot = p.B * p.P;
    const int* base = K<int>(p.rows_off) + (size_t)l * 3 * tot;
    return RowMap{base, base + tot, base + 2 * tot};
  }
  RowMap dec_rows(int j) const {
    const int* base = K<int>(p.decrows_off) + (size_t)j * 3 * p.B;
    return RowMap{base, base + p.B, base + 2 * p.B};
  }
  RowMap head_rows() const {
    const int n = p.B * p.head_rows;
    const int* base = K<int>(p.headrows_off);
    return RowMap{base, base + n, base + 2 * n};
  }
};

namespace {

// Token tiling and k split of one GEMM launch: one workgroup per (work
// unit, tile of at most kMaxNT blocks of 16 token rows); its waves split the
// k range 4 ways (8 for long k ranges with few units).  Measured on the 7B
// prompt pass: more concurrent weight streams beat reading the weights once
// per 160 rows (two token groups sharing a k share were 10-50% slower), so
// each token tile streams the weights itself.  8 waves for long k ranges or
// at most 128 units (7B output projection: 24.5 instead of 28 µs).
// GVC_FORCE_SPLITS (4 or 8) overrides the wave count (testing).
void tile_gemm(GemmArgs& a, int M, int force_splits) {
  a.M = M;
  a.mblocks = (M + 15) / 16;
  a.tgroups = 1;
  a.mtiles = (a.mblocks + kMaxNT - 1) / kMaxNT;
  int KW = (a.n_pairs < 256 && (a.KB > 200 || a.n_pairs <= 128)) ? 8 : 4;
  if (force_splits == 4 || force_splits == 8) KW = force_splits;
  a.splits = KW;
  a.kb_per_split = (a.KB + KW - 1) / KW;
}

int nt_of(const GemmArgs& a) {
  return (a.mblocks + a.mtiles * a.tgroups - 1) / (a.mtiles * a.tgroups);
}

// Start / stop events around a launch of class `cls` when it is profiled.
struct ProfScope {
  gvc_ctx* c;
  bool on;
  ProfScope(gvc_ctx* ctx, int cls) : c(ctx), on(ctx->prof_cls == cls && 2 * ctx->prof_n + 1 < (int)ctx->prof_ev.size()) {
    if (on) (void)hipEventRecord(c->prof_ev[2 * c->prof_n], c->stream);
  }
  ~ProfScope() {
    if (on) {
      (void)hipEventRecord(c->prof_ev[2 * c->prof_n + 1], c->stream);
      ++c->prof_n;
    }
  }
};

GemmArgs base_args(const gvc_ctx* c) {
  GemmArgs a;
  memset(&a, 0, sizeof(a));
  a.e.d = c->p.d.d_model;
  a.e.head_dim = c->p.dh;
  a.e.n_heads = c->p.H;
  a.e.kv_pad = c->p.kv_pad;
  a.e.rope = c->K<float2>(c->p.rope_off);
  a.e.vis_scale = 1.0f / 255.0f;
  return a;
}


// Split-k launch of a prompt-pass projection (k_gemm_sk + slice sum and
// epilogue); the slices depend only on the matrix shape.
int32_t run_gemm_sk(gvc_ctx* c, GemmArgs& a, int epi, int M, int cls, int slices, int shape = SK_GU) {
  if (M <= 0) return GVC_OK;
  const Plan& p = c->p;
  a.M = M;
  a.mblocks = (M + 15) / 16;
  const int kps = (a.KB + slices - 1) / slices;
  a.sk_steps = kps;
  a.sk_slices = (a.KB + kps - 1) / kps;
  const int nblk = a.wblk[0] * (a.map == MAP_QKV ? 3 : (a.map == MAP_GU ? 2 : 1));
  const int gb = gemm_sk_group_blocks(shape);
  a.sk_groups = (nblk + gb - 1) / gb;
  a.part = c->K<float>(p.part_off);
  a.sk_dx = c->sk_dx;
  a.sk_shape = shape;
  a.sk_tall = c->sk_tall ? 1 : 0;
  a.part_ld = nblk * 16;
  a.part_rows = a.mblocks * 16;
  if ((size_t)a.sk_slices * a.part_rows * a.part_ld * 4 > p.part_bytes) return fail(GVC_EINVAL, "split-k buffer");
  ProfScope ps(c, cls);
  HIP_TRY(launch_gemm_sk(a, epi, c->stream));
  return GVC_OK;
}

int32_t run_gemm(gvc_ctx* c, GemmArgs& a, int epi, int M, int cls, bool big = false) {
  if (M <= 0) return GVC_OK;
  if (big) {
    a.M = M;
    a.mblocks = (M + 15) / 16;
    a.big_tw = c->big_tw;
    ProfScope ps(c, cls);
    HIP_TRY(launch_gemm_big(a, epi, c->stream));
    return GVC_OK;
  }
  tile_gemm(a, M, c->force_splits);
  if (cls == GVC_K_VIT && a.mblocks <= 16 && a.n_pairs <= 64) a.mtiles = (a.mblocks + kVitNT - 1) / kVitNT;
  // the folded RMSNorm reads at most 16 partial sums per lane, 4 lanes per wave per row
  if (a.e.ssq_in && (a.mblocks > 1 || a.e.ssq_parts > 16 * 4 * a.splits))
    return fail(GVC_EINVAL, "folded norm needs one token block and at most 32 parts per wave");
  ProfScope ps(c, cls);
  HIP_TRY(launch_gemm(a, epi, nt_of(a), c->stream));
  return GVC_OK;
}

// GEMM arguments of a vision front end launch: row width Dv, heads of dhv,
// no rotary embedding.
GemmArgs vit_args(const gvc_ctx* c) {
  GemmArgs a = base_args(c);
  a.e.d = c->p.Dv;
  a.e.head_dim = c->p.dhv;
  a.e.n_heads = c->p.Hv;
  a.e.kv_pad = c->p.kvpad_v;
  a.e.rope = nullptr;
  return a;
}

// The vision front end over every view of frame_t: patch embedding, the ViT
// blocks, the final LayerNorm and the first projector layer (GELU), leaving
// bf16 [B*N][d] in frag layout at vp_off for the embedding step.
int32_t run_vit(gvc_ctx* c, const uint8_t* frame_t) {
  const Plan& p = c->p;
  hipStream_t s = c->stream;
  const int Mv = p.Mv;
  const int* vr = c->K<int>(p.vrows_off);
  const RowMap rows{vr, vr + Mv, vr + 2 * Mv};   // idx (for the patch gather), view pass, position in view
  const int* posl = vr + 3 * Mv;                 // prompt position of the row's visual token
  const float* vec = c->W<float>(p.vvec_off);
  bf16* X = c->K<bf16>(p.vx_off);
  bf16* Q = c->K<bf16>(p.vq_off);
  bf16* Kv = c->K<bf16>(p.vk_off);
  bf16* Vv = c->K<bf16>(p.vv_off);
  bf16* O = c->K<bf16>(p.vo_off);
  float* h = c->K<float>(p.vh_off);
  bf16* A = c->K<bf16>(p.va_off);
  const float eps = p.d.vit_eps;
  {
    ProfScope ps(c, GVC_K_VIT);
    HIP_TRY(launch_im2row(frame_t, p.d.n_views, p.d.img, p.d.patch, rows.idx, posl, Mv, p.P, p.KBp, X, s));
  }
  {
    GemmArgs a = vit_args(c);
    a.w[0] = c->packed(p.vpatch); a.wblk[0] = p.vpatch.Nblk;
    a.map = MAP_PLAIN; a.n_pairs = (p.vpatch.Nblk + 1) / 2; a.n_out = p.Dv; a.KB = p.KBp;
    a.x = reinterpret_cast<const bf16x8*>(X);
    a.e.rows = rows; a.e.store = h; a.e.ld_store = p.Dv; a.e.bias[0] = vec; a.e.pos_tab = vec + p.Dv;
    int32_t r = run_gemm(c, a, EPI_PATCH, Mv, GVC_K_VIT);
    if (r) return r;
  }
  for (int l = 0; l < p.d.vit_layers; ++l) {
    auto V = [&](int which) { return vec + vit_vec_layer(p, l, which); };
    {
      ProfScope ps(c, GVC_K_VIT);
      HIP_TRY(launch_layernorm(h, Mv, p.Dv, V(VV_LN1G), V(VV_LN1B), eps, X, p.KBv, s));
    }
    {
      GemmArgs a = vit_args(c);
      a.w[0] = c->packed(p.vq[l]); a.w[1] = c->packed(p.vk[l]); a.w[2] = c->packed(p.vv[l]);
      a.wblk[0] = a.wblk[1] = a.wblk[2] = p.vq[l].Nblk;
      a.map = MAP_QKV; a.n_pairs = 3 * p.vq[l].Nblk / 2; a.n_out = p.Dv; a.KB = p.KBv;
      a.x = reinterpret_cast<const bf16x8*>(X);
      a.e.rows = rows; a.e.q = Q; a.e.kc = Kv; a.e.vc = Vv;
      a.e.bias[0] = V(VV_BQ); a.e.bias[1] = V(VV_BK); a.e.bias[2] = V(VV_BV);
      int32_t r = run_gemm(c, a, EPI_QKV, Mv, GVC_K_VIT);
      if (r) return r;
    }
    {
      ProfScope ps(c, GVC_K_VIT);
      HIP_TRY(launch_attn_prefill(Q, Kv, Vv, rows.pos, c->K<int>(p.vepc_off), c->K<int>(p.vepo_off), p.E, p.Hv,
                                  p.dhv, p.kvpad_v, (p.Sv + 15) / 16, O, p.KBv, 0, p.Sv - 1, false, s));
    }
    {
      GemmArgs a = vit_args(c);
      a.w[0] = c->packed(p.vo[l]); a.wblk[0] = p.vo[l].Nblk;
      a.map = MAP_PLAIN; a.n_pairs = (p.vo[l].Nblk + 1) / 2; a.n_out = p.Dv; a.KB = p.KBv;
      a.x = reinterpret_cast<const bf16x8*>(O);
      a.e.rows = rows; a.e.resid = h; a.e.out = h; a.e.bias[0] = V(VV_BO);   // in place: each element once
      int32_t r = run_gemm(c, a, EPI_RESID, Mv, GVC_K_VIT);
      if (r) return r;
    }
    {
      ProfScope ps(c, GVC_K_VIT);
      HIP_TRY(launch_layernorm(h, Mv, p.Dv, V(VV_LN2G), V(VV_LN2B), eps, X, p.KBv, s));
    }
    {
      GemmArgs a = vit_args(c);
      a.w[0] = c->packed(p.v1[l]); a.wblk[0] = p.v1[l].Nblk;
      a.map = MAP_PLAIN; a.n_pairs = (p.v1[l].Nblk + 1) / 2; a.n_out = p.Fv; a.KB = p.KBv;
      a.x = reinterpret_cast<const bf16x8*>(X);
      a.e.rows = rows; a.e.act = A; a.e.kb_act = p.KBvf; a.e.n_feat = p.Fv; a.e.bias[0] = V(VV_B1);
      int32_t r = run_gemm(c, a, EPI_GELU, Mv, GVC_K_VIT);
      if (r) return r;
    }
    {
      GemmArgs a = vit_args(c);
      a.w[0] = c->packed(p.v2[l]); a.wblk[0] = p.v2[l].Nblk;
      a.map = MAP_PLAIN; a.n_pairs = (p.v2[l].Nblk + 1) / 2; a.n_out = p.Dv; a.KB = p.KBvf;
      a.x = reinterpret_cast<const bf16x8*>(A);
      a.e.rows = rows; a.e.resid = h; a.e.out = h; a.e.bias[0] = V(VV_B2);
      int32_t r = run_gemm(c, a, EPI_RESID, Mv, GVC_K_VIT);
      if (r) return r;
    }
  }
  const size_t glob_ln = (size_t)p.Dv * (1 + p.Sv);   // final LayerNorm gain, then bias
  {
    ProfScope ps(c, GVC_K_VIT);
    HIP_TRY(launch_layernorm(h, Mv, p.Dv, vec + glob_ln, vec + glob_ln + p.Dv, eps, X, p.KBv, s));
  }
  {
    GemmArgs a = vit_args(c);
    a.w[0] = c->packed(p.vproj1); a.wblk[0] = p.vproj1.Nblk;
    a.map = MAP_PLAIN; a.n_pairs = (p.vproj1.Nblk + 1) / 2; a.n_out = p.d.d_model; a.KB = p.KBv;
    a.x = reinterpret_cast<const bf16x8*>(X);
    a.e.rows = rows; a.e.act = c->K<bf16>(p.vp_off); a.e.kb_act = p.KBd; a.e.n_feat = p.d.d_model;
    a.e.bias[0] = vec + glob_ln + 2 * p.Dv;
    int32_t r = run_gemm(c, a, EPI_GELU, Mv, GVC_K_VIT);
    if (r) return r;
  }
  return GVC_OK;
}

// One decoder layer over M rows: `src` holds the layer input rows (mapped by
// rows.idx when src_mapped), `dst` receives the outputs (same mapping rule).
int32_t run_layer(gvc_ctx* c, int l, const RowMap& rows, int M, float* src, float* dst, bool mapped,
                  int max_tiles, const int* epc, const int* epo) {
  const Plan& p = c->p;
  const float* gains = c->W<float>(p.gains_off) + (size_t)l * 2 * p.d.d_model;
  bf16* X = c->K<bf16>(p.x_off);
  bf16* Q = c->K<bf16>(p.q_off);
  bf16* O = c->K<bf16>(p.o_off);
  float* R = c->K<float>(p.r_off);
  bf16* A = c->K<bf16>(p.act_off);
  const int k0 = GVC_K_PREFILL_QKV;   // class of this layer's QKV launch; the others follow in order
  {
    ProfScope ps(c, GVC_K_NORM);
    HIP_TRY(launch_rmsnorm(src, mapped ? rows.idx : nullptr, M, p.d.d_model, gains, p.d.rms_eps, X, p.KBd,
                           c->big_gemm, c->stream));
  }
  {
    GemmArgs a = base_args(c);
    a.w[0] = c->packed(p.wq[l]); a.w[1] = c->packed(p.wk[l]); a.w[2] = c->packed(p.wv[l]);
    a.wblk[0] = a.wblk[1] = a.wblk[2] = p.wq[l].Nblk;
    a.map = MAP_QKV; a.n_pairs = 3 * p.wq[l].Nblk / 2; a.n_out = p.d.d_model; a.KB = p.KBd;
    a.x = reinterpret_cast<const bf16x8*>(X);
    a.e.rows = rows; a.e.q = Q; a.e.kc = c->Kc(l); a.e.vc = c->Vc(l);
    int32_t r = c->sk_qkv && c->sk_dx && !c->big_gemm ? run_gemm_sk(c, a, EPI_QKV, M, k0, kSkQkvSlices, SK_WIDE)
                                                       : run_gemm(c, a, EPI_QKV, M, k0, c->big_gemm);
    if (r) return r;
  }
  {
    ProfScope ps(c, k0 + 1);
    HIP_TRY(launch_attn_prefill(Q, c->Kc(l), c->Vc(l), rows.pos, epc, epo, p.B, p.H, p.dh, p.kv_pad, max_tiles, O,
                                p.KBd, p.block_first, p.block_last, c->big_gemm, c->stream));
  }
  if (p.stage2 || p.stage3) {   // Stage 2 / 3 signals of this layer, for the next step's selection
    ProfScope ps(c, GVC_K_STAGE2);
    float* tv = p.stage2 ? c->S<float>(p.tv_off) + (size_t)l * p.H * p.N : nullptr;
    float* ent = p.stage3 ? c->S<float>(p.ent_off) + (size_t)l * p.H : nullptr;
    HIP_TRY(launch_text_vis(Q, c->Kc(l), epc, epo, p.B, p.H, p.dh, p.kv_pad, p.N, p.P, p.d.n_text - 1, tv,
                            (size_t)p.L * p.H * p.N, ent, (size_t)p.L * p.H, c->stream));
  }
  {
    GemmArgs a = base_args(c);
    a.w[0] = c->packed(p.wo[l]); a.wblk[0] = p.wo[l].Nblk;
    a.map = MAP_PLAIN; a.n_pairs = (p.wo[l].Nblk + 1) / 2; a.n_out = p.d.d_model; a.KB = p.KBd;
    a.x = reinterpret_cast<const bf16x8*>(O);
    a.e.rows = rows; a.e.resid = src; a.e.resid_mapped = mapped; a.e.out = R; a.e.out_mapped = 0;
    // 8 k slices: the per-pair kernel's 8 k shares, summed in the same order
    const bool o_sk = c->sk_o && c->sk_tall && c->sk_dx && !c->big_gemm && gemm_sk_tall_rows(M);
    int32_t r = o_sk ? run_gemm_sk(c, a, EPI_RESID, M, k0 + 2, kSkDownSlices, SK_NARROW)
                     : run_gemm(c, a, EPI_RESID, M, k0 + 2, c->big_gemm);
    if (r) return r;
  }
  {
    ProfScope ps(c, GVC_K_NORM);
    HIP_TRY(launch_rmsnorm(R, nullptr, M, p.d.d_model, gains + p.d.d_model, p.d.rms_eps, X, p.KBd, c->big_gemm,
                           c->stream));
  }
  {
    GemmArgs a = base_args(c);
    a.w[0] = c->packed(p.wg[l]); a.w[1] = c->packed(p.wu[l]);
    a.wblk[0] = a.wblk[1] = p.wg[l].Nblk;
    a.map = MAP_GU; a.n_pairs = p.wg[l].Nblk; a.n_out = p.F; a.KB = p.KBd;
    a.x = reinterpret_cast<const bf16x8*>(X);
    a.e.rows = rows; a.e.act = A; a.e.kb_act = p.KBf; a.e.n_feat = p.F;
    int32_t r = c->sk_gemm && !c->big_gemm ? run_gemm_sk(c, a, EPI_SILU, M, k0 + 3, kSkGuSlices, c->sk_dx ? SK_WIDE : SK_GU)
                                           : run_gemm(c, a, EPI_SILU, M, k0 + 3, c->big_gemm);
    if (r) return r;
  }
  {
    GemmArgs a = base_args(c);
    a.w[0] = c->packed(p.wd[l]); a.wblk[0] = p.wd[l].Nblk;
    a.map = MAP_PLAIN; a.n_pairs = (p.wd[l].Nblk + 1) / 2; a.n_out = p.d.d_model; a.KB = p.KBf;
    a.x = reinterpret_cast<const bf16x8*>(A);
    a.e.rows = rows; a.e.resid = R; a.e.resid_mapped = 0; a.e.out = dst; a.e.out_mapped = mapped;
    int32_t r = c->sk_down && c->sk_dx && !c->big_gemm
                    ? run_gemm_sk(c, a, EPI_RESID, M, k0 + 4, kSkDownSlices, SK_NARROW)
                    : run_gemm(c, a, EPI_RESID, M, k0 + 4, c->big_gemm);
    if (r) return r;
  }
  return GVC_OK;
}

// One decoder layer of a single-token decode pass over the B rows of xdec,
// with every RMSNorm folded into the GEMMs: the projection input is
// bf16(x * gain) written by the previous epilogue (or the token embedding)
// and the accumulator is scaled by 1/rms from per-workgroup partial sums of
// squares, summed in a fixed order.  ssq_parts_in: parts of the input rows'
// sums of squares (1 after the embedding, d/32 after a down projection).
int32_t run_layer_decode(gvc_ctx* c, int l, const RowMap& rows, int n_keys, int ssq_parts_in) {
  const Plan& p = c->p;
  const int B = p.B, dm = p.d.d_model;
  const float* gains = c->W<float>(p.gains_off) + (size_t)l * 2 * dm;
  const float* next_gain = l + 1 < p.L ? gains + 2 * dm : c->W<float>(p.final_gain_off);
  bf16* X = c->K<bf16>(p.x_off);
  bf16* XF = c->K<bf16>(p.xf_off);
  bf16* O = c->K<bf16>(p.o_off);
  float* R = c->K<float>(p.r_off);
  bf16* A = c->K<bf16>(p.act_off);
  float* xdec = c->K<float>(p.xdec_off);
  float* ssq_a = c->K<float>(p.ssq_a_off);
  float* ssq_f = c->K<float>(p.ssq_f_off);
  const int parts_d = dm / 16;   // one partial sum of squares per 16-row block of the producing GEMM
  float* qraw = c->K<float>(p.qraw_off);
  float* kraw = c->K<float>(p.kraw_off);
  {
    // q and k leave un-rotated in fp32; the decode attention applies RoPE
    GemmArgs a = base_args(c);
    a.w[0] = c->packed(p.wq[l]); a.w[1] = c->packed(p.wk[l]); a.w[2] = c->packed(p.wv[l]);
    a.wblk[0] = a.wblk[1] = a.wblk[2] = p.wq[l].Nblk;
    a.map = MAP_QKV_SINGLE; a.n_pairs = 3 * p.wq[l].Nblk; a.n_out = dm; a.KB = p.KBd;
    a.x = reinterpret_cast<const bf16x8*>(X);
    a.e.rows = rows; a.e.qraw = qraw; a.e.kraw = kraw; a.e.vc = c->Vc(l);
    a.e.ssq_in = ssq_a; a.e.ssq_parts = ssq_parts_in; a.e.norm_eps = p.d.rms_eps; a.e.norm_dim = dm;
    int32_t r = run_gemm(c, a, EPI_QKV_RAW, B, GVC_K_DECODE_QKV);
    if (r) return r;
  }
  {
    ProfScope ps(c, GVC_K_DECODE_ATTN);
    HIP_TRY(launch_attn_decode(qraw, kraw, c->Kc(l), c->Vc(l), c->K<float2>(p.rope_off), B, p.H, p.dh, p.kv_pad,
                               n_keys - 1, O, p.KBd, c->stream));
  }
  {
    GemmArgs a = base_args(c);
    a.w[0] = c->packed(p.wo[l]); a.wblk[0] = p.wo[l].Nblk;
    a.map = MAP_SINGLE; a.n_pairs = p.wo[l].Nblk; a.n_out = dm; a.KB = p.KBd;
    a.x = reinterpret_cast<const bf16x8*>(O);
    a.e.rows = rows; a.e.resid = xdec; a.e.out = R;
    a.e.xn = XF; a.e.xn_gain = gains + dm; a.e.ssq_out = ssq_f; a.e.xn_kb = p.KBd; a.e.ssq_out_parts = parts_d;
    int32_t r = run_gemm(c, a, EPI_RESID, B, GVC_K_DECODE_O);
    if (r) return r;
  }
  {
    GemmArgs a = base_args(c);
    a.w[0] = c->packed(p.wg[l]); a.w[1] = c->packed(p.wu[l]);
    a.wblk[0] = a.wblk[1] = p.wg[l].Nblk;
    a.map = MAP_GU; a.n_pairs = p.wg[l].Nblk; a.n_out = p.F; a.KB = p.KBd;
    a.x = reinterpret_cast<const bf16x8*>(XF);
    a.e.rows = rows; a.e.act = A; a.e.kb_act = p.KBf; a.e.n_feat = p.F;
    a.e.ssq_in = ssq_f; a.e.ssq_parts = parts_d; a.e.norm_eps = p.d.rms_eps; a.e.norm_dim = dm;
    int32_t r = run_gemm(c, a, EPI_SILU, B, GVC_K_DECODE_GU);
    if (r) return r;
  }
  {
    GemmArgs a = base_args(c);
    a.w[0] = c->packed(p.wd[l]); a.wblk[0] = p.wd[l].Nblk;
    a.map = MAP_SINGLE; a.n_pairs = p.wd[l].Nblk; a.n_out = dm; a.KB = p.KBf;
    a.x = reinterpret_cast<const bf16x8*>(A);
    a.e.rows = rows; a.e.resid = R; a.e.out = xdec;
    a.e.xn = X; a.e.xn_gain = next_gain; a.e.ssq_out = ssq_a; a.e.xn_kb = p.KBd; a.e.ssq_out_parts = parts_d;
    int32_t r = run_gemm(c, a, EPI_RESID, B, GVC_K_DECODE_DOWN);
    if (r) return r;
  }
  return GVC_OK;
}

// Final RMSNorm + LM head over M rows of `src` (mapped through rows.idx when given).
int32_t run_head(gvc_ctx* c, const RowMap& rows, const float* src, int M, float* logits, int cls) {
  const Plan& p = c->p;
  bf16* X = c->K<bf16>(p.x_off);
  {
    ProfScope ps(c, GVC_K_NORM);
    HIP_TRY(launch_rmsnorm(src, rows.idx, M, p.d.d_model, c->W<float>(p.final_gain_off), p.d.rms_eps, X, p.KBd,
                           c->big_gemm, c->stream));
  }
  GemmArgs a = base_args(c);
  a.w[0] = c->packed(p.lm); a.wblk[0] = p.lm.Nblk;
  a.map = MAP_PLAIN; a.n_pairs = (p.lm.Nblk + 1) / 2; a.n_out = p.V; a.KB = p.KBd;
  a.x = reinterpret_cast<const bf16x8*>(X);
  a.e.rows = rows; a.e.store = logits; a.e.ld_store = p.V;
  return run_gemm(c, a, EPI_STORE, M, cls);
}

}  // namespace

extern "C" {

const char* gvc_last_error(void) { return g_err.c_str(); }

int32_t gvc_sizes(const gvc_desc* desc, size_t* weight_bytes, size_t* state_bytes, size_t* workspace_bytes) {
  Plan p;
  int32_t r = make_plan(desc, p);
  if (r) return r;
  if (weight_bytes) *weight_bytes = p.weight_bytes;
  if (state_bytes) *state_bytes = p.state_bytes;
  if (workspace_bytes) *workspace_bytes = p.ws_bytes;
  return GVC_OK;
}

namespace {

// The persistent decode pass serves one episode with sequential decoding,
// when every layer's packed matrices sit at one uniform stride, each
// workgroup's share of a step fits kDecodeMaxSeg blocks and the grid of one
// workgroup per compute unit can be co-resident.  GVC_DECODE=legacy turns
// it off (per-step launches).
bool setup_persist(gvc_ctx* c) {
  const Plan& p = c->p;
  const char* mode = getenv("GVC_DECODE");
  if (mode && strcmp(mode, "legacy") == 0) return false;
  if (p.B != 1 || p.d.parallel_decode || p.D < 2) return false;
  const int d = p.d.d_model, F = p.F;
  if (d % 256 || d > 4096 || F > 16384 || (p.dh != 64 && p.dh != 128) || F % 16) return false;
  const size_t u = sizeof(bf16x8);
  auto at = [&](const Packed& m) { return (long long)(m.off / u); };
  const long long qkv_stride = at(p.wk[0]) - at(p.wq[0]), gu_stride = at(p.wu[0]) - at(p.wg[0]);
  const long long layer_stride = p.L > 1 ? at(p.wq[1]) - at(p.wq[0]) : 0;
  for (int l = 0; l < p.L; ++l) {
    const long long s = l * layer_stride;
    if (at(p.wq[l]) != at(p.wq[0]) + s || at(p.wk[l]) != at(p.wq[l]) + qkv_stride ||
        at(p.wv[l]) != at(p.wq[l]) + 2 * qkv_stride || at(p.wo[l]) != at(p.wo[0]) + s ||
        at(p.wg[l]) != at(p.wg[0]) + s || at(p.wu[l]) != at(p.wg[l]) + gu_stride || at(p.wd[l]) != at(p.wd[0]) + s)
      return false;
  }
  int G = 0, coop = 0;
  if (hipDeviceGetAttribute(&G, hipDeviceAttributeMultiprocessorCount, c->device) != hipSuccess) return false;
  if (hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, c->device) != hipSuccess || !coop) return false;
  auto ceil_div = [](int a, int b) { return (a + b - 1) / b; };
  if (G < 1 || G > kDecodeMaxGrid || p.H > G || p.H > kDecodeMaxHeads) return false;
  const int n_slices = std::min(G / p.H, d / 16);
  if (3 * ceil_div(p.dh / 16, n_slices) > kDecodeMaxSeg || 2 * ceil_div(F / 16, G) > kDecodeMaxSeg ||
      ceil_div(d / 16, G) > kDecodeMaxSeg || ceil_div(ceil_div(d / 16, n_slices), 8) > kDecodeMaxSeg)
    return false;
  int act = std::max({d * 4, p.KBf * 32 * 2, p.KBd * 32 * 2, decode_pass_score_offset() + p.kv_pad * 4});
  act = (act + 15) / 16 * 16;
  const void* f = decode_pass_kernel(p.dh, d);
  const size_t lds = decode_pass_lds_bytes(act);
  if (hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  int per_cu = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, f, decode_pass_threads(), lds) != hipSuccess ||
      per_cu < 1) {
    (void)hipGetLastError();
    return false;
  }
  DecodeArgs& a = c->dargs;
  memset(&a, 0, sizeof(a));
  a.wq = c->packed(p.wq[0]); a.wo = c->packed(p.wo[0]); a.wg = c->packed(p.wg[0]); a.wd = c->packed(p.wd[0]);
  a.qkv_stride = (size_t)qkv_stride; a.gu_stride = (size_t)gu_stride; a.layer_stride = (size_t)layer_stride;
  a.kc = c->Kc(0); a.vc = c->Vc(0); a.kv_layer_elems = p.layer_kv_elems;
  a.gains = c->W<float>(p.gains_off);
  a.rope = c->K<float2>(p.rope_off);
  a.x = c->K<float>(p.xdec_off);
  a.racc = c->K<unsigned long long>(p.r_off);   // d int64 accumulators (the region holds Mp >= 16 rows of d floats)
  a.qkv = c->K<float>(p.qkv3_off);
  a.act = c->K<bf16>(p.act_off);
  a.bar = c->K<unsigned>(p.bar_off);
  a.timeout_ticks = 50000000;   // 0.5 s at the 100 MHz wall clock
  a.L = p.L; a.d = d; a.F = F; a.H = p.H; a.head_dim = p.dh; a.KBd = p.KBd; a.KBf = p.KBf; a.kv_pad = p.kv_pad;
  a.act_bytes = act;
  a.eps = p.d.rms_eps;
  // Weights are read once per pass: marked non-temporal they stop evicting
  // the activations, barrier words and key/value lines from L2 (7B: 2.93
  // instead of 3.09 ms per pass; warming the keys and values adds 1%).
  // GVC_DECODE_FLAGS overrides the flags (measurement).
  // The LM head and the token choice join the pass when its blocks fit
  // kDecodeMaxSeg per workgroup.
  const bool head = ceil_div(p.lm.Nblk, G) <= kDecodeMaxSeg;
  a.flags = kDecodeNtWeights | kDecodeWarmKv | (head ? kDecodeHead : 0);
  if (const char* e = getenv("GVC_DECODE_FLAGS"))
    a.flags = atoi(e) & (kDecodeNtWeights | kDecodeWarmKv | (head ? kDecodeHead : 0));
  a.wlm = c->packed(p.lm); a.nlm = p.lm.Nblk;
  a.final_gain = c->W<float>(p.final_gain_off);
  a.logits = c->K<float>(p.logits_off);
  a.head_part = c->K<float>(p.hpart_off);
  a.V = p.V; a.bin_lo = p.bin_lo; a.full_vocab = p.d.norm_full_vocab ? 1 : 0;
  c->persist_wg = G;
  return true;
}

}  // namespace

int32_t gvc_init_cache(const gvc_desc* desc, const gvc_weights* wt, void* weight_arena, size_t weight_bytes,
                       void* state, size_t state_bytes, void* workspace, size_t workspace_bytes, void* stream,
                       gvc_ctx** out) {
  if (!out) return fail(GVC_EINVAL, "null out");
  *out = nullptr;
  Plan p;
  int32_t r = make_plan(desc, p);
  if (r) return r;
  if (!wt || !wt->embed || (!wt->patch_proj && !p.vit) || !wt->lm_head || !wt->final_norm || !wt->layers)
    return fail(GVC_EINVAL, "null weight pointer");
  if (p.vit) {
    const gvc_vit_weights* vw = wt->vit;
    if (!vw || !vw->patch_w || !vw->patch_b || !vw->pos || !vw->post_g || !vw->post_b || !vw->proj1 ||
        !vw->proj1_b || !vw->proj2 || !vw->proj2_b || !vw->layers)
      return fail(GVC_EINVAL, "null vision front end weight pointer");
    for (int l = 0; l < p.d.vit_layers; ++l) {
      const gvc_vit_layer_weights& v = vw->layers[l];
      const void* ptrs[16] = {v.ln1_g, v.ln1_b, v.wq, v.bq, v.wk, v.bk, v.wv, v.bv,
                              v.wo, v.bo, v.ln2_g, v.ln2_b, v.w1, v.b1, v.w2, v.b2};
      for (const void* q : ptrs)
        if (!q) return fail(GVC_EINVAL, "null vision front end weight pointer at block " + std::to_string(l));
    }
  }
  for (int l = 0; l < p.L; ++l) {
    const gvc_layer_weights& lw = wt->layers[l];
    if (!lw.wq || !lw.wk || !lw.wv || !lw.wo || !lw.wg || !lw.wu || !lw.wd || !lw.attn_norm || !lw.ffn_norm)
      return fail(GVC_EINVAL, "null layer weight pointer at layer " + std::to_string(l));
  }
  if (!weight_arena || !state || !workspace) return fail(GVC_EINVAL, "null arena");
  if (((uintptr_t)weight_arena | (uintptr_t)state | (uintptr_t)workspace) % kAlign)
    return fail(GVC_EINVAL, "arenas must be 256-byte aligned");
  if (weight_bytes < p.weight_bytes || state_bytes < p.state_bytes || workspace_bytes < p.ws_bytes)
    return fail(GVC_ENOMEM, "arena smaller than gvc_sizes reported");

  gvc_ctx* c = new gvc_ctx();
  c->p = p;
  c->stream = reinterpret_cast<hipStream_t>(stream);
  c->w = static_cast<char*>(weight_arena);
  c->st = static_cast<char*>(state);
  c->ws = static_cast<char*>(workspace);
  c->counts.assign(p.L, 0);
  auto bail = [&](int32_t code) { delete c; return code; };
  hipStream_t s = c->stream;
  const int dm = p.d.d_model;

#define INIT_TRY(x)                                                                                   \
  do {                                                                                                \
    hipError_t e_ = (x);                                                                              \
    if (e_ != hipSuccess) return bail(fail(GVC_EDEVICE, std::string(#x) + ": " + hipGetErrorString(e_))); \
  } while (0)

  INIT_TRY(hipGetDevice(&c->device));
  if (const char* fs = getenv("GVC_FORCE_SPLITS")) c->force_splits = atoi(fs);
  c->big_gemm = p.B * p.P >= kBigRows;
  if (const char* sk = getenv("GVC_SK")) c->sk_gemm = atoi(sk) != 0;
  if (const char* sc = getenv("GVC_SK_CORE")) c->sk_dx = atoi(sc) != 0;
  if (const char* e = getenv("GVC_SK_QKV")) c->sk_qkv = atoi(e) != 0;
  if (const char* e = getenv("GVC_SK_DOWN")) c->sk_down = atoi(e) != 0;
  if (const char* e = getenv("GVC_SK_TALL")) c->sk_tall = atoi(e) != 0;
  if (const char* e = getenv("GVC_SK_O")) c->sk_o = atoi(e) != 0;
  if (const char* tw = getenv("GVC_BIG_TW")) c->big_tw = atoi(tw);
  if (const char* g = getenv("GVC_GEMM")) {
    if (!strcmp(g, "big")) c->big_gemm = true;
    if (!strcmp(g, "small")) c->big_gemm = false;
  }
  // GVC_POISON=1 (testing): every state and workspace byte starts as 0xFF
  // (NaN in fp32 and bf16, -1 in int32) instead of 0, except what the library
  // relies on starting at zero: the cache-valid flags, the decode barrier
  // words, the key/value positions past the prompt (the prompt attention's
  // last key tile reads them with zero weight) and, when the FFN width is not
  // a multiple of 32, the activation fragments' padding columns.  A step that
  // reads anything else before writing it then yields NaN.
  if (const char* pz = getenv("GVC_POISON")) c->poison = atoi(pz) != 0;
  if (const char* va = getenv("GVC_VALIDATE")) c->validate = atoi(va);
  const uint32_t fill = c->poison ? 0xFFFFFFFFu : 0u;
  INIT_TRY(launch_fill_u32(reinterpret_cast<uint32_t*>(c->st), fill, p.state_bytes / 4, s));
  INIT_TRY(launch_fill_u32(reinterpret_cast<uint32_t*>(c->ws), fill, p.ws_bytes / 4, s));
  if (c->poison) {
    INIT_TRY(launch_fill_u32(c->S<uint32_t>(p.valid_off), 0u, p.B, s));
    INIT_TRY(launch_fill_u32(c->K<uint32_t>(p.bar_off), 0u, kDecodeBarWords, s));
    INIT_TRY(launch_zero_kv_tail(c->S<bf16>(p.K_off), c->S<bf16>(p.V_off), (size_t)p.L * p.B * p.H, p.kv_pad, p.dh,
                                 p.P, s));
    if (p.d.ffn % 32)
      INIT_TRY(launch_fill_u32(c->K<uint32_t>(p.act_off), 0u, (size_t)p.Mp * p.KBf * 32 / 2, s));
    if (p.vit)
      INIT_TRY(launch_zero_kv_tail(c->K<bf16>(p.vk_off), c->K<bf16>(p.vv_off), (size_t)p.E * p.Hv, p.kvpad_v, p.dhv,
                                   p.Sv, s));
  }
  for (int l = 0; l < p.L; ++l) {
    const gvc_layer_weights& lw = wt->layers[l];
    const Packed* mats[7] = {&p.wq[l], &p.wk[l], &p.wv[l], &p.wo[l], &p.wg[l], &p.wu[l], &p.wd[l]};
    const void* srcs[7] = {lw.wq, lw.wk, lw.wv, lw.wo, lw.wg, lw.wu, lw.wd};
    for (int i = 0; i < 7; ++i)
      INIT_TRY(launch_pack(static_cast<const bf16*>(srcs[i]), mats[i]->N, mats[i]->K, c->W<bf16>(mats[i]->off),
                           mats[i]->Nblk, mats[i]->KB, s));
    float* g = c->W<float>(p.gains_off) + (size_t)l * 2 * dm;
    INIT_TRY(launch_convert_gain(static_cast<const bf16*>(lw.attn_norm), g, dm, s));
    INIT_TRY(launch_convert_gain(static_cast<const bf16*>(lw.ffn_norm), g + dm, dm, s));
  }
  if (wt->patch_proj)
    INIT_TRY(launch_pack(static_cast<const bf16*>(wt->patch_proj), p.patch.N, p.patch.K, c->W<bf16>(p.patch.off),
                         p.patch.Nblk, p.patch.KB, s));
  if (p.vit) {
    const gvc_vit_weights* vw = wt->vit;
    auto pack = [&](const void* src, const Packed& m) {
      return launch_pack(static_cast<const bf16*>(src), m.N, m.K, c->W<bf16>(m.off), m.Nblk, m.KB, s);
    };
    float* vec = c->W<float>(p.vvec_off);
    auto cvt = [&](const void* src, size_t off, int n) {
      return launch_convert_gain(static_cast<const bf16*>(src), vec + off, n, s);
    };
    const int Dv = p.Dv;
    INIT_TRY(pack(vw->patch_w, p.vpatch));
    INIT_TRY(pack(vw->proj1, p.vproj1));
    INIT_TRY(pack(vw->proj2, p.vproj2));
    INIT_TRY(cvt(vw->patch_b, 0, Dv));
    INIT_TRY(cvt(vw->pos, Dv, p.Sv * Dv));
    INIT_TRY(cvt(vw->post_g, (size_t)Dv * (1 + p.Sv), Dv));
    INIT_TRY(cvt(vw->post_b, (size_t)Dv * (2 + p.Sv), Dv));
    INIT_TRY(cvt(vw->proj1_b, (size_t)Dv * (3 + p.Sv), dm));
    INIT_TRY(cvt(vw->proj2_b, (size_t)Dv * (3 + p.Sv) + dm, dm));
    for (int l = 0; l < p.d.vit_layers; ++l) {
      const gvc_vit_layer_weights& v = vw->layers[l];
      INIT_TRY(pack(v.wq, p.vq[l]));
      INIT_TRY(pack(v.wk, p.vk[l]));
      INIT_TRY(pack(v.wv, p.vv[l]));
      INIT_TRY(pack(v.wo, p.vo[l]));
      INIT_TRY(pack(v.w1, p.v1[l]));
      INIT_TRY(pack(v.w2, p.v2[l]));
      const void* vecs[9] = {v.ln1_g, v.ln1_b, v.bq, v.bk, v.bv, v.bo, v.ln2_g, v.ln2_b, v.b2};
      for (int i = 0; i < 9; ++i) INIT_TRY(cvt(vecs[i], vit_vec_layer(p, l, i), Dv));
      INIT_TRY(cvt(v.b1, vit_vec_layer(p, l, VV_B1), p.Fv));
    }
    // rows of the front end: visual token n of episode b is row b*N + n, in
    // view pass e = b*views + n / Sv at position n % Sv
    std::vector<int> vr((size_t)4 * p.Mv), epc(p.E, p.Sv), epo(p.E);
    for (int b = 0; b < p.B; ++b)
      for (int n = 0; n < p.N; ++n) {
        const int m = b * p.N + n;
        vr[m] = b * p.P + 1 + n;
        vr[p.Mv + m] = b * p.d.n_views + n / p.Sv;
        vr[2 * p.Mv + m] = n % p.Sv;
        vr[3 * p.Mv + m] = 1 + n;
      }
    for (int e = 0; e < p.E; ++e) epo[e] = e * p.Sv;
    INIT_TRY(hipMemcpyAsync(c->K<int>(p.vrows_off), vr.data(), vr.size() * 4, hipMemcpyHostToDevice, s));
    INIT_TRY(hipMemcpyAsync(c->K<int>(p.vepc_off), epc.data(), epc.size() * 4, hipMemcpyHostToDevice, s));
    INIT_TRY(hipMemcpyAsync(c->K<int>(p.vepo_off), epo.data(), epo.size() * 4, hipMemcpyHostToDevice, s));
    INIT_TRY(hipStreamSynchronize(s));   // the host vectors end here
  }
  INIT_TRY(launch_pack(static_cast<const bf16*>(wt->lm_head), p.lm.N, p.lm.K, c->W<bf16>(p.lm.off), p.lm.Nblk,
                       p.lm.KB, s));
  INIT_TRY(hipMemcpyAsync(c->W<char>(p.embed_off), wt->embed, (size_t)p.V * dm * 2, hipMemcpyDeviceToDevice, s));
  INIT_TRY(launch_convert_gain(static_cast<const bf16*>(wt->final_norm), c->W<float>(p.final_gain_off), dm, s));
  INIT_TRY(launch_rope_table(c->K<float2>(p.rope_off), p.kv_pad, p.dh, p.d.rope_theta, s));

  // static row maps: decode pass j (token at position P + j - 1) and the head rows
  std::vector<int> dec((size_t)p.D * 3 * p.B), head((size_t)3 * p.B * p.head_rows);
  for (int j = 0; j < p.D; ++j)
    for (int b = 0; b < p.B; ++b) {
      dec[((size_t)j * 3 + 0) * p.B + b] = b;
      dec[((size_t)j * 3 + 1) * p.B + b] = b;
      dec[((size_t)j * 3 + 2) * p.B + b] = p.P + j - 1;
    }
  const int nh = p.B * p.head_rows;
  for (int b = 0; b < p.B; ++b)
    for (int i = 0; i < p.head_rows; ++i) {
      const int pos = p.d.parallel_decode ? p.N + p.d.n_text + p.d.n_proprio + i : p.P - 1;
      const int r = b * p.head_rows + i;
      head[r] = b * p.P + pos;
      head[nh + r] = b;
      head[2 * nh + r] = pos;
    }
  INIT_TRY(hipMemcpyAsync(c->K<int>(p.decrows_off), dec.data(), dec.size() * 4, hipMemcpyHostToDevice, s));
  INIT_TRY(hipMemcpyAsync(c->K<int>(p.headrows_off), head.data(), head.size() * 4, hipMemcpyHostToDevice, s));
  INIT_TRY(hipStreamSynchronize(s));
  c->persist = setup_persist(c);
#undef INIT_TRY
  *out = c;
  return GVC_OK;
}

int32_t gvc_select_static(gvc_ctx* c, const uint8_t* frame_t, const uint8_t* frame_prev, int32_t tau_num,
                          int32_t tau_den, const int32_t* reuse_permille, uint8_t* reuse_mask, int32_t* n_static) {
  if (!c || !frame_t || !frame_prev || !reuse_mask) return fail(GVC_EINVAL, "null argument");
  if (!(tau_num > 0 && tau_num <= tau_den && tau_den <= (1 << 20)))
    return fail(GVC_EINVAL, "tau must satisfy 0 < num <= den <= 2^20");
  const Plan& p = c->p;
  std::vector<int> q(p.L, 1000);
  if (reuse_permille)
    for (int l = 0; l < p.L; ++l) {
      if (reuse_permille[l] < 0 || reuse_permille[l] > 1000) return fail(GVC_EINVAL, "permille out of [0, 1000]");
      q[l] = reuse_permille[l];
    }
  int* stats = c->K<int>(p.stats_off);
  ProfScope ps(c, GVC_K_SELECT);
  HIP_TRY(launch_patch_stats(frame_t, frame_prev, p.B, p.d.n_views, p.d.img, p.d.patch, stats, c->stream));
  const float* tv = p.stage2 && c->tv_ready ? c->S<float>(p.tv_off) : nullptr;
  const float* ent = p.stage3 && c->tv_ready ? c->S<float>(p.ent_off) : nullptr;
  HIP_TRY(launch_rank_mask(stats, p.B, p.N, p.L, tau_num, tau_den, q.data(), reuse_mask, n_static, tv, p.L * p.H,
                           p.d.task_topk, ent, p.H, p.d.n_text - 1, ent ? c->S<int>(p.lq_off) : nullptr,
                           c->stream));
  return GVC_OK;
}

int32_t gvc_select_static_noalloc(const gvc_desc* desc, const uint8_t* frame_t, const uint8_t* frame_prev,
                                  int32_t tau_num, int32_t tau_den, const int32_t* reuse_permille,
                                  uint8_t* reuse_mask, int32_t* n_static, void* stream) {
  if (!desc || !frame_t || !frame_prev || !reuse_mask) return fail(GVC_EINVAL, "null argument");
  const gvc_desc& d = *desc;
  if (d.batch < 1 || d.n_layers < 1 || d.n_layers > 128) return fail(GVC_EINVAL, "batch >= 1 and n_layers in [1, 128]");
  if (d.patch < 1 || d.img < d.patch || d.img % d.patch) return fail(GVC_EINVAL, "img must be a multiple of patch");
  if (d.n_views < 1) return fail(GVC_EINVAL, "n_views must be >= 1");
  if (d.task_topk != 0 || d.entropy_reuse != 0)
    return fail(GVC_EINVAL, "Stages 2 and 3 need the previous prompt pass: use gvc_select_static");
  const long long side = d.img / d.patch, N = (long long)d.n_views * side * side;
  if (d.batch > kSelectScratchEpisodes || N > kSelectScratchPatches)
    return fail(GVC_EINVAL, "the allocation-free selection takes at most " + std::to_string(kSelectScratchEpisodes) +
                                " episodes of " + std::to_string(kSelectScratchPatches) + " patches");
  if (!(tau_num > 0 && tau_num <= tau_den && tau_den <= (1 << 20)))
    return fail(GVC_EINVAL, "tau must satisfy 0 < num <= den <= 2^20");
  std::vector<int> q(d.n_layers, 1000);
  if (reuse_permille)
    for (int l = 0; l < d.n_layers; ++l) {
      if (reuse_permille[l] < 0 || reuse_permille[l] > 1000) return fail(GVC_EINVAL, "permille out of [0, 1000]");
      q[l] = reuse_permille[l];
    }
  int* stats = nullptr;
  HIP_TRY(select_scratch(&stats));
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  HIP_TRY(launch_patch_stats(frame_t, frame_prev, d.batch, d.n_views, d.img, d.patch, stats, s));
  HIP_TRY(launch_rank_mask(stats, d.batch, (int)N, d.n_layers, tau_num, tau_den, q.data(), reuse_mask, n_static,
                           nullptr, 0, 0, nullptr, 0, 0, nullptr, s));
  return GVC_OK;
}

int32_t gvc_check_rows(int32_t B, int32_t L, int32_t N, int32_t P, const uint8_t* mask, const int32_t* valid,
                       const int32_t* rows, const int32_t* counts, const int32_t* ep_counts,
                       const int32_t* ep_offsets) {
  if (B < 1 || L < 1 || N < 0 || P < 1 || N >= P) return fail(GVC_EINVAL, "bad shape");
  if (!valid || !rows || !counts || !ep_counts || !ep_offsets) return fail(GVC_EINVAL, "null argument");
  const size_t tot = (size_t)B * P;
  for (int l = 0; l < L; ++l) {
    const int32_t* idx = rows + (size_t)l * 3 * tot;
    const int32_t* ep = idx + tot;
    const int32_t* pos = ep + tot;
    auto bad = [&](const std::string& what) {
      return fail(GVC_EINVAL, "layer " + std::to_string(l) + ": " + what);
    };
    size_t n = 0;   // rows the rule recomputes so far
    for (int b = 0; b < B; ++b) {
      const size_t first = n;
      for (int q = 0; q < P; ++q) {
        const bool reused = valid[b] && mask && q >= 1 && q <= N && mask[((size_t)b * L + l) * N + q - 1];
        if (reused) continue;
        if (n >= (size_t)counts[l] || counts[l] > (int32_t)tot)
          return bad("count " + std::to_string(counts[l]) + " misses row " + std::to_string(b * P + q));
        if (idx[n] != b * P + q || ep[n] != b || pos[n] != q)
          return bad("entry " + std::to_string(n) + " is (" + std::to_string(idx[n]) + ", " + std::to_string(ep[n]) +
                     ", " + std::to_string(pos[n]) + "), expected (" + std::to_string(b * P + q) + ", " +
                     std::to_string(b) + ", " + std::to_string(q) + ")");
        ++n;
      }
      if (ep_offsets[l * B + b] != (int32_t)first || ep_counts[l * B + b] != (int32_t)(n - first))
        return bad("episode " + std::to_string(b) + " has offset " + std::to_string(ep_offsets[l * B + b]) +
                   " and count " + std::to_string(ep_counts[l * B + b]) + ", expected " + std::to_string(first) +
                   " and " + std::to_string(n - first));
    }
    if (counts[l] != (int32_t)n)
      return bad("count " + std::to_string(counts[l]) + ", expected " + std::to_string(n));
  }
  return GVC_OK;
}

int32_t gvc_step_prefill(gvc_ctx* c, const uint8_t* frame_t, const int32_t* text_ids, const float* extra_rows,
                         const uint8_t* reuse_mask) {
  if (!c || !frame_t || !text_ids) return fail(GVC_EINVAL, "null argument");
  const Plan& p = c->p;
  if (p.n_extra > 0 && !extra_rows) return fail(GVC_EINVAL, "extra_rows required");
  hipStream_t s = c->stream;
  int* counts = c->K<int>(p.counts_off);
  int* epc = c->K<int>(p.epc_off);
  int* epo = c->K<int>(p.epo_off);
  HIP_TRY(launch_build_rows(reuse_mask, c->S<int>(p.valid_off), p.B, p.L, p.N, p.P, c->K<int>(p.rows_off), counts, epc,
                            epo, s));
  HIP_TRY(hipMemcpyAsync(c->S<int>(p.rowcount_off), counts, (size_t)p.L * 4, hipMemcpyDeviceToDevice, s));
  HIP_TRY(hipMemcpyAsync(c->counts.data(), counts, (size_t)p.L * 4, hipMemcpyDeviceToHost, s));
  HIP_TRY(hipStreamSynchronize(s));
  for (int l = 0; l < p.L; ++l)
    if (c->counts[l] < 1 || c->counts[l] > p.B * p.P) return fail(GVC_EDEVICE, "corrupt row count");
  if (c->validate) {
    const size_t tot = (size_t)p.B * p.P;
    std::vector<int32_t> rows((size_t)p.L * 3 * tot), valid(p.B), epcs((size_t)p.L * p.B), epos((size_t)p.L * p.B);
    std::vector<uint8_t> mask(reuse_mask ? (size_t)p.B * p.L * p.N : 0);
    HIP_TRY(hipMemcpyAsync(rows.data(), c->K<int>(p.rows_off), rows.size() * 4, hipMemcpyDeviceToHost, s));
    HIP_TRY(hipMemcpyAsync(valid.data(), c->S<int>(p.valid_off), valid.size() * 4, hipMemcpyDeviceToHost, s));
    HIP_TRY(hipMemcpyAsync(epcs.data(), epc, epcs.size() * 4, hipMemcpyDeviceToHost, s));
    HIP_TRY(hipMemcpyAsync(epos.data(), epo, epos.size() * 4, hipMemcpyDeviceToHost, s));
    if (reuse_mask) HIP_TRY(hipMemcpyAsync(mask.data(), reuse_mask, mask.size(), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    if (c->validate == 2) rows[0] += 1;
    if (gvc_check_rows(p.B, p.L, p.N, p.P, reuse_mask ? mask.data() : nullptr, valid.data(), rows.data(),
                       c->counts.data(), epcs.data(), epos.data()) != GVC_OK)
      return fail(GVC_EDEVICE, "row lists fail the host check: " + std::string(gvc_last_error()));
  }

  // layer-0 embeddings of the rows recomputed at layer 0
  if (p.vit) {
    int32_t r = run_vit(c, frame_t);
    if (r) return r;
  }
  {
    const RowMap r0 = c->rows(0);
    bf16* X = c->K<bf16>(p.x_off);
    GemmArgs a = base_args(c);
    if (p.vit) {   // visual rows: the projector's second layer over the ViT rows recomputed at layer 0
      HIP_TRY(launch_gather_visual(c->K<bf16>(p.vp_off), r0.idx, r0.pos, c->counts[0], p.P, p.N, p.KBd, X, s));
      a.w[0] = c->packed(p.vproj2); a.wblk[0] = p.vproj2.Nblk;
      a.map = MAP_PLAIN; a.n_pairs = (p.vproj2.Nblk + 1) / 2; a.n_out = p.d.d_model; a.KB = p.KBd;
      a.e.vis_scale = 1.0f;
      a.e.bias[0] = c->W<float>(p.vvec_off) + (size_t)p.Dv * (3 + p.Sv) + p.d.d_model;
    } else {
      HIP_TRY(launch_im2row(frame_t, p.d.n_views, p.d.img, p.d.patch, r0.idx, r0.pos, c->counts[0], p.P, p.KBp, X,
                            s));
      a.w[0] = c->packed(p.patch); a.wblk[0] = p.patch.Nblk;
      a.map = MAP_PLAIN; a.n_pairs = (p.patch.Nblk + 1) / 2; a.n_out = p.d.d_model; a.KB = p.KBp;
    }
    a.x = reinterpret_cast<const bf16x8*>(X);
    a.e.rows = r0; a.e.h0 = c->H(0); a.e.embed = c->W<bf16>(p.embed_off); a.e.text_ids = text_ids; a.e.n_vocab = p.V;
    a.e.extra = extra_rows; a.e.n_patches = p.N; a.e.n_text = p.d.n_text; a.e.n_extra = p.n_extra;
    int32_t r = run_gemm(c, a, EPI_EMBED, c->counts[0], GVC_K_EMBED, c->big_gemm);
    if (r) return r;
  }
  const int max_tiles = (p.P + 15) / 16;
  for (int l = 0; l < p.L; ++l) {
    int32_t r = run_layer(c, l, c->rows(l), c->counts[l], c->H(l), c->H(l + 1), true, max_tiles, epc + l * p.B,
                          epo + l * p.B);
    if (r) return r;
  }
  if (p.stage2 || p.stage3) c->tv_ready = true;
  int32_t r = run_head(c, c->head_rows(), c->H(p.L), p.B * p.head_rows, c->S<float>(p.head_logits_off),
                       GVC_K_PREFILL_HEAD);
  if (r) return r;
  HIP_TRY(launch_fill_u32(reinterpret_cast<uint32_t*>(c->S<int>(p.valid_off)), 1u, p.B, s));
  c->prefill_done = true;
  return GVC_OK;
}

int32_t gvc_decode_actions(gvc_ctx* c, int32_t* tokens_out, float* margins_out, float* logits_out,
                           const int32_t* forced_tokens) {
  if (!c || !tokens_out || !margins_out) return fail(GVC_EINVAL, "null argument");
  if (!c->prefill_done) return fail(GVC_ESTATE, "decode_actions needs a prompt pass first");
  const Plan& p = c->p;
  hipStream_t s = c->stream;
  int* tok = c->K<int>(p.tokens_off);
  float* mg = c->S<float>(p.margins_off);
  const float* hl = c->S<float>(p.head_logits_off);
  const int full = p.d.norm_full_vocab ? 1 : 0;
  if (p.d.parallel_decode) {
    HIP_TRY(launch_logits_reduce(hl, p.B * p.head_rows, p.V, p.bin_lo, full, tok, mg, p.D, 0, p.head_rows, s));
    if (logits_out)
      HIP_TRY(hipMemcpyAsync(logits_out, hl, (size_t)p.B * p.D * p.V * 4, hipMemcpyDeviceToDevice, s));
  } else {
    HIP_TRY(launch_logits_reduce(hl, p.B, p.V, p.bin_lo, full, tok, mg, p.D, 0, 1, s));
    if (logits_out)
      HIP_TRY(hipMemcpy2DAsync(logits_out, (size_t)p.D * p.V * 4, hl, (size_t)p.V * 4, (size_t)p.V * 4, p.B,
                               hipMemcpyDeviceToDevice, s));
    float* xdec = c->K<float>(p.xdec_off);
    float* lg = c->K<float>(p.logits_off);
    for (int j = 1; j < p.D; ++j) {
      const int* src = forced_tokens ? forced_tokens + (j - 1) : tok + (j - 1);
      HIP_TRY(launch_embed_tokens(c->W<bf16>(p.embed_off), src, p.D, p.B, p.d.d_model, p.V, xdec,
                                  c->W<float>(p.gains_off), c->K<bf16>(p.x_off), p.KBd, c->K<float>(p.ssq_a_off), s));
      const RowMap rows = c->dec_rows(j);
      const int pos = p.P + j - 1;
      bool fused = false;   // the decode pass also ran the LM head and the token choice
      GemmArgs hd = base_args(c);
      hd.w[0] = c->packed(p.lm); hd.wblk[0] = p.lm.Nblk;
      hd.map = MAP_PLAIN; hd.n_pairs = (p.lm.Nblk + 1) / 2; hd.n_out = p.V; hd.KB = p.KBd;
      hd.x = c->K<bf16x8>(p.x_off);
      hd.e.rows = rows; hd.e.store = lg; hd.e.ld_store = p.V;
      if (c->persist) {
        // all layers in one cooperative launch, then the final norm and the head
        if (j == 1) {   // every barrier word but the abort word, which stays set until a gate reports it
          HIP_TRY(launch_fill_u32(c->K<uint32_t>(p.bar_off), 0u, kDecodeAbortWord, s));
          HIP_TRY(launch_fill_u32(c->K<uint32_t>(p.bar_off) + kDecodeAbortWord + 1, 0u,
                                  kDecodeBarWords - kDecodeAbortWord - 1, s));
        }
        DecodeArgs a = c->dargs;
        fused = (a.flags & kDecodeHead) != 0;
        a.pos = pos;
        a.bar_base = (unsigned)((j - 1) * decode_grid_barriers(p.L, fused));
        a.hbar_base = (unsigned)((j - 1) * decode_head_barriers(p.L));
        a.tok_out = tok + j;   // B = 1: token j of the episode
        a.margin_out = mg + j;
        {
          ProfScope ps(c, GVC_K_DECODE_PASS);
          HIP_TRY(launch_decode_pass(a, c->persist_wg, s));
        }
        c->persist_ran = true;
        if (!fused) {
          ProfScope ps(c, GVC_K_NORM);
          HIP_TRY(launch_rmsnorm(xdec, nullptr, p.B, p.d.d_model, c->W<float>(p.final_gain_off), p.d.rms_eps,
                                 c->K<bf16>(p.x_off), p.KBd, c->big_gemm, s));
        }
      } else {
        for (int l = 0; l < p.L; ++l) {
          int32_t r = run_layer_decode(c, l, rows, pos + 1, l == 0 ? 1 : p.d.d_model / 16);
          if (r) return r;
        }
        // the LM head reads the folded final norm written by the last down projection
        hd.e.ssq_in = c->K<float>(p.ssq_a_off); hd.e.ssq_parts = p.d.d_model / 16;
        hd.e.norm_eps = p.d.rms_eps; hd.e.norm_dim = p.d.d_model;
      }
      if (!fused) {
        int32_t r = run_gemm(c, hd, EPI_STORE, p.B, GVC_K_DECODE_HEAD);
        if (r) return r;
        HIP_TRY(launch_logits_reduce(lg, p.B, p.V, p.bin_lo, full, tok, mg, p.D, j, 1, s));
      }
      if (logits_out)
        HIP_TRY(hipMemcpy2DAsync(logits_out + (size_t)j * p.V, (size_t)p.D * p.V * 4, lg, (size_t)p.V * 4,
                                 (size_t)p.V * 4, p.B, hipMemcpyDeviceToDevice, s));
    }
  }
  HIP_TRY(hipMemcpyAsync(tokens_out, tok, (size_t)p.B * p.D * 4, hipMemcpyDeviceToDevice, s));
  HIP_TRY(hipMemcpyAsync(margins_out, mg, (size_t)p.B * p.D * 4, hipMemcpyDeviceToDevice, s));
  c->prefill_done = false;
  c->decode_done = true;
  return GVC_OK;
}

int32_t gvc_margin_gate(gvc_ctx* c, float theta, int32_t reduce, float* margin_out, uint8_t* fire_out,
                        const int8_t* force) {
  if (!c) return fail(GVC_EINVAL, "null context");
  if (theta != theta) return fail(GVC_EINVAL, "theta is NaN");
  if (reduce != GVC_REDUCE_MEAN && reduce != GVC_REDUCE_MIN) return fail(GVC_EINVAL, "bad reduce");
  if (!c->decode_done) return fail(GVC_ESTATE, "margin_gate needs a decode first");
  const Plan& p = c->p;
  float* m = c->K<float>(p.gate_m_off);
  int* f = c->K<int>(p.gate_f_off);
  // The abort word of the single-launch decode pass stays set from a timed-out
  // barrier until this gate reports it: the gate kernel then invalidates every
  // episode instead of deciding on that decode's margins.
  const bool check_abort = c->persist_ran;
  uint32_t* abort_dev = c->K<uint32_t>(p.bar_off) + kDecodeAbortWord;
  HIP_TRY(launch_gate(c->S<float>(p.margins_off), p.B, p.D, theta, reduce == GVC_REDUCE_MIN, force,
                      check_abort ? abort_dev : nullptr, c->S<int>(p.valid_off), m, f, c->stream));
  std::vector<float> hm(p.B);
  std::vector<int> hf(p.B);
  HIP_TRY(hipMemcpyAsync(hm.data(), m, (size_t)p.B * 4, hipMemcpyDeviceToHost, c->stream));
  HIP_TRY(hipMemcpyAsync(hf.data(), f, (size_t)p.B * 4, hipMemcpyDeviceToHost, c->stream));
  if (check_abort)
    HIP_TRY(hipMemcpyAsync(&c->abort_word, abort_dev, 4, hipMemcpyDeviceToHost, c->stream));
  HIP_TRY(hipStreamSynchronize(c->stream));
  if (check_abort) {
    c->persist_ran = false;
    if (c->abort_word) {
      c->decode_done = false;
      HIP_TRY(launch_fill_u32(abort_dev, 0u, 1, c->stream));   // reported: later passes may run again
      return fail(GVC_EDEVICE, "decode pass: grid barrier timed out; every episode's cache was invalidated");
    }
  }
  for (int b = 0; b < p.B; ++b) {
    if (margin_out) margin_out[b] = hm[b];
    if (fire_out) fire_out[b] = (uint8_t)(hf[b] != 0);
  }
  return GVC_OK;
}

int32_t gvc_invalidate(gvc_ctx* c, int32_t b) {
  if (!c) return fail(GVC_EINVAL, "null context");
  const Plan& p = c->p;
  if (b < -1 || b >= p.B) return fail(GVC_EINVAL, "episode out of range");
  int* v = c->S<int>(p.valid_off);
  if (b < 0)
    HIP_TRY(launch_fill_u32(reinterpret_cast<uint32_t*>(v), 0u, p.B, c->stream));
  else
    HIP_TRY(launch_fill_u32(reinterpret_cast<uint32_t*>(v + b), 0u, 1, c->stream));
  return GVC_OK;
}

size_t gvc_state_item_bytes(const gvc_ctx* c, int32_t item) {
  if (!c) return 0;
  const Plan& p = c->p;
  switch (item) {
    case GVC_STATE_H: return (size_t)p.B * p.P * p.d.d_model * 4;
    case GVC_STATE_K:
    case GVC_STATE_V: return p.layer_kv_elems * 2;
    case GVC_STATE_HEAD_LOGITS: return (size_t)p.B * p.head_rows * p.V * 4;
    case GVC_STATE_VALID: return (size_t)p.B * 4;
    case GVC_STATE_ROWS: return (size_t)p.L * 4;
    case GVC_STATE_MARGINS: return (size_t)p.B * p.D * 4;
    case GVC_STATE_TV: return p.stage2 ? (size_t)p.B * p.L * p.H * p.N * 4 : 0;
    case GVC_STATE_ENTROPY: return p.stage3 ? (size_t)p.B * p.L * p.H * 4 : 0;
    case GVC_STATE_LAYER_Q: return p.stage3 ? (size_t)p.B * p.L * 4 : 0;
    default: return 0;
  }
}

int32_t gvc_read_state(gvc_ctx* c, int32_t item, int32_t layer, void* dst, size_t dst_bytes) {
  if (!c || !dst) return fail(GVC_EINVAL, "null argument");
  const Plan& p = c->p;
  const size_t n = gvc_state_item_bytes(c, item);
  if (n == 0) return fail(GVC_EINVAL, "bad state item");
  if (dst_bytes < n) return fail(GVC_EINVAL, "destination too small");
  const void* src = nullptr;
  switch (item) {
    case GVC_STATE_H:
      if (layer < 0 || layer > p.L) return fail(GVC_EINVAL, "layer out of range");
      src = c->H(layer);
      break;
    case GVC_STATE_K:
    case GVC_STATE_V:
      if (layer < 0 || layer >= p.L) return fail(GVC_EINVAL, "layer out of range");
      src = item == GVC_STATE_K ? (const void*)c->Kc(layer) : (const void*)c->Vc(layer);
      break;
    case GVC_STATE_HEAD_LOGITS: src = c->S<float>(p.head_logits_off); break;
    case GVC_STATE_VALID: src = c->S<int>(p.valid_off); break;
    case GVC_STATE_ROWS: src = c->S<int>(p.rowcount_off); break;
    case GVC_STATE_MARGINS: src = c->S<float>(p.margins_off); break;
    case GVC_STATE_TV: src = c->S<float>(p.tv_off); break;
    case GVC_STATE_ENTROPY: src = c->S<float>(p.ent_off); break;
    case GVC_STATE_LAYER_Q: src = c->S<int>(p.lq_off); break;
  }
  HIP_TRY(hipMemcpyAsync(dst, src, n, hipMemcpyDeviceToDevice, c->stream));
  HIP_TRY(hipStreamSynchronize(c->stream));
  return GVC_OK;
}

int32_t gvc_profile_begin(gvc_ctx* c, int32_t cls, int32_t max_launches) {
  if (!c) return fail(GVC_EINVAL, "null context");
  if (cls < 0 || cls >= GVC_K_COUNT || max_launches < 1) return fail(GVC_EINVAL, "bad kernel class or count");
  for (hipEvent_t e : c->prof_ev) (void)hipEventDestroy(e);
  c->prof_ev.assign((size_t)2 * max_launches, nullptr);
  for (auto& e : c->prof_ev) HIP_TRY(hipEventCreate(&e));
  c->prof_n = 0;
  c->prof_cls = cls;
  return GVC_OK;
}

int32_t gvc_profile_end(gvc_ctx* c, double* total_ms, int32_t* launches) {
  if (!c) return fail(GVC_EINVAL, "null context");
  if (c->prof_cls < 0) return fail(GVC_ESTATE, "no profile running");
  HIP_TRY(hipStreamSynchronize(c->stream));
  double tot = 0.0;
  for (int i = 0; i < c->prof_n; ++i) {
    float ms = 0.f;
    HIP_TRY(hipEventElapsedTime(&ms, c->prof_ev[2 * i], c->prof_ev[2 * i + 1]));
    tot += ms;
  }
  if (total_ms) *total_ms = tot;
  if (launches) *launches = c->prof_n;
  for (hipEvent_t e : c->prof_ev) (void)hipEventDestroy(e);
  c->prof_ev.clear();
  c->prof_cls = -1;
  c->prof_n = 0;
  return GVC_OK;
}

int32_t gvc_destroy(gvc_ctx* c) {
  if (c)
    for (hipEvent_t e : c->prof_ev) (void)hipEventDestroy(e);
  delete c;
  return GVC_OK;
}

}  // extern "C"
