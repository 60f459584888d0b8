"""The Gated VLA-Cache control step (Alg. 1) over the float64 decoder.

Sec. III-A: the frame is cut into patches, each projected to an embedding and
concatenated with the language tokens; the prompt pass runs all layers over
all prompt tokens, then D action tokens are decoded autoregressively.
Alg. 1: if the previous step's margin is below theta_m the cache is
invalidated and the pass runs over all tokens, storing fresh K/V; otherwise
static patches reuse their cached K/V and only the other tokens are
recomputed; then the actions are decoded.

Readings (the paper does not fix them):
  * token order: [text token 0] [visual tokens, view-major, raster]
    [text tokens 1..] [proprio rows] [action-query rows], at positions
    0..P-1; only visual tokens are reuse candidates;
  * the visual embedding is (pixel / 255) . W_patch^T over the flattened
    patch, the text embedding a table row; extra rows are given;
  * K is stored after the rotary embedding, at the token's absolute
    position, which does not change between frames;
  * the hidden state entering every layer persists across steps like K/V:
    a token not recomputed at layer l keeps its output of layer l from the
    last pass that computed it;
  * the D-th action token is never fed back, so D-1 single-token passes
    follow the prompt pass; their K/V are dropped after the step;
  * with a parallel-decoded action chunk the head reads the action-query
    rows of the prompt pass and no extra pass runs.
"""
import numpy as np
import torch

from .patches import select_static as _select_one
from .llama import layer_rows, layer_rows_batched, head_row, rmsnorm
from .relevance import text_vision_attention, text_attention_entropy, entropy_permille, relevant_patches
from .margin import position_margin, reduce_margin, gate_fires
from .vit import visual_embeddings


def _f64(t):
    # exact (bf16 -> float64); torch's CPU conversion runs on all cores
    return t.detach().to("cpu").to(torch.float64).numpy()


def convert_weights(w: dict) -> dict:
    """bf16 torch weights (synth layout) -> float64 numpy."""
    out = {k: _f64(v) for k, v in w.items() if k not in ("layers", "vit")}
    if "layers" in w:
        out["layers"] = [{k: _f64(v) for k, v in lw.items()} for lw in w["layers"]]
    if "vit" in w:
        out["vit"] = convert_weights(w["vit"])
    return out


class Layout:
    """Row <-> position map of one episode's prompt (row index == position)."""

    def __init__(self, cfg):
        self.cfg = cfg
        N, T, E = cfg.n_patches, cfg.n_text, cfg.n_extra
        self.P = N + T + E
        self.visual_pos = np.arange(1, N + 1)
        self.text_pos = np.array([0] + list(range(N + 1, N + T)))
        self.extra_pos = np.arange(N + T, N + T + E)
        if cfg.parallel_decode:
            self.head_pos = self.extra_pos[cfg.n_proprio:]
        else:
            self.head_pos = np.array([self.P - 1])


class OracleVLA:
    """Alg. 1 over the float64 decoder.  batched=True takes each layer's
    projections as matrix products over the recomputed rows
    (layer_rows_batched) instead of one row at a time: the same arithmetic
    up to the summation order inside the products, fast enough for the 7B
    shape.  The row-at-a-time default keeps a row's value independent of
    which other rows a pass computes, so the invariants below hold
    bit-exactly."""

    def __init__(self, cfg, weights, batched=False):
        self.cfg = cfg
        self.layer = layer_rows_batched if batched else layer_rows
        self.w = weights if isinstance(weights["embed"], np.ndarray) else convert_weights(weights)
        B, L, d = cfg.batch, cfg.n_layers, cfg.d_model
        self.lay = Layout(cfg)
        P = self.lay.P
        self.H = np.zeros((L + 1, B, P, d))
        self.K = np.zeros((L, B, cfg.kv_len, cfg.n_heads, cfg.head_dim))
        self.V = np.zeros_like(self.K)
        self.valid = np.zeros(B, dtype=bool)
        self.head_logits = None
        self.margins = None
        self.tokens = None
        self.recomputed = None     # [B][L] rows recomputed by the last prefill
        self.tv = None             # [B][L][H][N] Stage 2 attention of the last prefill (task_topk > 0)
        self.ent = None            # [B][L][H] Stage 3 entropy sums of the last prefill (entropy_reuse)
        self.vis_emb = None        # [B][N][d] visual embeddings of the last prefill's frame (vit_layers > 0)

    # ---------------------------------------------------------- Stage 1 + 3
    def relevant(self, b, scores=None):
        """Stage 2: episode b's task-relevant patches [N] bool from the last
        prefill's attention (or from given per-patch scores), or None."""
        cfg = self.cfg
        if cfg.task_topk <= 0 or cfg.n_text < 2:
            return None
        if scores is None:
            if self.tv is None:
                return None
            scores = self.tv[b].sum(axis=(0, 1))
        return relevant_patches(np.asarray(scores, dtype=np.float64), cfg.task_topk)

    def layer_permille(self, b):
        """Stage 3: episode b's per-layer proportions from the last prefill's
        attention entropy, or None (fixed proportions)."""
        cfg = self.cfg
        if not cfg.entropy_reuse or cfg.n_text < 2 or self.ent is None:
            return None
        return entropy_permille(self.ent[b], cfg.n_text - 1)

    def select_static(self, frame_t, frame_prev, tau=None, permille=None, scores=None, layer_q=None):
        """Per episode: reuse masks [B][L][N] and |S| [B] (Stages 1-3).
        scores [B][N] / layer_q [B][L], if given, replace the oracle's own
        Stage 2 scores / Stage 3 proportions."""
        cfg = self.cfg
        tau = tau or cfg.tau
        ft, fp = np.asarray(frame_t), np.asarray(frame_prev)
        masks = np.zeros((cfg.batch, cfg.n_layers, cfg.n_patches), dtype=bool)
        n_static = np.zeros(cfg.batch, dtype=np.int64)
        for b in range(cfg.batch):
            excl = self.relevant(b, None if scores is None else scores[b])
            q = list(layer_q[b]) if layer_q is not None else self.layer_permille(b)
            q = q or permille or cfg.permille()
            masks[b], n_static[b], _, _ = _select_one(ft[b], fp[b], cfg.patch, tau, q, excl)
        return masks, n_static

    # ---------------------------------------------------------- prompt pass
    def key_last(self, rows):
        """Last key slot each row attends to: its own position (causal), or,
        for the OFT model's parallel action-dimension decoding (Sec. V-A,
        models and baselines; the mask is not given there, the reading is
        that the action-query rows see each other both ways), the last
        prompt position for the action-query rows.  None when every row is
        causal."""
        cfg = self.cfg
        if not cfg.action_bidir:
            return None
        a0 = self.lay.P - cfg.n_action_q
        return [self.lay.P - 1 if p >= a0 else p for p in rows]

    def embed_row(self, b, pos, frame_t, text_ids, extra_rows):
        cfg, lay = self.cfg, self.lay
        N = cfg.n_patches
        if 1 <= pos <= N and self.vis_emb is not None:
            return self.vis_emb[b, pos - 1].copy()
        if 1 <= pos <= N:
            n = pos - 1
            v, rc = divmod(n, cfg.patches_per_side ** 2)
            r, c = divmod(rc, cfg.patches_per_side)
            p = cfg.patch
            px = np.asarray(frame_t[b, v, r * p:(r + 1) * p, c * p:(c + 1) * p, :]).reshape(-1)
            return self.w["patch_proj"] @ (px.astype(np.float64) / 255.0)
        if pos == 0:
            return self.w["embed"][int(text_ids[b, 0])].copy()
        if pos < N + cfg.n_text:
            return self.w["embed"][int(text_ids[b, pos - N])].copy()
        return np.asarray(extra_rows[b, pos - N - cfg.n_text], dtype=np.float64).copy()

    def step_prefill(self, frame_t, text_ids, extra_rows=None, masks=None):
        """a2-a7: the (partial) prompt pass; rows of an invalid cache run full."""
        cfg, lay = self.cfg, self.lay
        frame_t = np.asarray(frame_t)
        text_ids = np.asarray(text_ids)
        if extra_rows is not None:
            extra_rows = np.asarray(extra_rows, dtype=np.float64)
        P, L = lay.P, cfg.n_layers
        self.head_logits = np.zeros((cfg.batch, len(lay.head_pos), cfg.vocab))
        self.recomputed = np.zeros((cfg.batch, L), dtype=np.int64)
        stage2 = cfg.task_topk > 0 and cfg.n_text >= 2
        stage3 = cfg.entropy_reuse and cfg.n_text >= 2
        if stage2:
            self.tv = np.zeros((cfg.batch, L, cfg.n_heads, cfg.n_patches))
        if stage3:
            self.ent = np.zeros((cfg.batch, L, cfg.n_heads))
        if cfg.vit_layers > 0:   # the front end runs on the whole frame every pass
            self.vis_emb = np.stack([visual_embeddings(self.w["vit"], frame_t[b], cfg.patch, cfg.vit_heads,
                                                       cfg.vit_eps) for b in range(cfg.batch)])
        for b in range(cfg.batch):
            use_mask = masks is not None and self.valid[b]
            for l in range(L):
                reused = set()
                if use_mask:
                    reused = {1 + n for n in np.nonzero(np.asarray(masks[b][l]))[0]}
                rows = [p for p in range(P) if p not in reused]
                if l == 0:
                    for p in rows:
                        self.H[0, b, p] = self.embed_row(b, p, frame_t, text_ids, extra_rows)
                out = self.layer(self.w["layers"][l], self.H[l, b], rows, rows,
                                 self.K[l, b], self.V[l, b], cfg.n_heads, cfg.rms_eps, cfg.rope_theta,
                                 self.key_last(rows))
                if stage2:
                    self.tv[b, l] = text_vision_attention(self.w["layers"][l], self.H[l, b], self.K[l, b],
                                                          cfg.n_patches, cfg.n_text, cfg.n_heads, cfg.rms_eps,
                                                          cfg.rope_theta)
                if stage3:
                    self.ent[b, l] = text_attention_entropy(self.w["layers"][l], self.H[l, b], self.K[l, b],
                                                            cfg.n_patches, cfg.n_text, cfg.n_heads, cfg.rms_eps,
                                                            cfg.rope_theta)
                self.H[l + 1, b, rows] = out
                self.recomputed[b, l] = len(rows)
            for i, p in enumerate(lay.head_pos):
                self.head_logits[b, i] = head_row(self.H[L, b, p], self.w["final_norm"],
                                                  self.w["lm_head"], cfg.rms_eps)
            self.valid[b] = True
        return self.head_logits

    # ---------------------------------------------------------- action decode
    def decode_pass(self, b, token, pos):
        """One single-token pass at absolute position pos; returns its logits."""
        cfg = self.cfg
        x = self.w["embed"][int(token)][None, :].copy()
        for l in range(cfg.n_layers):
            x = self.layer(self.w["layers"][l], x, [0], [pos], self.K[l, b], self.V[l, b],
                           cfg.n_heads, cfg.rms_eps, cfg.rope_theta)
        return head_row(x[0], self.w["final_norm"], self.w["lm_head"], cfg.rms_eps)

    def decode_actions(self, forced_tokens=None):
        """a8-a9: tokens [B][D], per-position margins [B][D], logits [B][D][V].
        forced_tokens [B][D], if given, are fed back instead of the argmax."""
        cfg = self.cfg
        D, P = cfg.n_decode, self.lay.P
        tokens = np.zeros((cfg.batch, D), dtype=np.int64)
        margins = np.zeros((cfg.batch, D))
        logits = np.zeros((cfg.batch, D, cfg.vocab))
        for b in range(cfg.batch):
            if cfg.parallel_decode:
                for d in range(D):
                    z = self.head_logits[b, d]
                    tokens[b, d], margins[b, d] = position_margin(z, cfg.bin_lo, cfg.norm_full_vocab)
                    logits[b, d] = z
                continue
            z = self.head_logits[b, 0]
            for d in range(D):
                logits[b, d] = z
                tokens[b, d], margins[b, d] = position_margin(z, cfg.bin_lo, cfg.norm_full_vocab)
                if d + 1 < D:
                    fed = tokens[b, d] if forced_tokens is None else int(forced_tokens[b][d])
                    z = self.decode_pass(b, fed, P + d)
        self.tokens, self.margins = tokens, margins
        return tokens, margins, logits

    # ---------------------------------------------------------- gate
    def margin_gate(self, theta=None, use_min=None, force=None):
        """a10: reduce the last decode's margins, fire when below theta, and
        invalidate the fired episodes' caches.  force[b] in {-1, 0, 1}
        overrides the decision (lock-step testing)."""
        cfg = self.cfg
        theta = cfg.theta if theta is None else theta
        use_min = cfg.reduce_min if use_min is None else use_min
        m = np.array([reduce_margin(self.margins[b], use_min) for b in range(cfg.batch)])
        fire = np.array([gate_fires(m[b], theta) for b in range(cfg.batch)])
        if force is not None:
            for b in range(cfg.batch):
                if force[b] >= 0:
                    fire[b] = bool(force[b])
        self.valid &= ~fire
        return m, fire

    def invalidate(self, b=-1):
        if b < 0:
            self.valid[:] = False
        else:
            self.valid[b] = False

    # ---------------------------------------------------------- Alg. 1
    def control_step(self, frame_t, frame_prev, text_ids, extra_rows=None, theta=None,
                     first=False, force_reuse=False):
        """One step of Alg. 1: gate on the previous margins, Stage 1+3, the
        (partial) prompt pass, the action decode."""
        fire = None
        if not first and not force_reuse:
            _, fire = self.margin_gate(theta)
        masks = None
        if not first:
            masks, _ = self.select_static(frame_t, frame_prev)
        self.step_prefill(frame_t, text_ids, extra_rows, masks)
        tokens, margins, logits = self.decode_actions()
        return tokens, margins, fire
