"""Helpers shared by the GPU parity tests (comparison rules, device copies)."""
import numpy as np
import torch

TOL = 2e-2   # max |gpu - oracle| / max |oracle| on logits, K/V and hidden states
TOL_SLICE = 5e-2   # the same per row of H / logits and per (row, head) of K and V (rel_err_slices)


def rel_err(g, o) -> float:
    g = np.asarray(g, dtype=np.float64)
    o = np.asarray(o, dtype=np.float64)
    den = np.abs(o).max()
    return float(np.abs(g - o).max() / (den if den > 0 else 1.0))


def to_dev(w, dev):
    out = {k: v.to(dev) for k, v in w.items() if k not in ("layers", "vit")}
    out["layers"] = [{k: v.to(dev) for k, v in lw.items()} for lw in w["layers"]]
    if "vit" in w:
        out["vit"] = to_dev(w["vit"], dev)
    return out


def gpu_k(sess, l, P):
    """K of layer l as [B][pos][H][dh] float64 for pos < P."""
    from paper_2608_10824_amd import gvc
    k = sess.read(gvc.STATE_K, l).float().cpu().numpy()      # [B][H][kv_pad][dh]
    return k[:, :, :P, :].transpose(0, 2, 1, 3)


def gpu_v(sess, l, P):
    from paper_2608_10824_amd import gvc
    v = sess.read(gvc.STATE_V, l).float().cpu().numpy()      # [B][H][dh][kv_pad]
    return v[:, :, :, :P].transpose(0, 3, 1, 2)


def check_tokens(tok_g, logits_g, tok_o, logits_o, bin_lo):
    """Tokens must be the argmax of the GPU's own logits (ties to the lower
    id), and equal the oracle's except where the oracle's top-2 bin gap is
    within twice the largest logit error at that position.  Returns the
    number of accepted near-ties."""
    ties = 0
    tok_g, tok_o = np.asarray(tok_g), np.asarray(tok_o)
    for idx in np.ndindex(tok_g.shape):
        zg = np.asarray(logits_g[idx], dtype=np.float64)
        zo = np.asarray(logits_o[idx], dtype=np.float64)
        bins_g = zg[bin_lo:]
        assert tok_g[idx] == bin_lo + int(np.argmax(bins_g)), "token is not the argmax of its own logits"
        if tok_g[idx] != tok_o[idx]:
            eps = np.abs(zg - zo).max()
            s = np.sort(zo[bin_lo:])[::-1]
            assert s[0] - s[1] < 2 * eps, "token differs at %s beyond the near-tie band" % (idx,)
            ties += 1
    return ties


def margin_bounds(logits_g, logits_o, bin_lo, full_vocab=True):
    """Per-position bound on |m_gpu - m_oracle| implied by the logit error.

    If every logit of a position moves by at most eps, every softmax
    probability moves by a factor within [e^-2eps, e^2eps], so the margin
    p1 - p2 moves by at most (p1 + p2)(e^2eps - 1), whichever ids end up
    first and second.  fp32 rounding of the margin itself adds 1e-6."""
    zg = np.asarray(logits_g, dtype=np.float64)
    zo = np.asarray(logits_o, dtype=np.float64)
    out = np.zeros(zo.shape[:-1])
    for idx in np.ndindex(out.shape):
        eps = np.abs(zg[idx] - zo[idx]).max()
        dom = zo[idx] if full_vocab else zo[idx][bin_lo:]
        p = np.exp(dom - dom.max())
        p /= p.sum()
        b = np.sort(np.exp(zo[idx][bin_lo:] - dom.max()) / np.exp(dom - dom.max()).sum())[::-1]
        out[idx] = (b[0] + b[1]) * np.expm1(2 * eps) + 1e-6
    return out


def check_margins(m_g, m_o, logits_g, logits_o, bin_lo, full_vocab=True):
    bound = margin_bounds(logits_g, logits_o, bin_lo, full_vocab)
    diff = np.abs(np.asarray(m_g, dtype=np.float64) - np.asarray(m_o))
    assert (diff <= bound).all(), "margin error %s exceeds bound %s" % (diff, bound)
    return bound


# ---------------------------------------------------------------- 7B helpers
def layer_w64(w_dev, l):
    """float64 CPU copy of layer l of device weights (synth layout)."""
    return {k: v.float().cpu().numpy().astype(np.float64) for k, v in w_dev["layers"][l].items()}


def glob_w64(w_dev):
    return {k: w_dev[k].float().cpu().numpy().astype(np.float64) for k in ("embed", "lm_head", "final_norm")}


def state64(sess, item, layer, b, P):
    """One episode's state item as float64: H [P][d], K/V [kv][H][dh]."""
    from paper_2608_10824_amd import gvc
    if item == gvc.STATE_H:
        return sess.read(item, layer)[b].double().cpu().numpy()
    if item == gvc.STATE_K:
        return sess.read(item, layer)[b].double().cpu().numpy().transpose(1, 0, 2)[:P]
    return sess.read(item, layer)[b].double().cpu().numpy().transpose(2, 0, 1)[:P]


def check_layer_sampled(cfg, wl, h_in, h_out, K, V, sample_pos):
    """Recompute one layer for the sampled rows with the oracle from the GPU's
    own inputs (h_in = GPU H[l], K/V = GPU cache of layer l for the other
    keys) and compare fresh K/V and the layer output.  Returns the errors."""
    from oracle.llama import layer_rows
    Ko, Vo = K.copy(), V.copy()
    key_last = None
    if cfg.action_bidir:   # the action-query rows see every prompt key
        a0 = cfg.prompt_len - cfg.n_action_q
        key_last = [cfg.prompt_len - 1 if p >= a0 else p for p in sample_pos]
    out = layer_rows(wl, h_in, list(sample_pos), list(sample_pos), Ko, Vo, cfg.n_heads, cfg.rms_eps,
                     cfg.rope_theta, key_last)
    sp = list(sample_pos)
    errs = {"k": rel_err(K[sp], Ko[sp]), "v": rel_err(V[sp], Vo[sp]), "out": rel_err(h_out[sp], out)}
    return errs


def rel_err_slices(g, o, n_lead) -> float:
    """Largest per-slice relative error: the arrays are cut into the slices
    indexed by their first n_lead axes (a row of H, a (row, head) of K or V)
    and each slice's max |g - o| is divided by that slice's own max |o|, so a
    wrong low-magnitude row or head cannot hide under the tensor's maximum."""
    g = np.asarray(g, dtype=np.float64)
    o = np.asarray(o, dtype=np.float64)
    lead = int(np.prod(o.shape[:n_lead]))
    g, o = g.reshape(lead, -1), o.reshape(lead, -1)
    den = np.abs(o).max(axis=1)
    den = np.where(den > 0, den, 1.0)
    return float((np.abs(g - o).max(axis=1) / den).max())


# ---------------------------------------------------------------- Stage 2 / 3 decisions
# The selection turns floating-point signals into integers (which patches
# are task-relevant, each layer's per-mille proportion).  Both sides take
# those decisions in the kernel's precision: the oracle's own float64
# signals go through the same fp32 steps the GPU applies to its signals.
# The two decisions may differ only where the oracle's value lies within the
# measured signal error of a decision boundary (several answers are correct).

def fp32_scores(tv):
    """Per-patch Stage 2 scores [B][N] as the kernel forms them: fp32 sums
    over the (layer, head) columns of tv [B][L][H][N], in order."""
    B, L, H, N = tv.shape
    flat = np.asarray(tv).reshape(B, L * H, N).astype(np.float32)
    acc = np.zeros((B, N), dtype=np.float32)
    for c in range(L * H):
        acc = (acc + flat[:, c, :]).astype(np.float32)
    return acc


def fp32_layer_q(ent, n_instr):
    """Stage 3 per-layer proportions from ent [L][H], taking the kernel's fp32
    steps in its order: E_l summed over heads, u_l = 1 - E_l / (H n_instr),
    s_l = s_{l-1} + (u_l - s_{l-1}) / 2, q_l = floor(1000 clamp(s_l))."""
    f = np.float32
    L, H = ent.shape
    out, sl = [], f(0)
    for l in range(L):
        e = f(0)
        for h in range(H):
            e = f(e + f(ent[l, h]))
        u = f(f(1) - f(e / f(H * n_instr)))
        sl = u if l == 0 else f(sl + f(f(u - sl) * f(0.5)))
        c = min(max(sl, f(0)), f(1))
        out.append(int(np.floor(f(f(1000) * c))))
    return out


def layer_q_near_ties(ent_o, ent_g, n_instr, q_o, q_g):
    """Layers whose proportions differ; each must be a near tie: the oracle's
    1000 s_l within 1000 max|dE| (+1e-3 for fp32 rounding) of the boundary
    between the two values (s_l is a convex mix of the u_j, so its error is at
    most max|dE|)."""
    L, H = ent_o.shape
    dE = np.abs(np.asarray(ent_g, np.float64).sum(axis=1) - np.asarray(ent_o).sum(axis=1)).max() / (H * n_instr)
    s, out = 0.0, []
    for l in range(L):
        u = 1.0 - ent_o[l].sum() / (H * n_instr)
        s = u if l == 0 else s + (u - s) / 2
        if q_o[l] != q_g[l]:
            boundary = max(q_o[l], q_g[l])
            assert abs(q_o[l] - q_g[l]) == 1 and abs(1000 * min(max(s, 0.0), 1.0) - boundary) <= 1000 * dE + 1e-3, \
                "layer %d proportion %d vs %d beyond the signal error" % (l, q_o[l], q_g[l])
            out.append(l)
    return out


def relevant_near_ties(score_o, score_g, k, rel_o, rel_g):
    """Patches selected as task-relevant by one side only; each must sit
    within twice the measured score error of the k-th / (k+1)-th boundary of
    the oracle's scores."""
    diff = np.nonzero(rel_o != rel_g)[0]
    if len(diff) == 0:
        return []
    eps = np.abs(np.asarray(score_g, np.float64) - np.asarray(score_o, np.float64)).max()
    srt = np.sort(np.asarray(score_o, np.float64))[::-1]
    lo, hi = srt[min(k, len(srt) - 1)], srt[k - 1]
    for n in diff:
        assert lo - 2 * eps <= score_o[n] <= hi + 2 * eps, "patch %d selected beyond the score error" % n
    return diff.tolist()
