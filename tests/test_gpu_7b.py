"""Parity at the full 7B sizes (32 layers, d=4096, 32 heads, FFN 11008,
vocab 32000), in the launch configuration the benchmark times.

The oracle cannot run every row of every layer here, so the checks are:
  * every reuse mask and static count, bit-exact (integer path);
  * per-layer recompute counts;
  * rows reused at a layer keep their K/V and layer output bit-identical to
    the previous step (nothing rewrites them);
  * sampled layers: the oracle recomputes the layer for sampled rows from the
    GPU's own layer input and K/V cache, and the fresh K/V and outputs must
    match within the tolerance;
  * the head logits of the head rows from the GPU's final hidden state;
  * (C2) the whole decode chain: 6 fed-back tokens through all 32 layers in
    float64 over the GPU's prompt K/V, against the GPU's decode logits,
    tokens and margins.
"""
import os

import numpy as np
import pytest
import torch

import synth
from oracle import patches as op
from oracle.llama import head_row, layer_rows
from oracle.margin import position_margin, gate_fires
from tests._parity import (TOL, rel_err, check_tokens, check_margins, layer_w64, glob_w64, state64,
                           check_layer_sampled)

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def _session(cfg):
    from paper_2608_10824_amd.session import Session
    w = synth.model_weights(cfg, device=DEV)
    return Session(cfg, w, device=DEV), w


def _two_steps(cfg, s, si):
    """Full step on frame_prev, then a reuse step on frame_t (gate kept)."""
    from paper_2608_10824_amd import gvc
    fp, ft = si["frame_prev"].to(DEV), si["frame_t"].to(DEV)
    ids = si["text_ids"].to(DEV)
    ex = None if si["extra_rows"] is None else si["extra_rows"].to(DEV)
    s.step_prefill(fp, ids, ex)
    s.decode_actions()
    s.margin_gate(force=[0] * cfg.batch)
    return fp, ft, ids, ex


def _oracle_masks(cfg, si):
    out, ns = [], []
    for b in range(cfg.batch):
        m, n, _, _ = op.select_static(si["frame_t"][b].numpy(), si["frame_prev"][b].numpy(), cfg.patch, cfg.tau,
                                      cfg.permille())
        out.append(m)
        ns.append(n)
    return np.stack(out), np.array(ns)


def _sample_rows(cfg, rows_recomputed):
    P = cfg.prompt_len
    vis = [p for p in rows_recomputed if 1 <= p <= cfg.n_patches]
    pick = [0, P - 1] + vis[:1] + vis[-1:]
    return sorted(set(pick))


def _oracle_decode_chain(cfg, w, h_last, Ks, Vs, fed):
    """Logits [D][V] of the prompt's last row and of the D - 1 single-token
    passes fed with `fed`, in float64 over one episode's prompt K/V."""
    g = glob_w64(w)
    P, D, L = cfg.prompt_len, cfg.n_decode, cfg.n_layers
    z0 = head_row(h_last, g["final_norm"], g["lm_head"], cfg.rms_eps)
    x = g["embed"][fed].copy()
    pos = [P + j for j in range(D - 1)]
    for l in range(L):
        K = np.zeros((cfg.kv_len, cfg.n_heads, cfg.head_dim))
        V = np.zeros_like(K)
        K[:P], V[:P] = Ks[l], Vs[l]
        x = layer_rows(layer_w64(w, l), x, list(range(D - 1)), pos, K, V, cfg.n_heads, cfg.rms_eps, cfg.rope_theta)
    return np.stack([z0] + [head_row(x[j], g["final_norm"], g["lm_head"], cfg.rms_eps) for j in range(D - 1)])


@pytest.fixture(scope="module")
def c2():
    from paper_2608_10824_amd import gvc
    cfg = synth.config_c2()
    s, w = _session(cfg)
    si = synth.step_inputs(cfg, 128)
    fp, ft, ids, ex = _two_steps(cfg, s, si)
    layers = [0, 15, cfg.n_layers - 1]
    P = cfg.prompt_len
    before = {l: (state64(s, gvc.STATE_K, l, 0, P), state64(s, gvc.STATE_V, l, 0, P),
                  state64(s, gvc.STATE_H, l + 1, 0, P)) for l in layers}
    mask, n_static = s.select_static(ft, fp)
    mask = mask.cpu().numpy().astype(bool)
    s.step_prefill(ft, ids, ex, s.mask)
    prompt_K = [state64(s, gvc.STATE_K, l, 0, P) for l in range(cfg.n_layers)]
    prompt_V = [state64(s, gvc.STATE_V, l, 0, P) for l in range(cfg.n_layers)]
    H = {l: state64(s, gvc.STATE_H, l, 0, P) for l in set(layers) | {l + 1 for l in layers} | {cfg.n_layers}}
    rows = s.read(gvc.STATE_ROWS).cpu().numpy()
    head = s.read(gvc.STATE_HEAD_LOGITS).cpu().numpy()
    tok, mg, lg = s.decode_actions(logits=True)
    torch.cuda.synchronize()
    res = dict(cfg=cfg, si=si, w=w, mask=mask, n_static=n_static.cpu().numpy(), before=before, K=prompt_K,
               V=prompt_V, H=H, rows=rows, head=head, tok=tok.cpu().numpy(), mg=mg.cpu().numpy(),
               lg=lg.cpu().numpy(), layers=layers)
    yield res
    s.close()


def test_c2_masks_and_counts(c2):
    cfg = c2["cfg"]
    mo, ns = _oracle_masks(cfg, c2["si"])
    assert np.array_equal(c2["mask"], mo)
    assert c2["n_static"].tolist() == ns.tolist() == [128]
    assert (mo[0, 0] == c2["si"]["unchanged"][0]).all()
    assert c2["rows"].tolist() == [cfg.prompt_len - 128] * cfg.n_layers


def test_c2_reused_rows_untouched(c2):
    from paper_2608_10824_amd import gvc
    cfg = c2["cfg"]
    reused = [1 + n for n in np.nonzero(c2["mask"][0, 0])[0]]
    for l in c2["layers"]:
        K0, V0, H0 = c2["before"][l]
        assert np.array_equal(c2["K"][l][reused], K0[reused])
        assert np.array_equal(c2["V"][l][reused], V0[reused])
        assert np.array_equal(c2["H"][l + 1][reused], H0[reused])


def test_c2_sampled_layers(c2):
    cfg, w = c2["cfg"], c2["w"]
    recomputed = [p for p in range(cfg.prompt_len) if not (1 <= p <= cfg.n_patches and c2["mask"][0, 0, p - 1])]
    sample = _sample_rows(cfg, recomputed)
    for l in c2["layers"]:
        errs = check_layer_sampled(cfg, layer_w64(w, l), c2["H"][l], c2["H"][l + 1], c2["K"][l], c2["V"][l], sample)
        print("layer", l, {k: "%.2e" % v for k, v in errs.items()})
        assert all(v <= TOL for v in errs.values()), (l, errs)


def test_c2_head_and_decode_chain(c2):
    """Oracle decode over the GPU prompt K/V with the GPU's tokens fed back."""
    cfg, w = c2["cfg"], c2["w"]
    g = glob_w64(w)
    P, D, L = cfg.prompt_len, cfg.n_decode, cfg.n_layers
    z0 = head_row(c2["H"][L][P - 1], g["final_norm"], g["lm_head"], cfg.rms_eps)
    assert rel_err(c2["head"][0, 0], z0) <= TOL
    fed = c2["tok"][0, :D - 1]
    x = g["embed"][fed].copy()
    pos = [P + j for j in range(D - 1)]
    for l in range(L):
        K = np.zeros((cfg.kv_len, cfg.n_heads, cfg.head_dim))
        V = np.zeros_like(K)
        K[:P], V[:P] = c2["K"][l], c2["V"][l]
        x = layer_rows(layer_w64(w, l), x, list(range(D - 1)), pos, K, V, cfg.n_heads, cfg.rms_eps, cfg.rope_theta)
    zo = np.stack([z0] + [head_row(x[j], g["final_norm"], g["lm_head"], cfg.rms_eps) for j in range(D - 1)])
    lg = c2["lg"][0]
    err = rel_err(lg, zo)
    print("decode chain logits rel err %.2e" % err)
    assert err <= TOL
    tok_o = np.array([position_margin(zo[j], cfg.bin_lo)[0] for j in range(D)])
    m_o = np.array([position_margin(zo[j], cfg.bin_lo)[1] for j in range(D)])
    check_tokens(c2["tok"][0], lg, tok_o, zo, cfg.bin_lo)
    check_margins(c2["mg"][0], m_o, lg, zo, cfg.bin_lo)


# ---------------------------------------------------------------- C2 with the ViT front end
def test_c2v_front_end_and_layers():
    """ViT-L/14-shaped front end at the 7B shape: the layer-0 input of every
    prompt row (visual rows from the GPU's ViT and projector) against the
    oracle's, after a full and after a partial step; sampled layers; the
    head logits."""
    from paper_2608_10824_amd import gvc
    from oracle.vit import visual_embeddings
    from oracle.vla import convert_weights
    cfg = synth.config_c2v()
    s, w = _session(cfg)
    si = synth.step_inputs(cfg, 128)
    fp, ft, ids, ex = _two_steps(cfg, s, si)
    P, N, L = cfg.prompt_len, cfg.n_patches, cfg.n_layers
    vw = convert_weights({"vit": w["vit"]})["vit"]
    g = glob_w64(w)
    ids_np = si["text_ids"].numpy()[0]

    def h0_oracle(frame):
        h = np.empty((P, cfg.d_model))
        h[0] = g["embed"][ids_np[0]]
        h[1:N + 1] = visual_embeddings(vw, frame, cfg.patch, cfg.vit_heads, cfg.vit_eps)
        h[N + 1:] = g["embed"][ids_np[1:]]
        return h

    e_full = rel_err(state64(s, gvc.STATE_H, 0, 0, P), h0_oracle(si["frame_prev"].numpy()[0]))
    mask, _ = s.select_static(ft, fp)
    mask = mask.cpu().numpy().astype(bool)
    s.step_prefill(ft, ids, ex, s.mask)
    H0 = state64(s, gvc.STATE_H, 0, 0, P)
    ref = h0_oracle(si["frame_t"].numpy()[0])
    reused = [1 + n for n in np.nonzero(mask[0, 0])[0]]
    fresh = [p for p in range(P) if p not in reused]
    e_part = rel_err(H0[fresh], ref[fresh])
    print("layer-0 input rel err: full %.2e, recomputed rows of the partial step %.2e" % (e_full, e_part))
    assert e_full <= TOL and e_part <= TOL
    sample = _sample_rows(cfg, fresh)
    for l in (0, L - 1):
        errs = check_layer_sampled(cfg, layer_w64(w, l), state64(s, gvc.STATE_H, l, 0, P),
                                   state64(s, gvc.STATE_H, l + 1, 0, P), state64(s, gvc.STATE_K, l, 0, P),
                                   state64(s, gvc.STATE_V, l, 0, P), sample)
        print("layer", l, {k: "%.2e" % v for k, v in errs.items()})
        assert all(v <= TOL for v in errs.values()), (l, errs)
    z0 = head_row(state64(s, gvc.STATE_H, L, 0, P)[P - 1], g["final_norm"], g["lm_head"], cfg.rms_eps)
    assert rel_err(s.read(gvc.STATE_HEAD_LOGITS).cpu().numpy()[0, 0], z0) <= TOL
    s.close()


# ---------------------------------------------------------------- C2 with Stages 2 and 3
def test_c2_stage2_stage3_signals_and_selection():
    """The benchmark's Stage 2 (k = 120) + Stage 3 (entropy) configuration at
    the 7B shape: the recorded signals of sampled layers against the oracle
    recomputed from the GPU's own layer input and key cache; the selection
    bit-exact against the oracle's ranking with the GPU's fp32 scores and
    proportions (the proportions themselves exact against the same fp32
    steps on the GPU's signal)."""
    from paper_2608_10824_amd import gvc
    from oracle.relevance import text_vision_attention, text_attention_entropy, relevant_patches
    from tests.test_gpu_stage3 import _q_fp32
    cfg = synth.config_c2().with_(task_topk=120, entropy_reuse=True)
    s, w = _session(cfg)
    si = synth.step_inputs(cfg, 128)
    fp, ft, ids = si["frame_prev"].to(DEV), si["frame_t"].to(DEV), si["text_ids"].to(DEV)
    s.step_prefill(fp, ids)
    P, N, L, H = cfg.prompt_len, cfg.n_patches, cfg.n_layers, cfg.n_heads
    tv = s.read(gvc.STATE_TV).cpu().numpy()[0]        # [L][H][N]
    ent = s.read(gvc.STATE_ENTROPY).cpu().numpy()[0]  # [L][H]
    for l in (0, L - 1):
        wl = layer_w64(w, l)
        h_in, K = state64(s, gvc.STATE_H, l, 0, P), state64(s, gvc.STATE_K, l, 0, P)
        a = text_vision_attention(wl, h_in, K, N, cfg.n_text, H, cfg.rms_eps, cfg.rope_theta)
        e = text_attention_entropy(wl, h_in, K, N, cfg.n_text, H, cfg.rms_eps, cfg.rope_theta)
        errs = (rel_err(tv[l], a), rel_err(ent[l], e))
        print("layer %d signal rel err: attention %.2e, entropy %.2e" % (l, *errs))
        assert max(errs) <= TOL
    mask, n_static = s.select_static(ft, fp)
    q = s.read(gvc.STATE_LAYER_Q).cpu().numpy()[0]
    assert q.tolist() == _q_fp32(ent, cfg.n_text - 1)
    acc = np.zeros(N, dtype=np.float32)
    for c in range(L * H):
        acc = (acc + tv.reshape(L * H, N)[c].astype(np.float32)).astype(np.float32)
    rel = relevant_patches(acc.astype(np.float64), 120)
    mo, no, _, _ = op.select_static(si["frame_t"].numpy()[0], si["frame_prev"].numpy()[0], cfg.patch, cfg.tau,
                                    q.tolist(), rel)
    assert np.array_equal(mask.cpu().numpy()[0].astype(bool), mo) and n_static.item() == no
    print("static after Stage 2: %d of 128; proportions %s" % (no, q.tolist()[:4]))
    s.close()


# ---------------------------------------------------------------- C4
@pytest.fixture(scope="module", params=["causal", "bidir"])
def c4(request):
    from paper_2608_10824_amd import gvc
    cfg = synth.config_c4().with_(action_bidir=request.param == "bidir")
    s, w = _session(cfg)
    si = synth.step_inputs(cfg, 307)
    fp, ft, ids, ex = _two_steps(cfg, s, si)
    mask, n_static = s.select_static(ft, fp)
    mask = mask.cpu().numpy().astype(bool)
    s.step_prefill(ft, ids, ex, s.mask)
    P, L = cfg.prompt_len, cfg.n_layers
    layers = [0, L - 1]
    res = dict(cfg=cfg, si=si, w=w, mask=mask, n_static=n_static.cpu().numpy(), layers=layers,
               K={l: state64(s, gvc.STATE_K, l, 0, P) for l in layers},
               V={l: state64(s, gvc.STATE_V, l, 0, P) for l in layers},
               H={l: state64(s, gvc.STATE_H, l, 0, P) for l in (0, 1, L - 1, L)},
               rows=s.read(gvc.STATE_ROWS).cpu().numpy())
    tok, mg, lg = s.decode_actions(logits=True)
    m, fire = s.margin_gate()
    torch.cuda.synchronize()
    res.update(tok=tok.cpu().numpy(), mg=mg.cpu().numpy(), lg=lg.cpu().numpy(), m=m, fire=fire)
    yield res
    s.close()


def test_c4_masks_counts_layers(c4):
    cfg = c4["cfg"]
    mo, ns = _oracle_masks(cfg, c4["si"])
    assert np.array_equal(c4["mask"], mo) and c4["n_static"].tolist() == ns.tolist() == [307]
    assert c4["rows"].tolist() == [cfg.prompt_len - 307] * cfg.n_layers
    recomputed = [p for p in range(cfg.prompt_len) if not (1 <= p <= cfg.n_patches and mo[0, 0, p - 1])]
    # plus the proprio row and the first action-query row (with the block it
    # sees all the later action rows)
    sample = _sample_rows(cfg, recomputed) + [cfg.n_patches + cfg.n_text, cfg.prompt_len - cfg.n_action_q]
    for l in c4["layers"]:
        errs = check_layer_sampled(cfg, layer_w64(c4["w"], l), c4["H"][l], c4["H"][l + 1], c4["K"][l], c4["V"][l],
                                   sorted(set(sample)))
        print("layer", l, {k: "%.2e" % v for k, v in errs.items()})
        assert all(v <= TOL for v in errs.values()), (l, errs)


def test_c4_action_chunk_head_and_min_gate(c4):
    cfg = c4["cfg"]
    g = glob_w64(c4["w"])
    L = cfg.n_layers
    rows = range(cfg.prompt_len - cfg.n_action_q, cfg.prompt_len)
    zo = np.stack([head_row(c4["H"][L][p], g["final_norm"], g["lm_head"], cfg.rms_eps) for p in rows])
    lg = c4["lg"][0]
    assert rel_err(lg, zo) <= TOL
    tok_o = np.array([position_margin(z, cfg.bin_lo)[0] for z in zo])
    m_o = np.array([position_margin(z, cfg.bin_lo)[1] for z in zo])
    check_tokens(c4["tok"][0], lg, tok_o, zo, cfg.bin_lo)
    check_margins(c4["mg"][0], m_o, lg, zo, cfg.bin_lo)
    # the gate reduces with the minimum over the 56 positions
    assert abs(c4["m"][0] - float(np.min(c4["mg"][0]))) <= 1e-6
    assert c4["fire"][0] == gate_fires(float(np.min(c4["mg"][0])), cfg.theta)


# ---------------------------------------------------------------- C5
@pytest.fixture(scope="module")
def c5():
    cfg = synth.config_c5()
    s, w = _session(cfg)
    yield cfg, s, w
    s.close()


@pytest.mark.parametrize("k_static", [0, 64, 128, 192, 230])
def test_c5_sweep_masks_counts_and_layers(c5, k_static):
    from paper_2608_10824_amd import gvc
    cfg, s, w = c5
    si = synth.step_inputs(cfg, k_static, stream=k_static + 1)
    fp, ft, ids, ex = _two_steps(cfg, s, si)
    mask, n_static = s.select_static(ft, fp)
    mo, ns = _oracle_masks(cfg, si)
    assert np.array_equal(mask.cpu().numpy().astype(bool), mo)
    assert n_static.cpu().tolist() == ns.tolist() == [k_static] * cfg.batch
    s.step_prefill(ft, ids, ex, s.mask)
    assert s.read(gvc.STATE_ROWS).cpu().tolist() == [cfg.batch * (cfg.prompt_len - k_static)] * cfg.n_layers
    if k_static == 128:
        P, L = cfg.prompt_len, cfg.n_layers
        for b in (0, cfg.batch - 1):
            recomputed = [p for p in range(P) if not (1 <= p <= cfg.n_patches and mo[b, 0, p - 1])]
            sample = _sample_rows(cfg, recomputed)
            for l in (0, L - 1):
                errs = check_layer_sampled(cfg, layer_w64(w, l), state64(s, gvc.STATE_H, l, b, P),
                                           state64(s, gvc.STATE_H, l + 1, b, P), state64(s, gvc.STATE_K, l, b, P),
                                           state64(s, gvc.STATE_V, l, b, P), sample)
                print("episode", b, "layer", l, {k: "%.2e" % v for k, v in errs.items()})
                assert all(v <= TOL for v in errs.values()), (b, l, errs)
        g = glob_w64(w)
        head = s.read(gvc.STATE_HEAD_LOGITS).cpu().numpy()
        for b in range(cfg.batch):
            zo = head_row(state64(s, gvc.STATE_H, L, b, P)[P - 1], g["final_norm"], g["lm_head"], cfg.rms_eps)
            assert rel_err(head[b, 0], zo) <= TOL
    if k_static == 128:   # the batched decode of the last episode, as a float64 chain over its prompt K/V
        b = cfg.batch - 1
        P, L = cfg.prompt_len, cfg.n_layers
        Ks = [state64(s, gvc.STATE_K, l, b, P) for l in range(L)]
        Vs = [state64(s, gvc.STATE_V, l, b, P) for l in range(L)]
        hL = state64(s, gvc.STATE_H, L, b, P)[P - 1]
    tok, mg, lg = s.decode_actions(logits=True)
    torch.cuda.synchronize()
    lgn = lg.cpu().numpy()
    for b in range(cfg.batch):
        for j in range(cfg.n_decode):
            assert tok[b, j].item() == cfg.bin_lo + int(np.argmax(lgn[b, j, cfg.bin_lo:]))
    if k_static == 128:
        b = cfg.batch - 1
        zo = _oracle_decode_chain(cfg, w, hL, Ks, Vs, tok[b].cpu().numpy()[: cfg.n_decode - 1])
        err = rel_err(lgn[b], zo)
        print("episode %d batched decode chain logits rel err %.2e" % (b, err))
        assert err <= TOL


# ---------------------------------------------------------------- C3
def test_c3_episode_masks_gate_and_layers():
    """50-frame moving-rectangle episode with the decaying per-layer
    proportion and the margin gate applied (Alg. 1): every mask bit-exact,
    every gate decision equal to the threshold test on the GPU's own
    margins, and two sampled layers checked mid-episode."""
    from paper_2608_10824_amd import gvc
    cfg = synth.config_c3()
    s, w = _session(cfg)
    frames = synth.c3_episode_frames(cfg)
    ids = synth.text_ids(cfg).to(DEV)
    fdev = frames.to(DEV)
    s.step_prefill(fdev[0:1], ids)
    s.decode_actions()
    fired, full_steps = [], 0
    P, L = cfg.prompt_len, cfg.n_layers
    for t in range(1, frames.shape[0]):
        prev_m = s.read(gvc.STATE_MARGINS)[0].double().cpu().numpy()
        m, fire = s.margin_gate()
        assert fire[0] == gate_fires(float(np.mean(prev_m)), cfg.theta) or abs(np.mean(prev_m) - cfg.theta) < 1e-6
        fired.append(fire[0])
        mask, n_static = s.select_static(fdev[t:t + 1], fdev[t - 1:t])
        mo, n_o, _, _ = op.select_static(frames[t].numpy(), frames[t - 1].numpy(), cfg.patch, cfg.tau, cfg.permille())
        assert np.array_equal(mask[0].cpu().numpy().astype(bool), mo), t
        s.step_prefill(fdev[t:t + 1], ids, None, s.mask)
        rows = s.read(gvc.STATE_ROWS).cpu().tolist()
        if fire[0]:
            assert rows == [P] * L
            full_steps += 1
        else:
            assert rows == [P - (q * int(n_o)) // 1000 for q in cfg.permille()]
        if t in (10, 40):
            recomputed = [p for p in range(P) if not (1 <= p <= cfg.n_patches and not fire[0] and mo[0, p - 1])]
            for l in (0, L - 1):
                rec_l = [p for p in range(P) if not (1 <= p <= cfg.n_patches and not fire[0] and mo[l, p - 1])]
                errs = check_layer_sampled(cfg, layer_w64(w, l), state64(s, gvc.STATE_H, l, 0, P),
                                           state64(s, gvc.STATE_H, l + 1, 0, P), state64(s, gvc.STATE_K, l, 0, P),
                                           state64(s, gvc.STATE_V, l, 0, P), _sample_rows(cfg, rec_l))
                print("step", t, "layer", l, {k: "%.2e" % v for k, v in errs.items()})
                assert all(v <= TOL for v in errs.values()), (t, l, errs)
        s.decode_actions()
    print("C3 recompute rate %.3f (%d of %d steps fired)" % (full_steps / len(fired), full_steps, len(fired)))
    s.close()
