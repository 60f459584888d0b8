"""Checks at the full 7B sizes (32 layers, d=4096, 32 heads, FFN 11008,
vocab 32000) that need no oracle state, in the launch configuration the
benchmark times:
  * every reuse mask and static count, bit-exact against the oracle's
    Stage 1 (integer path), on C2, C4, all five C5 reuse levels and all 49
    steps of the C3 episode;
  * per-layer recompute counts;
  * rows reused at a layer keep their K/V and layer output bit-identical to
    the previous step (nothing rewrites them);
  * the GPU's tokens are the argmax of its own logits, and each C3 gate
    decision is the threshold test on the GPU's own margins;
  * the ViT front end's layer-0 rows against the oracle's own front end.
Every element of the state against the oracle's own Alg. 1 walk is in
test_gpu_chain.py.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import patches as op
from oracle.margin import gate_fires
from tests._parity import TOL, rel_err, glob_w64, state64

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def _session(cfg):
    from paper_2608_10824_amd.session import Session
    w = synth.model_weights(cfg, device=DEV)
    return Session(cfg, w, device=DEV), w


def _two_steps(cfg, s, si):
    """Full step on frame_prev (gate kept); returns the device inputs."""
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


def _argmax_tokens(cfg, tok, lg):
    for b in range(tok.shape[0]):
        for j in range(tok.shape[1]):
            assert tok[b, j] == cfg.bin_lo + int(np.argmax(lg[b, j, cfg.bin_lo:]))


# ---------------------------------------------------------------- C2
def test_c2_masks_counts_and_reused_rows_untouched():
    """C2 at 50% reuse: masks and counts against the oracle's Stage 1, and
    every reused row's K, V and layer output left bit-identical by the
    partial step, at every layer."""
    from paper_2608_10824_amd import gvc
    cfg = synth.config_c2()
    s, w = _session(cfg)
    del w
    si = synth.step_inputs(cfg, 128)
    fp, ft, ids, ex = _two_steps(cfg, s, si)
    P, L = cfg.prompt_len, cfg.n_layers
    before = [(state64(s, gvc.STATE_K, l, 0, P), state64(s, gvc.STATE_V, l, 0, P),
               state64(s, gvc.STATE_H, l + 1, 0, P)) for l in range(L)]
    mask, n_static = s.select_static(ft, fp)
    mo, ns = _oracle_masks(cfg, si)
    assert np.array_equal(mask.cpu().numpy().astype(bool), mo)
    assert n_static.cpu().tolist() == ns.tolist() == [128]
    assert (mo[0, 0] == si["unchanged"][0]).all()
    s.step_prefill(ft, ids, ex, s.mask)
    assert s.read(gvc.STATE_ROWS).cpu().tolist() == [P - 128] * L
    reused = [1 + n for n in np.nonzero(mo[0, 0])[0]]
    for l in range(L):
        K0, V0, H0 = before[l]
        assert np.array_equal(state64(s, gvc.STATE_K, l, 0, P)[reused], K0[reused])
        assert np.array_equal(state64(s, gvc.STATE_V, l, 0, P)[reused], V0[reused])
        assert np.array_equal(state64(s, gvc.STATE_H, l + 1, 0, P)[reused], H0[reused])
    tok, mg, lg = s.decode_actions(logits=True)
    torch.cuda.synchronize()
    _argmax_tokens(cfg, tok.cpu().numpy(), lg.cpu().numpy())
    s.close()


# ---------------------------------------------------------------- C2 with the ViT front end
def test_c2v_front_end_layer0_rows():
    """ViT-L/14-shaped front end at the 7B shape: the layer-0 input of every
    prompt row (visual rows from the GPU's ViT and projector) against the
    oracle's own front end on the same frame, after a full and after a
    partial step (every element; the decoder above it is followed element
    by element in test_gpu_chain.py)."""
    from paper_2608_10824_amd import gvc
    from oracle.vit import visual_embeddings
    from oracle.vla import convert_weights
    cfg = synth.config_c2v()
    s, w = _session(cfg)
    si = synth.step_inputs(cfg, 128)
    fp, ft, ids, ex = _two_steps(cfg, s, si)
    P, N = cfg.prompt_len, cfg.n_patches
    vw = convert_weights({"vit": w["vit"]})["vit"]
    g = glob_w64(w)
    del w
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
    s.close()


# ---------------------------------------------------------------- C4
@pytest.mark.parametrize("mode", ["causal", "bidir"])
def test_c4_masks_counts_and_argmax(mode):
    from paper_2608_10824_amd import gvc
    cfg = synth.config_c4().with_(action_bidir=mode == "bidir")
    s, w = _session(cfg)
    del w
    si = synth.step_inputs(cfg, 307)
    fp, ft, ids, ex = _two_steps(cfg, s, si)
    mask, n_static = s.select_static(ft, fp)
    mo, ns = _oracle_masks(cfg, si)
    assert np.array_equal(mask.cpu().numpy().astype(bool), mo) and n_static.cpu().tolist() == ns.tolist() == [307]
    s.step_prefill(ft, ids, ex, s.mask)
    assert s.read(gvc.STATE_ROWS).cpu().tolist() == [cfg.prompt_len - 307] * cfg.n_layers
    tok, mg, lg = s.decode_actions(logits=True)
    m, fire = s.margin_gate()
    tok, mg, lg = tok.cpu().numpy(), mg.cpu().numpy(), lg.cpu().numpy()
    _argmax_tokens(cfg, tok, lg)
    # the gate reduces with the minimum over the 56 positions
    assert abs(m[0] - float(np.min(mg[0]))) <= 1e-6
    assert fire[0] == gate_fires(float(np.min(mg[0])), cfg.theta)
    s.close()


# ---------------------------------------------------------------- C5
@pytest.fixture(scope="module")
def c5():
    cfg = synth.config_c5()
    s, w = _session(cfg)
    del w
    yield cfg, s
    s.close()


@pytest.mark.parametrize("k_static", [0, 64, 128, 192, 230])
def test_c5_sweep_masks_counts_and_argmax(c5, k_static):
    from paper_2608_10824_amd import gvc
    cfg, s = c5
    si = synth.step_inputs(cfg, k_static, stream=k_static + 1)
    fp, ft, ids, ex = _two_steps(cfg, s, si)
    mask, n_static = s.select_static(ft, fp)
    mo, ns = _oracle_masks(cfg, si)
    assert np.array_equal(mask.cpu().numpy().astype(bool), mo)
    assert n_static.cpu().tolist() == ns.tolist() == [k_static] * cfg.batch
    s.step_prefill(ft, ids, ex, s.mask)
    assert s.read(gvc.STATE_ROWS).cpu().tolist() == [cfg.batch * (cfg.prompt_len - k_static)] * cfg.n_layers
    tok, mg, lg = s.decode_actions(logits=True)
    torch.cuda.synchronize()
    _argmax_tokens(cfg, tok.cpu().numpy(), lg.cpu().numpy())


# ---------------------------------------------------------------- C3
def test_c3_episode_masks_and_gate():
    """50-frame moving-rectangle episode with the decaying per-layer
    proportion and the margin gate applied (Alg. 1): every mask bit-exact
    against the oracle's Stage 1, every recompute count, and every gate
    decision equal to the threshold test on the GPU's own margins."""
    from paper_2608_10824_amd import gvc
    cfg = synth.config_c3()
    s, w = _session(cfg)
    del w
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
        s.decode_actions()
    print("C3 recompute rate %.3f (%d of %d steps fired)" % (full_steps / len(fired), full_steps, len(fired)))
    assert 0 < full_steps < len(fired)
    s.close()
