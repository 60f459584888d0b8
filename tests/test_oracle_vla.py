"""Invariants of the oracle's control step (Alg. 1) on the tiny config (CPU)."""
import copy

import numpy as np
import pytest

import synth
from oracle.vla import OracleVLA
from oracle import patches as op


@pytest.fixture(scope="module")
def c1():
    cfg = synth.config_c1()
    w = synth.model_weights(cfg)
    si = synth.step_inputs(cfg, 45)
    return cfg, w, si


def _full(cfg, w, frame, si):
    o = OracleVLA(cfg, w)
    o.step_prefill(frame, si["text_ids"].numpy(), None, None)
    return o


def test_empty_mask_is_full_recompute(c1):
    cfg, w, si = c1
    ft, fp = si["frame_t"].numpy(), si["frame_prev"].numpy()
    a = _full(cfg, w, fp, si)
    a.step_prefill(ft, si["text_ids"].numpy(), None, np.zeros((1, cfg.n_layers, cfg.n_patches), bool))
    b = _full(cfg, w, ft, si)
    assert np.array_equal(a.H, b.H) and np.array_equal(a.K, b.K) and np.array_equal(a.V, b.V)
    assert np.array_equal(a.head_logits, b.head_logits)


def test_invalid_cache_ignores_mask(c1):
    cfg, w, si = c1
    ft, fp = si["frame_t"].numpy(), si["frame_prev"].numpy()
    a = _full(cfg, w, fp, si)
    masks, _ = a.select_static(ft, fp)
    a.invalidate()
    a.step_prefill(ft, si["text_ids"].numpy(), None, masks)
    b = _full(cfg, w, ft, si)
    assert np.array_equal(a.H, b.H) and np.array_equal(a.head_logits, b.head_logits)
    assert (a.recomputed == cfg.prompt_len).all()


def test_identical_frame_full_reuse_reproduces_previous_step(c1):
    cfg, w, si = c1
    fp = si["frame_prev"].numpy()
    a = _full(cfg, w, fp, si)
    H, K, V, z = a.H.copy(), a.K.copy(), a.V.copy(), a.head_logits.copy()
    masks, ns = a.select_static(fp, fp)
    assert ns[0] == cfg.n_patches and masks.all()
    a.step_prefill(fp, si["text_ids"].numpy(), None, masks)
    assert (a.recomputed == cfg.n_text).all()
    assert np.array_equal(a.K, K) and np.array_equal(a.V, V) and np.array_equal(a.H, H)
    assert np.array_equal(a.head_logits, z)


def test_identical_frame_any_schedule_equals_full(c1):
    cfg, w, si = c1
    fp = si["frame_prev"].numpy()
    a = _full(cfg, w, fp, si)
    ref = (a.H.copy(), a.K.copy(), a.head_logits.copy())
    masks, _ = a.select_static(fp, fp, permille=[900, 200])
    assert masks[0, 0].sum() == 57 and masks[0, 1].sum() == 12
    a.step_prefill(fp, si["text_ids"].numpy(), None, masks)
    assert np.array_equal(a.H, ref[0]) and np.array_equal(a.K, ref[1])
    assert np.array_equal(a.head_logits, ref[2])


def test_reused_patch_layer0_kv_equals_recomputed(c1):
    cfg, w, si = c1
    ft, fp = si["frame_t"].numpy(), si["frame_prev"].numpy()
    a = _full(cfg, w, fp, si)
    masks, _ = a.select_static(ft, fp)
    a.step_prefill(ft, si["text_ids"].numpy(), None, masks)
    b = _full(cfg, w, ft, si)
    reused_pos = 1 + np.nonzero(masks[0, 0])[0]
    # layer-0 K/V of an unchanged patch depend only on its pixels and position
    assert np.allclose(a.K[0, 0, reused_pos], b.K[0, 0, reused_pos], rtol=0, atol=1e-13)
    assert np.allclose(a.V[0, 0, reused_pos], b.V[0, 0, reused_pos], rtol=0, atol=1e-13)
    # recomputed rows are the text rows plus the changed patches
    assert (a.recomputed == cfg.prompt_len - 45).all()


def test_gate_theta_limits_and_first_step(c1):
    cfg, w, si = c1
    ft, fp = si["frame_t"].numpy(), si["frame_prev"].numpy()
    # theta > 1: every step fires, so the reuse step equals full inference
    a = OracleVLA(cfg, w)
    a.control_step(fp, None, si["text_ids"].numpy(), first=True)
    tok_a, m_a, fire = a.control_step(ft, fp, si["text_ids"].numpy(), theta=1.5)
    assert fire.all() and (a.recomputed == cfg.prompt_len).all()
    b = OracleVLA(cfg, w)
    b.control_step(ft, None, si["text_ids"].numpy(), first=True)
    assert np.array_equal(a.H, b.H) and np.array_equal(tok_a, b.tokens) and np.array_equal(m_a, b.margins)
    # theta <= 0 never fires: the method is plain visual-similarity caching
    c = OracleVLA(cfg, w)
    c.control_step(fp, None, si["text_ids"].numpy(), first=True)
    _, _, fire = c.control_step(ft, fp, si["text_ids"].numpy(), theta=0.0)
    assert not fire.any() and (c.recomputed == cfg.prompt_len - 45).all()


def test_one_step_lag(c1):
    """The margin of step t-1 decides step t: a step's own margin never
    affects that step."""
    cfg, w, si = c1
    ft, fp = si["frame_t"].numpy(), si["frame_prev"].numpy()
    a = OracleVLA(cfg, w)
    a.control_step(fp, None, si["text_ids"].numpy(), first=True)
    m_prev = float(np.mean(a.margins[0]))
    theta = m_prev + 1e-9          # just above the previous step's margin
    _, m_now, fire = a.control_step(ft, fp, si["text_ids"].numpy(), theta=theta)
    assert fire[0]
    b = OracleVLA(cfg, w)
    b.control_step(fp, None, si["text_ids"].numpy(), first=True)
    _, _, fire_b = b.control_step(ft, fp, si["text_ids"].numpy(), theta=m_prev - 1e-9)
    assert not fire_b[0]


def test_gate_invalidates_only_fired_episodes():
    cfg = synth.config_c1().with_(batch=2)
    w = synth.model_weights(cfg)
    o = OracleVLA(cfg, w)
    o.valid[:] = True
    o.margins = np.array([[0.5] * 7, [0.01] * 7])
    m, fire = o.margin_gate(0.1)
    assert list(fire) == [False, True] and list(o.valid) == [True, False]
    o.valid[:] = True
    _, fire = o.margin_gate(0.1, force=[1, 0])
    assert list(fire) == [True, False] and list(o.valid) == [False, True]


# ---------------------------------------------------------------- embeddings (Sec. III-A)
def test_embed_row_single_pixel_closed_form():
    """A frame that is zero except one pixel: only the embedding of the patch
    holding it is non-zero, and it equals the patch projection's column for
    that pixel's place in the patch's H, W, C flattening, times value / 255.
    Pins the raster order of the patches, the view-major order, the H, W, C
    flattening within a patch and the 1/255 scaling independently of the
    oracle's own patch extraction."""
    cfg = synth.config_c1().with_(n_views=2)
    w = synth.model_weights(cfg)
    o = OracleVLA(cfg, w)
    p, side = cfg.patch, cfg.patches_per_side
    ids = np.zeros((1, cfg.n_text), dtype=np.int64)
    W = w["patch_proj"].double().numpy()
    for (v, y, x, c, val) in [(0, 0, 0, 0, 255), (0, 13, 1, 2, 17), (1, 20, 97, 1, 200), (1, 111, 111, 2, 3)]:
        frame = np.zeros((1, cfg.n_views, cfg.img, cfg.img, 3), dtype=np.uint8)
        frame[0, v, y, x, c] = val
        n_hit = v * side * side + (y // p) * side + x // p
        col = (y % p) * p * 3 + (x % p) * 3 + c
        for n in range(cfg.n_patches):
            e = o.embed_row(0, 1 + n, frame, ids, None)
            if n == n_hit:
                assert np.allclose(e, W[:, col] * (val / 255.0), rtol=1e-15, atol=0)
            else:
                assert not e.any()


def test_embed_rows_of_a_prompt(c1):
    """Every prompt row at layer 0: visual rows are patchify(frame)/255 times
    the patch projection (patchify is pinned on its own), text token 0 sits at
    position 0 and tokens 1.. after the image, given extra rows after the
    text; the prompt pass stores exactly these rows as H[0]."""
    cfg = synth.config_c1().with_(n_proprio=1, n_action_q=2)
    w = synth.model_weights(cfg)
    si = synth.step_inputs(cfg, 45)
    frame, ids = si["frame_t"].numpy(), si["text_ids"].numpy()
    extra = si["extra_rows"].numpy()
    o = OracleVLA(cfg, w)
    o.step_prefill(frame, ids, extra, None)
    N, T = cfg.n_patches, cfg.n_text
    Wp, E = w["patch_proj"].double().numpy(), w["embed"].double().numpy()
    vis = op.patchify(frame[0], cfg.patch).astype(np.float64) / 255.0 @ Wp.T
    H0 = o.H[0, 0]
    assert np.allclose(H0[1:N + 1], vis, rtol=0, atol=1e-14)
    assert np.array_equal(H0[0], E[ids[0, 0]])
    assert np.array_equal(H0[N + 1:N + T], E[ids[0, 1:]])
    assert np.array_equal(H0[N + T:], extra[0].astype(np.float64))
    for pos in (0, 1, N, N + 1, N + T):
        assert np.array_equal(o.embed_row(0, pos, frame, ids, extra), H0[pos])
