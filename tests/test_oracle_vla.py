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
