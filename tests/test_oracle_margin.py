"""Pins of Eq. 1 and the gate test (CPU only)."""
import json
import math
import os

import numpy as np
import pytest

from oracle import margin as om
from oracle import flops as of
import synth

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_numbers.json")))
BIN_LO = 768


def _logits_for_probs(probs, V=1024):
    """Logits whose full-vocabulary softmax puts the given probabilities on
    the first bins and nothing elsewhere."""
    z = np.full(V, -np.inf)
    z[BIN_LO:BIN_LO + len(probs)] = np.log(probs)
    return z


def test_hand_worked_margins():
    tok, m = om.position_margin(_logits_for_probs([0.5, 0.3, 0.2]), BIN_LO)
    assert tok == BIN_LO and abs(m - 0.2) < 1e-15
    for key in ("confident", "unconfident"):
        g = GOLD["margin_examples"][key]
        rest = 1.0 - g["p1"] - g["p2"]
        probs = [g["p2"], g["p1"]] + [rest / 10] * 10
        tok, m = om.position_margin(_logits_for_probs(probs), BIN_LO)
        assert tok == BIN_LO + 1
        assert abs(m - g["margin"]) < 1e-12


def test_uniform_onehot_and_bounds():
    _, m = om.position_margin(np.zeros(1024), BIN_LO)
    assert m == 0.0
    z = np.zeros(1024); z[900] = 800.0
    tok, m = om.position_margin(z, BIN_LO)
    assert tok == 900 and m == 1.0
    rng = np.random.default_rng(0)
    for _ in range(50):
        z = rng.normal(size=1024) * rng.uniform(0.1, 20)
        _, m = om.position_margin(z, BIN_LO)
        assert 0.0 <= m <= 1.0


def test_ties_go_to_lower_id():
    z = np.zeros(1024); z[800] = z[790] = 3.0
    tok, m = om.position_margin(z, BIN_LO)
    assert tok == 790 and m == 0.0


def test_non_bin_mass_only_enters_normaliser():
    rng = np.random.default_rng(1)
    z = rng.normal(size=1024)
    z_bins_only = z.copy(); z_bins_only[:BIN_LO] = -np.inf
    # full-vocab normaliser equals bins-only when non-bins carry no mass
    t1, m1 = om.position_margin(z_bins_only, BIN_LO, full_vocab=True)
    t2, m2 = om.position_margin(z, BIN_LO, full_vocab=False)
    assert t1 == t2 and abs(m1 - m2) < 1e-15
    # a non-bin logit above every bin never becomes the token
    z[5] = 50.0
    t3, m3 = om.position_margin(z, BIN_LO, full_vocab=True)
    assert t3 >= BIN_LO and m3 < 1e-15


def test_reduce_and_gate():
    assert om.reduce_margin([0.2, 0.4, 0.9]) == pytest.approx(0.5)
    assert om.reduce_margin([0.2, 0.4, 0.9], use_min=True) == 0.2
    assert om.gate_fires(0.099, 0.1) and not om.gate_fires(0.1, 0.1)    # strict <
    assert om.gate_fires(float("nan"), 0.1)
    assert not om.gate_fires(0.0, 0.0)          # theta <= 0 never fires
    assert om.gate_fires(1.0, 1.0000001)        # theta > 1 always fires


def test_compute_accounting_matches_tables():
    """One multiply-add per backbone parameter per prompt token reproduces the
    tables' full-inference figures, and the gated figure is the blend of
    cached and full steps at the reported fire rate."""
    t1, t2 = GOLD["table1_openvla_tflops"], GOLD["table2_oft_tflops"]
    c2, c4 = synth.config_c2(), synth.config_c4()
    full = of.paper_step_tflops(c2, c2.prompt_len)
    assert min(t1["full"].values()) <= full <= max(t1["full"].values())
    assert abs(of.paper_step_tflops(c4, c4.prompt_len) - t2["full"]["avg"]) < 0.01
    f = GOLD["long_fire_rate"]["value"]
    blend = (1 - f) * t1["cache"]["long"] + f * t1["full"]["long"]
    assert abs(blend - t1["gated"]["long"]) < 0.01
    # 2*MAC count of a full C2 step is twice the per-token-parameter count of
    # the decoder layers plus attention, head and decode passes
    rows = [c2.prompt_len] * c2.n_layers
    qpos = [list(range(c2.prompt_len))] * c2.n_layers
    fl = of.step_flops(c2, rows, qpos, 1, 0, c2.prompt_len)
    layer_params = c2.n_layers * (4 * c2.d_model ** 2 + 3 * c2.d_model * c2.ffn)
    assert fl > 2 * layer_params * c2.prompt_len
