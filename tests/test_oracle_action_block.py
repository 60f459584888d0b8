"""Pins of the OFT action block in the oracle (parallel action-dimension
decoding, Sec. V-A; reading: the action-query rows attend to each other both
ways, every other row stays causal) -- CPU only."""
import numpy as np
import torch

import synth
import oracle.llama as ol
from oracle.vla import OracleVLA
from tests.test_oracle_llama import _hf_model, _rel


def _prefill(cfg, w, si, masks=None, o=None):
    o = o or OracleVLA(cfg, w)
    o.step_prefill(si["frame_t"].numpy(), si["text_ids"].numpy(), si["extra_rows"].numpy(), masks)
    return o


def _block_mask(P, a0, bidir):
    m = torch.full((P, P), float("-inf"), dtype=torch.float64)
    for i in range(P):
        m[i, : (P if bidir and i >= a0 else i + 1)] = 0
    return m[None, None]


def test_action_block_matches_hf_with_a_block_mask():
    """The whole prompt pass equals Hugging Face's Llama forward given the
    same block mask as an explicit 4-D additive mask; under HF's plain causal
    mask the action rows differ by far more than the tolerance."""
    cfg = synth.config_c4_tiny().with_(action_bidir=True)
    w = synth.model_weights(cfg)
    si = synth.step_inputs(cfg, 90)
    o = _prefill(cfg, w, si)
    P = o.lay.P
    a0 = P - cfg.n_action_q
    mine = np.stack([ol.head_row(o.H[cfg.n_layers, 0, p], o.w["final_norm"], o.w["lm_head"], cfg.rms_eps)
                     for p in range(P)])
    m = _hf_model(cfg, w)
    emb = torch.from_numpy(o.H[0, 0][None])
    with torch.no_grad():
        block = m(inputs_embeds=emb, attention_mask=_block_mask(P, a0, True), position_ids=torch.arange(P)[None],
                  use_cache=False).logits[0].numpy()
        causal = m(inputs_embeds=emb, attention_mask=_block_mask(P, a0, False), position_ids=torch.arange(P)[None],
                   use_cache=False).logits[0].numpy()
    assert _rel(mine, block) < 1e-5
    assert _rel(o.head_logits[0], block[a0:]) < 1e-5
    assert _rel(mine[:a0], causal[:a0]) < 1e-5          # rows before the block are causal either way
    assert _rel(mine[a0:], causal[a0:]) > 1e-3


def test_action_block_reaches_forward_only_inside_the_block():
    """Changing the last action-query row moves the first action row's output
    with the block and leaves it untouched without; rows before the block
    never see it."""
    cfg = synth.config_c4_tiny()
    w = synth.model_weights(cfg)
    si = synth.step_inputs(cfg, 90)
    si2 = dict(si)
    ex = si["extra_rows"].clone()
    ex[0, -1] += 0.5
    si2["extra_rows"] = ex
    L = cfg.n_layers
    for bidir in (False, True):
        c = cfg.with_(action_bidir=bidir)
        o1, o2 = _prefill(c, w, si), _prefill(c, w, si2)
        a0 = o1.lay.P - cfg.n_action_q
        assert np.array_equal(o1.H[L, 0, :a0], o2.H[L, 0, :a0])
        moved = np.abs(o1.H[L, 0, a0] - o2.H[L, 0, a0]).max()
        assert (moved > 1e-6) if bidir else (moved == 0.0)


def test_action_block_partial_pass_invariants():
    """With the block: an identical frame after a full step reproduces it
    under full reuse, and causal rows are bit-identical to the causal
    model's."""
    cfg = synth.config_c4_tiny().with_(action_bidir=True)
    w = synth.model_weights(cfg)
    si = synth.step_inputs(cfg, 90)
    o = _prefill(cfg, w, si)
    H_full = o.H.copy()
    logits_full = o.head_logits.copy()
    masks = np.ones((1, cfg.n_layers, cfg.n_patches), dtype=bool)
    _prefill(cfg, w, si, masks=masks, o=o)
    assert np.array_equal(o.H, H_full) and np.array_equal(o.head_logits, logits_full)
    oc = _prefill(cfg.with_(action_bidir=False), w, si)
    a0 = o.lay.P - cfg.n_action_q
    assert np.array_equal(oc.H[:, 0, :a0], o.H[:, 0, :a0])
