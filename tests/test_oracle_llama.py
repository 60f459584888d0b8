"""Pins of the oracle's decoder block (CPU only): closed forms and invariants
of each op, brute-force attention against torch's library routine, and the
whole decoder against the Hugging Face Llama implementation in float64."""
import numpy as np
import pytest
import torch

import synth
from oracle import llama as ol
from oracle.vla import OracleVLA, convert_weights


def test_rmsnorm_closed_forms():
    g = np.ones(16)
    for c in [0.3, -2.0, 7.5]:
        y = ol.rmsnorm(np.full(16, c), g, 1e-5)
        assert np.allclose(y, c / np.sqrt(c * c + 1e-5), rtol=0, atol=1e-15)
    x = np.random.default_rng(0).normal(size=64)
    g = np.ones(64)
    y = ol.rmsnorm(x, g, 0.0)
    assert abs(np.sqrt(np.mean(y * y)) - 1.0) < 1e-14          # unit RMS
    assert np.allclose(ol.rmsnorm(5.0 * x, g, 0.0), y, atol=1e-14)  # scale invariant
    gg = np.linspace(0.5, 1.5, 64)
    assert np.allclose(ol.rmsnorm(x, gg, 0.0), y * gg, atol=1e-14)


def test_rope_invariants_and_complex_form():
    rng = np.random.default_rng(1)
    H, dh = 3, 16
    q, k = rng.normal(size=(H, dh)), rng.normal(size=(H, dh))
    assert np.allclose(ol.rope_row(q, 0, 1e4), q, atol=0)              # identity at 0
    for pos in [1, 17, 300]:
        r = ol.rope_row(q, pos, 1e4)
        assert np.allclose(np.linalg.norm(r, axis=1), np.linalg.norm(q, axis=1), atol=1e-12)
    # the dot product depends only on the position difference
    a = np.sum(ol.rope_row(q, 9, 1e4) * ol.rope_row(k, 4, 1e4), axis=1)
    b = np.sum(ol.rope_row(q, 105, 1e4) * ol.rope_row(k, 100, 1e4), axis=1)
    assert np.allclose(a, b, atol=1e-12)
    # complex form: pair (i, i + dh/2) is the complex number x_i + j x_{i+dh/2},
    # multiplied by exp(j * pos * base^(-2i/dh))
    pos = 37
    z = q[:, : dh // 2] + 1j * q[:, dh // 2:]
    w = np.exp(1j * pos * 1e4 ** (-np.arange(dh // 2) * 2.0 / dh))
    zr = z * w
    assert np.allclose(ol.rope_row(q, pos, 1e4), np.concatenate([zr.real, zr.imag], axis=1), atol=1e-12)


def test_attention_against_torch_sdpa():
    rng = np.random.default_rng(2)
    T, H, dh = 11, 4, 8
    K, V = rng.normal(size=(T, H, dh)), rng.normal(size=(T, H, dh))
    Q = rng.normal(size=(T, H, dh))
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(Q).permute(1, 0, 2), torch.from_numpy(K).permute(1, 0, 2),
        torch.from_numpy(V).permute(1, 0, 2), is_causal=True).permute(1, 0, 2).numpy()
    for i in range(T):
        assert np.allclose(ol.attend_row(Q[i], i, K, V), ref[i], atol=1e-12)


def test_attention_special_cases():
    rng = np.random.default_rng(3)
    K, V = rng.normal(size=(5, 2, 4)), rng.normal(size=(5, 2, 4))
    q = rng.normal(size=(2, 4))
    assert np.allclose(ol.attend_row(q, 0, K, V), V[0], atol=0)       # one key
    Kc = np.repeat(K[:1], 5, axis=0)
    assert np.allclose(ol.attend_row(q, 4, Kc, V), V.mean(axis=0), atol=1e-14)  # equal keys


def test_silu_closed_form():
    assert ol.silu(0.0) == 0.0
    assert np.isclose(ol.silu(np.log(3.0)), np.log(3.0) * 0.75)


def _hf_model(cfg, w):
    from transformers import LlamaConfig, LlamaForCausalLM
    hc = LlamaConfig(vocab_size=cfg.vocab, hidden_size=cfg.d_model, intermediate_size=cfg.ffn,
                     num_hidden_layers=cfg.n_layers, num_attention_heads=cfg.n_heads,
                     num_key_value_heads=cfg.n_heads, rms_norm_eps=cfg.rms_eps,
                     max_position_embeddings=4096, hidden_act="silu", attention_bias=False,
                     mlp_bias=False, tie_word_embeddings=False,
                     rope_parameters={"rope_type": "default", "rope_theta": cfg.rope_theta})
    hc._attn_implementation = "eager"
    m = LlamaForCausalLM(hc).double().eval()
    f = lambda t: torch.nn.Parameter(t.double().clone())
    m.model.embed_tokens.weight = f(w["embed"])
    m.lm_head.weight = f(w["lm_head"])
    m.model.norm.weight = f(w["final_norm"])
    for l, lw in enumerate(w["layers"]):
        L = m.model.layers[l]
        L.self_attn.q_proj.weight = f(lw["wq"]); L.self_attn.k_proj.weight = f(lw["wk"])
        L.self_attn.v_proj.weight = f(lw["wv"]); L.self_attn.o_proj.weight = f(lw["wo"])
        L.mlp.gate_proj.weight = f(lw["wg"]); L.mlp.up_proj.weight = f(lw["wu"])
        L.mlp.down_proj.weight = f(lw["wd"])
        L.input_layernorm.weight = f(lw["attn_norm"]); L.post_attention_layernorm.weight = f(lw["ffn_norm"])
    return m


def _rel(a, b):
    return np.abs(a - b).max() / np.abs(b).max()


def test_full_forward_matches_hf_llama():
    """The oracle's full prompt pass equals Hugging Face's Llama forward on the
    same input embeddings (HF keeps norm statistics and rotary angles in fp32,
    hence the 1e-5 tolerance; a dropped term or a wrong index is O(1))."""
    cfg = synth.config_c1()
    w = synth.model_weights(cfg)
    o = OracleVLA(cfg, w)
    si = synth.step_inputs(cfg, 45)
    o.step_prefill(si["frame_t"].numpy(), si["text_ids"].numpy(), None, None)
    P = o.lay.P
    m = _hf_model(cfg, w)
    with torch.no_grad():
        out = m(inputs_embeds=torch.from_numpy(o.H[0, 0][None]), position_ids=torch.arange(P)[None],
                output_hidden_states=True, use_cache=False)
    hs = [h[0].numpy() for h in out.hidden_states]
    assert _rel(o.H[1, 0], hs[1]) < 1e-5
    logits = out.logits[0].numpy()
    mine = np.stack([ol.head_row(o.H[cfg.n_layers, 0, p], o.w["final_norm"], o.w["lm_head"], cfg.rms_eps)
                     for p in range(P)])
    assert _rel(mine, logits) < 1e-5
    assert _rel(o.head_logits[0, 0], logits[-1]) < 1e-5


def test_decode_passes_match_hf_on_extended_sequence():
    """Each single-token decode pass over the KV cache equals HF's full forward
    over the prompt plus the fed-back tokens."""
    cfg = synth.config_c1()
    w = synth.model_weights(cfg)
    o = OracleVLA(cfg, w)
    si = synth.step_inputs(cfg, 45)
    o.step_prefill(si["frame_t"].numpy(), si["text_ids"].numpy(), None, None)
    H0 = o.H[0, 0].copy()
    tokens, margins, logits = o.decode_actions()
    m = _hf_model(cfg, w)
    emb = o.w["embed"][tokens[0, :-1]]
    seq = np.concatenate([H0, emb], axis=0)
    with torch.no_grad():
        out = m(inputs_embeds=torch.from_numpy(seq[None]), position_ids=torch.arange(seq.shape[0])[None],
                use_cache=False)
    ref = out.logits[0].numpy()[o.lay.P - 1:]
    assert ref.shape == logits[0].shape
    assert _rel(logits[0], ref) < 1e-5


# ---------------------------------------------------------------- batched mode (7B-shape tests)
def test_attend_rows_matches_row_form_and_sdpa():
    """attend_rows against attend_row row by row and against torch's SDPA,
    causal and with a block of rows that see every key."""
    rng = np.random.default_rng(5)
    T, H, dh = 13, 3, 8
    K, V, Q = rng.normal(size=(T, H, dh)), rng.normal(size=(T, H, dh)), rng.normal(size=(T, H, dh))
    rows = [0, 2, 3, 7, 12]
    out = ol.attend_rows(Q[rows], rows, K, V)
    for i, r in enumerate(rows):
        assert np.allclose(out[i], ol.attend_row(Q[r], r, K, V), rtol=0, atol=1e-13)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(Q).permute(1, 0, 2), torch.from_numpy(K).permute(1, 0, 2),
        torch.from_numpy(V).permute(1, 0, 2), is_causal=True).permute(1, 0, 2).numpy()
    assert np.allclose(out, ref[rows], atol=1e-12)
    last = [12, 12, 3]
    out = ol.attend_rows(Q[[10, 11, 3]], last, K, V)
    for i, (r, l) in enumerate(zip([10, 11, 3], last)):
        assert np.allclose(out[i], ol.attend_row(Q[r], l, K, V), rtol=0, atol=1e-13)


def test_batched_layer_matches_row_layer_on_a_partial_pass():
    """layer_rows_batched over a row subset with carried-over K/V equals the
    row-at-a-time layer (outputs and the fresh K/V slots), and leaves the
    other slots alone."""
    cfg = synth.config_c1()
    w = convert_weights(synth.model_weights(cfg))["layers"][1]
    rng = np.random.default_rng(6)
    P, d, H = cfg.prompt_len, cfg.d_model, cfg.n_heads
    h = rng.normal(size=(P, d))
    K0, V0 = rng.normal(size=(P, H, d // H)), rng.normal(size=(P, H, d // H))
    rows = [0] + list(range(5, 40, 3)) + list(range(65, P))
    Ka, Va, Kb, Vb = K0.copy(), V0.copy(), K0.copy(), V0.copy()
    a = ol.layer_rows(w, h, rows, rows, Ka, Va, H, cfg.rms_eps, cfg.rope_theta)
    b = ol.layer_rows_batched(w, h, rows, rows, Kb, Vb, H, cfg.rms_eps, cfg.rope_theta)
    assert _rel(b, a) < 1e-13
    assert _rel(Kb, Ka) < 1e-13 and _rel(Vb, Va) < 1e-13
    keep = [p for p in range(P) if p not in rows]
    assert np.array_equal(Kb[keep], K0[keep]) and np.array_equal(Vb[keep], V0[keep])


def test_batched_oracle_matches_hf_llama():
    """The batched oracle's full prompt pass and decode passes against
    Hugging Face's Llama forward over the pinned embeddings."""
    cfg = synth.config_c1()
    w = synth.model_weights(cfg)
    o = OracleVLA(cfg, w, batched=True)
    si = synth.step_inputs(cfg, 45)
    o.step_prefill(si["frame_t"].numpy(), si["text_ids"].numpy(), None, None)
    H0 = o.H[0, 0].copy()
    tokens, margins, logits = o.decode_actions()
    m = _hf_model(cfg, w)
    seq = np.concatenate([H0, o.w["embed"][tokens[0, :-1]]], axis=0)
    with torch.no_grad():
        out = m(inputs_embeds=torch.from_numpy(seq[None]), position_ids=torch.arange(seq.shape[0])[None],
                output_hidden_states=True, use_cache=False)
    P = o.lay.P
    assert _rel(o.H[1, 0], out.hidden_states[1][0].numpy()[:P]) < 1e-5
    assert _rel(logits[0], out.logits[0].numpy()[P - 1:]) < 1e-5
