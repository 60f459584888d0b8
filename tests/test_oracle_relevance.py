"""Pins of the Stage 2 oracle (task-relevant filtering, Sec. III-B) against
closed forms, a library sort and invariants -- CPU only."""
import numpy as np
import pytest

import synth
from oracle.relevance import text_vision_attention, relevant_patches
from oracle.vla import OracleVLA


def _tiny_layer(rng, d, F):
    return {"wq": rng.standard_normal((d, d)) / np.sqrt(d), "wk": rng.standard_normal((d, d)) / np.sqrt(d),
            "wv": rng.standard_normal((d, d)) / np.sqrt(d), "wo": rng.standard_normal((d, d)) / np.sqrt(d),
            "wg": rng.standard_normal((F, d)) / np.sqrt(d), "wu": rng.standard_normal((F, d)) / np.sqrt(d),
            "wd": rng.standard_normal((d, F)) / np.sqrt(F), "attn_norm": 1.0 + 0.1 * rng.standard_normal(d),
            "ffn_norm": 1.0 + 0.1 * rng.standard_normal(d)}


def test_uniform_scores_closed_form():
    """All keys zero: every score is 0, so instruction token p spreads 1/(p+1)
    over keys 0..p and a[h][n] = sum_p 1/(p+1), the same for every patch."""
    rng = np.random.default_rng(0)
    N, T, H, dh = 9, 5, 2, 8
    d = H * dh
    P = 1 + N + T - 1
    w = _tiny_layer(rng, d, 24)
    h_in = rng.standard_normal((P, d))
    K = np.zeros((P, H, dh))
    a = text_vision_attention(w, h_in, K, N, T, H, 1e-5, 10000.0)
    expect = sum(1.0 / (p + 1) for p in range(N + 1, N + T))
    assert a.shape == (H, N)
    assert np.allclose(a, expect, rtol=0, atol=1e-14)


def test_visual_mass_is_a_probability_share():
    """Each instruction row's distribution sums to 1, so the visual share
    summed over the T-1 rows lies in (0, T-1]; a key aligned with every
    query dominates its column."""
    rng = np.random.default_rng(1)
    N, T, H, dh = 12, 4, 3, 8
    d = H * dh
    P = 1 + N + T - 1
    w = _tiny_layer(rng, d, 24)
    h_in = rng.standard_normal((P, d))
    K = rng.standard_normal((P, H, dh))
    a = text_vision_attention(w, h_in, K, N, T, H, 1e-5, 10000.0)
    assert np.all(a > 0) and np.all(a.sum(axis=1) < T - 1)
    # a huge key at visual position 1 + 5 in the direction of head 0's queries
    K2 = K.copy()
    from oracle.llama import rmsnorm, rope_row
    qsum = np.zeros(dh)
    for p in range(N + 1, N + T):
        q = rope_row((w["wq"] @ rmsnorm(h_in[p], w["attn_norm"], 1e-5)).reshape(H, dh), p, 10000.0)
        qsum += q[0] / np.linalg.norm(q[0])
    K2[1 + 5, 0] = 1e3 * qsum
    a2 = text_vision_attention(w, h_in, K2, N, T, H, 1e-5, 10000.0)
    assert a2[0, 5] > (T - 1) - 1e-6
    assert np.allclose(a2[1:], a[1:])


@pytest.mark.parametrize("k", [0, 1, 7, 120, 300])
def test_relevant_is_a_stable_descending_sort(k):
    rng = np.random.default_rng(k)
    score = rng.integers(0, 20, size=256).astype(np.float64)   # many ties
    got = relevant_patches(score, k)
    order = np.argsort(-score, kind="stable")                   # ties keep the lower index first
    expect = np.zeros(256, dtype=bool)
    expect[order[:k]] = True
    assert np.array_equal(got, expect)
    assert got.sum() == min(k, 256)


def test_stage2_filters_the_top_k_and_k0_is_stage1():
    cfg = synth.config_c1().with_(n_layers=1, task_topk=5)
    w = synth.model_weights(cfg)
    si = synth.step_inputs(cfg, 40)
    o = OracleVLA(cfg, w)
    ft, fp, ids = si["frame_t"].numpy(), si["frame_prev"].numpy(), si["text_ids"].numpy()
    o.step_prefill(fp, ids)
    assert o.tv.shape == (1, 1, cfg.n_heads, cfg.n_patches) and np.all(o.tv >= 0)
    assert np.all(o.tv.sum(axis=3) <= cfg.n_text - 1 + 1e-9)
    m2, n2 = o.select_static(ft, fp)
    # Stage 1 alone (k = 0)
    o0 = OracleVLA(cfg.with_(task_topk=0), w)
    m1, n1 = o0.select_static(ft, fp)
    score = o.tv[0].sum(axis=(0, 1))
    rel = relevant_patches(score, 5)
    from oracle.patches import select_static
    _, _, static1, _ = select_static(ft[0], fp[0], cfg.patch, cfg.tau, cfg.permille())
    assert n2[0] == int((static1 & ~rel).sum()) and n1[0] == int(static1.sum())
    assert not np.any(m2[0] & rel[None, :])
    # no earlier pass: nothing filtered
    o_fresh = OracleVLA(cfg, w)
    m3, n3 = o_fresh.select_static(ft, fp)
    assert np.array_equal(m3, m1) and n3[0] == n1[0]


# --- Stage 3 from attention entropy ---------------------------------------

from oracle.relevance import text_attention_entropy, entropy_permille  # noqa: E402


def test_entropy_uniform_is_one():
    """All keys zero: every instruction row is uniform over its p + 1 keys, so
    its normalized entropy is exactly 1 and the per-head sum is n_text - 1;
    such layers reuse nothing."""
    rng = np.random.default_rng(2)
    N, T, H, dh = 9, 5, 2, 8
    d = H * dh
    P = 1 + N + T - 1
    w = _tiny_layer(rng, d, 24)
    e = text_attention_entropy(w, rng.standard_normal((P, d)), np.zeros((P, H, dh)), N, T, H, 1e-5, 10000.0)
    assert np.allclose(e, T - 1, rtol=0, atol=1e-12)
    assert entropy_permille(np.tile(e, (3, 1)), T - 1) == [0, 0, 0]


def test_entropy_three_key_closed_form():
    """One instruction row (position 2) over keys 0, 1, 2: key 1 gets score
    alpha per head, the others 0, so p = (1, e^alpha, 1) / (e^alpha + 2) and
    the normalized entropy is (log Z - alpha e^alpha / Z) / log 3."""
    rng = np.random.default_rng(3)
    N, T, H, dh = 1, 2, 3, 8
    d = H * dh
    P = 3
    w = _tiny_layer(rng, d, 24)
    h_in = rng.standard_normal((P, d))
    from oracle.llama import rmsnorm, rope_row
    q = rope_row((w["wq"] @ rmsnorm(h_in[2], w["attn_norm"], 1e-5)).reshape(H, dh), 2, 10000.0)
    alphas = np.array([0.0, 1.5, -2.0])
    K = np.zeros((P, H, dh))
    for h in range(H):
        K[1, h] = alphas[h] * np.sqrt(dh) * q[h] / (q[h] @ q[h])
    e = text_attention_entropy(w, h_in, K, N, T, H, 1e-5, 10000.0)
    Z = np.exp(alphas) + 2.0
    expect = (np.log(Z) - alphas * np.exp(alphas) / Z) / np.log(3.0)
    assert np.allclose(e, expect, rtol=0, atol=1e-12)
    assert abs(e[0] - 1.0) < 1e-12


def test_entropy_dominant_key_is_zero():
    """A key aligned with every instruction query of head 0 takes all of its
    probability, so head 0's entropy vanishes; other heads are untouched."""
    rng = np.random.default_rng(4)
    N, T, H, dh = 12, 4, 3, 8
    d = H * dh
    P = 1 + N + T - 1
    w = _tiny_layer(rng, d, 24)
    h_in = rng.standard_normal((P, d))
    K = rng.standard_normal((P, H, dh))
    e = text_attention_entropy(w, h_in, K, N, T, H, 1e-5, 10000.0)
    assert np.all(e > 0) and np.all(e < T - 1)
    from oracle.llama import rmsnorm, rope_row
    qsum = np.zeros(dh)
    for p in range(N + 1, N + T):
        q = rope_row((w["wq"] @ rmsnorm(h_in[p], w["attn_norm"], 1e-5)).reshape(H, dh), p, 10000.0)
        qsum += q[0] / np.linalg.norm(q[0])
    K2 = K.copy()
    K2[1 + 5, 0] = 1e3 * qsum
    e2 = text_attention_entropy(w, h_in, K2, N, T, H, 1e-5, 10000.0)
    assert e2[0] < 1e-6
    assert np.allclose(e2[1:], e[1:])


def test_entropy_permille_is_a_halving_average():
    """s_l = s_{l-1} + (u_l - s_{l-1}) / 2 unrolled: s_l = 2^-l u_0 +
    sum_{1<=j<=l} 2^-(l-j+1) u_j; a single low-entropy first layer halves
    down the stack; values clamp into [0, 1000]."""
    H, n = 4, 3
    u = np.array([1.0, 0.0, 0.0, 0.0])
    ent = np.repeat(((1.0 - u) * n)[:, None], H, axis=1)    # every head's sum over n tokens is (1 - u_l) n
    assert entropy_permille(ent, n) == [1000, 500, 250, 125]
    rng = np.random.default_rng(5)
    u = rng.uniform(0.05, 0.95, size=7)
    ent = np.repeat(((1.0 - u) * n)[:, None], H, axis=1)
    got = entropy_permille(ent, n)
    for l in range(7):
        s = 2.0 ** -l * u[0] + sum(2.0 ** -(l - j + 1) * u[j] for j in range(1, l + 1))
        assert got[l] == int(np.floor(1000 * s)) or abs(1000 * s - round(1000 * s)) < 1e-9
    assert entropy_permille(np.full((2, H), 2.0 * n), n) == [0, 0]              # E = 2 > 1 clamps to 0
    assert entropy_permille(np.full((2, H), -1.0), n) == [1000, 1000]           # E < 0 clamps to 1000


def test_stage3_proportions_drive_the_masks():
    cfg = synth.config_c1().with_(n_layers=3, entropy_reuse=True)
    w = synth.model_weights(cfg)
    si = synth.step_inputs(cfg, 40)
    ft, fp, ids = si["frame_t"].numpy(), si["frame_prev"].numpy(), si["text_ids"].numpy()
    o = OracleVLA(cfg, w)
    # no earlier pass: the fixed proportions
    m0, n0 = o.select_static(ft, fp)
    o_fixed = OracleVLA(cfg.with_(entropy_reuse=False), w)
    mf, nf = o_fixed.select_static(ft, fp)
    assert np.array_equal(m0, mf) and n0[0] == nf[0]
    o.step_prefill(fp, ids)
    assert o.ent.shape == (1, 3, cfg.n_heads)
    assert np.all(o.ent > 0) and np.all(o.ent < cfg.n_text - 1)
    q = o.layer_permille(0)
    assert len(q) == 3 and all(0 <= v <= 1000 for v in q)
    m, n = o.select_static(ft, fp)
    assert n[0] == nf[0]                                   # Stage 3 does not change |S|
    for l in range(3):
        assert m[0, l].sum() == (q[l] * n[0]) // 1000
    # masks are nested prefixes of the same ranking: a larger share reuses a superset
    order = np.argsort([-v for v in q], kind="stable")
    for a, b in zip(order[:-1], order[1:]):
        assert not np.any(m[0, b] & ~m[0, a])
