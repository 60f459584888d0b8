"""Pins of the oracle's Stage 1 / Stage 3 code against closed forms, brute
force and the construction of the synthetic frames (CPU only)."""
import json
import math
import os

import numpy as np
import pytest

import synth
from oracle import patches as op

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_numbers.json")))


def test_patch_count_matches_paper():
    g = GOLD["patches"]
    frame = np.zeros((1, g["img"], g["img"], 3), dtype=np.uint8)
    assert op.patchify(frame, g["p"]).shape == (g["N"], g["p"] * g["p"] * 3)


def test_patch_raster_order_and_views():
    # every pixel of patch (v, r, c) holds its own raster index: each patch
    # row must then be constant and equal to its index.
    p, side, V = 14, 8, 2
    frame = np.zeros((V, side * p, side * p, 3), dtype=np.uint8)
    for v in range(V):
        for r in range(side):
            for c in range(side):
                frame[v, r * p:(r + 1) * p, c * p:(c + 1) * p, :] = v * side * side + r * side + c
    u = op.patchify(frame, p)
    assert u.shape == (V * side * side, p * p * 3)
    assert (u == np.arange(V * side * side)[:, None]).all()
    # flattening order inside a patch is H, W, C
    f2 = np.arange(p * p * 3, dtype=np.int64).reshape(1, p, p, 3) % 251
    assert (op.patchify(f2.astype(np.uint8), p)[0] == (np.arange(p * p * 3) % 251)).all()


def _stats(u, v):
    d, a, b = op.patch_stats(np.asarray([u], dtype=np.int64), np.asarray([v], dtype=np.int64))
    return int(d[0]), int(a[0]), int(b[0])


def test_static_closed_forms():
    rng = np.random.default_rng(0)
    u = rng.integers(1, 128, 588)
    # identical -> cos = 1 -> static for every tau <= 1 except tau = 1 (strict)
    assert op.is_static(*_stats(u, u), 249, 250)
    assert not op.is_static(*_stats(u, u), 1, 1)
    # v = 2u without saturation -> cos = 1
    assert op.is_static(*_stats(u, 2 * u), 999, 1000)
    # disjoint channel support -> cos = 0
    a = np.zeros(588, dtype=np.int64); a[0::3] = 200
    b = np.zeros(588, dtype=np.int64); b[1::3] = 200
    assert not op.is_static(*_stats(a, b), 1, 1000)
    # both zero -> static; exactly one zero -> dynamic
    z = np.zeros(588, dtype=np.int64)
    assert op.is_static(*_stats(z, z), 249, 250)
    assert not op.is_static(*_stats(z, u), 1, 1000)
    # independent uniform noise: cos ~ 3/4 -> dynamic at 0.99
    n1, n2 = rng.integers(0, 256, 588), rng.integers(0, 256, 588)
    d, na, nb = _stats(n1, n2)
    assert 0.7 < d / math.sqrt(na * nb) < 0.8
    assert not op.is_static(d, na, nb, 99, 100)


def test_static_exact_at_threshold():
    # (3,4) vs (5,0) scaled: cos = 15/25 = 3/5 exactly.  Strict ">" excludes it.
    u = np.zeros(588, dtype=np.int64); u[0], u[1] = 30, 40
    v = np.zeros(588, dtype=np.int64); v[0] = 50
    st = _stats(u, v)
    assert not op.is_static(*st, 3, 5)
    assert op.is_static(*st, 599, 1000)
    assert not op.is_static(*st, 601, 1000)


def test_static_matches_float_brute_force():
    rng = np.random.default_rng(1)
    base = rng.integers(0, 256, (400, 588))
    noise = rng.integers(-3, 4, (400, 588)) * rng.integers(0, 2, (400, 1)) * rng.integers(1, 6, (400, 1))
    other = np.clip(base + noise, 0, 255)
    d, na, nb = op.patch_stats(base, other)
    cos = d / np.sqrt(na.astype(np.float64) * nb)
    for tau in [(99, 100), (249, 250), (9999, 10000)]:
        t = tau[0] / tau[1]
        for n in range(400):
            if abs(cos[n] - t) < 1e-12:
                continue
            assert op.is_static(d[n], na[n], nb[n], *tau) == (cos[n] > t)


def test_ranking_brute_force_and_ties():
    rng = np.random.default_rng(2)
    base = rng.integers(0, 256, (60, 588))
    other = np.clip(base + rng.integers(-2, 3, (60, 588)) * rng.integers(0, 3, (60, 1)), 0, 255)
    other[7] = base[7]; other[3] = base[3]      # two exact ties at cos = 1
    d, na, nb = op.patch_stats(base, other)
    static = np.array([op.is_static(d[n], na[n], nb[n], 99, 100) for n in range(60)])
    ranked = op.rank_static(static, d, na, nb)
    cos = d / np.sqrt(na.astype(np.float64) * nb)
    expect = sorted(np.nonzero(static)[0].tolist(), key=lambda n: (-round(cos[n], 12), n))
    assert ranked == expect
    assert ranked.index(3) < ranked.index(7)


def test_layer_masks_counts_and_nesting():
    ranked = [5, 2, 9, 0, 7, 3, 1]
    q = [1000, 800 - 0, 600, 500, 143, 142, 0]
    m = op.layer_reuse_masks(12, ranked, q)
    for l, ql in enumerate(q):
        k = ql * len(ranked) // 1000
        assert m[l].sum() == k
        assert set(np.nonzero(m[l])[0]) == set(ranked[:k])
        if l:
            assert (m[l] <= m[l - 1]).all()


@pytest.mark.parametrize("name,n_static", [("C1", 45), ("C2", 128), ("C4", 307)])
def test_static_set_is_the_unchanged_set(name, n_static):
    cfg = synth.ALL_CONFIGS[name]()
    si = synth.step_inputs(cfg, n_static)
    for b in range(cfg.batch):
        masks, ns, static, _ = op.select_static(si["frame_t"][b].numpy(), si["frame_prev"][b].numpy(),
                                                cfg.patch, cfg.tau, cfg.permille())
        assert ns == n_static
        assert (static == si["unchanged"][b]).all()
        assert (masks[0] == si["unchanged"][b]).all()


def test_c3_episode_changed_fraction_band():
    cfg = synth.config_c3()
    fr = synth.c3_episode_frames(cfg, n_frames=12).numpy()
    p = cfg.patch
    for t in range(1, fr.shape[0]):
        a, b = fr[t - 1, 0], fr[t, 0]
        changed = (a != b).any(axis=2).reshape(16, p, 16, p).any(axis=(1, 3)).sum()
        assert 0.05 * 256 <= changed <= 0.40 * 256
        masks, ns, static, _ = op.select_static(fr[t], fr[t - 1], p, cfg.tau, cfg.permille())
        # every unchanged patch is static; at most the changed ones are not
        assert ns >= 256 - changed
        assert masks.sum(axis=1).tolist() == [(q * ns) // 1000 for q in cfg.permille()]
