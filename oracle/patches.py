"""Stage 1 (static patch detection) and the applied Stage 3 proportion.

Sec. III-B, Stage 1: corresponding patches of I_t and I_{t-1} are compared
by cosine similarity; a patch whose similarity exceeds tau is static.
Sec. III-A: an H x W frame is cut into N = (H/p)(W/p) non-overlapping p x p
patches.  Stage 3: each layer reuses its own proportion of the reusable set.

Readings (the paper does not fix them):
  * the cosine is taken over the raw uint8 values of the whole p x p x 3
    patch flattened in H, W, C order; no centring;
  * "above" is strict, cos > tau, with tau = num/den evaluated exactly in
    integers; a patch pair that is all zeros on both sides counts as
    identical (cos = 1), exactly one all-zero side as dynamic;
  * layer l reuses k_l = floor(q_l * |S| / 1000) patches (q_l in per-mille),
    namely the first k_l of S ranked by cosine, highest first, ties to the
    lower patch index; so the per-layer sets are nested.
Everything here is exact integer arithmetic on Python ints.
"""
from functools import cmp_to_key
import numpy as np


def patchify(frame: np.ndarray, p: int) -> np.ndarray:
    """[views][H][W][3] uint8 -> [N][p*p*3] int64; patch index is
    view * (H/p)(W/p) + row * (W/p) + col (raster order within a view)."""
    frame = np.asarray(frame)
    V, H, W, C = frame.shape
    out = []
    for v in range(V):
        for r in range(H // p):
            for c in range(W // p):
                out.append(frame[v, r * p:(r + 1) * p, c * p:(c + 1) * p, :].reshape(-1))
    return np.stack(out).astype(np.int64)


def patch_stats(u: np.ndarray, v: np.ndarray):
    """Exact dot(u, v), |u|^2, |v|^2 per patch pair (int64 is exact here:
    588 * 255^2 < 2^26)."""
    return (u * v).sum(axis=1), (u * u).sum(axis=1), (v * v).sum(axis=1)


def is_static(dot: int, na: int, nb: int, num: int, den: int) -> bool:
    """cos = dot / sqrt(na nb) > num/den, decided exactly."""
    dot, na, nb = int(dot), int(na), int(nb)
    if na == 0 and nb == 0:
        return True
    if na == 0 or nb == 0:
        return False
    assert 0 < num <= den, "tau must lie in (0, 1]"
    if dot <= 0:
        return False
    return dot * dot * den * den > num * num * na * nb


def _cos_key(dot, na, nb):
    """(numerator^2, denominator) of cos^2 for a static patch, as Python ints."""
    dot, na, nb = int(dot), int(na), int(nb)
    if na == 0 and nb == 0:
        return 1, 1
    return dot * dot, na * nb


def rank_static(static: np.ndarray, dot, na, nb) -> list:
    """Static patch indices ordered by cosine, highest first, ties to the
    lower index (static patches have dot > 0, so cos^2 orders them)."""
    idx = [n for n in range(len(static)) if static[n]]
    keys = {n: _cos_key(dot[n], na[n], nb[n]) for n in idx}

    def cmp(i, j):
        ni, di = keys[i]
        nj, dj = keys[j]
        a, b = ni * dj, nj * di
        if a != b:
            return -1 if a > b else 1
        return -1 if i < j else (1 if i > j else 0)

    return sorted(idx, key=cmp_to_key(cmp))


def layer_reuse_masks(n_patches: int, ranked: list, permille) -> np.ndarray:
    """[L][N] bool: layer l reuses the first floor(q_l |S| / 1000) ranked patches."""
    S = len(ranked)
    masks = np.zeros((len(permille), n_patches), dtype=bool)
    for l, q in enumerate(permille):
        k = (int(q) * S) // 1000
        masks[l, ranked[:k]] = True
    return masks


def select_static(frame_t: np.ndarray, frame_prev: np.ndarray, p: int, tau, permille, exclude=None):
    """One episode: returns (masks [L][N] bool, n_static, static [N] bool, ranked).
    exclude [N] bool (Stage 2's task-relevant patches) leaves the static set
    before the ranking."""
    u = patchify(frame_t, p)
    v = patchify(frame_prev, p)
    dot, na, nb = patch_stats(u, v)
    num, den = tau
    static = np.array([is_static(dot[n], na[n], nb[n], num, den) for n in range(len(dot))])
    if exclude is not None:
        static = static & ~np.asarray(exclude, dtype=bool)
    ranked = rank_static(static, dot, na, nb)
    return layer_reuse_masks(len(dot), ranked, permille), len(ranked), static, ranked
