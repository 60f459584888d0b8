"""Host-side check of the compacted row lists (gvc_check_rows, CPU only).

The expected lists are built here from the rule of Alg. 1's partial forward
pass as read in this implementation: row b*P + pos is recomputed at layer l
unless episode b's cache is valid, a reuse mask is given, pos is a visual
position (1..N) and the mask marks patch pos - 1 of layer l.  The check must
accept exactly those lists and reject each planted mistake."""
import ctypes

import numpy as np
import pytest


def _lists(mask, valid, B, L, N, P):
    tot = B * P
    rows = np.zeros((L, 3, tot), dtype=np.int32)
    counts = np.zeros(L, dtype=np.int32)
    epc = np.zeros((L, B), dtype=np.int32)
    epo = np.zeros((L, B), dtype=np.int32)
    for l in range(L):
        n = 0
        for b in range(B):
            epo[l, b] = n
            for q in range(P):
                if valid[b] and mask is not None and 1 <= q <= N and mask[b, l, q - 1]:
                    continue
                rows[l, :, n] = (b * P + q, b, q)
                n += 1
            epc[l, b] = n - epo[l, b]
        counts[l] = n
    return rows, counts, epc, epo


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p).value if a is not None else 0


def _check(B, L, N, P, mask, valid, rows, counts, epc, epo):
    from paper_2608_10824_amd import gvc
    return gvc.check_rows(B, L, N, P, _ptr(mask), _ptr(valid), _ptr(rows), _ptr(counts), _ptr(epc), _ptr(epo))


@pytest.fixture
def case():
    rng = np.random.default_rng(11)
    B, L, N, P = 3, 4, 9, 14
    mask = (rng.random((B, L, N)) < 0.5).astype(np.uint8)
    valid = np.array([1, 0, 1], dtype=np.int32)
    return B, L, N, P, mask, valid


def test_rule_lists_pass(case):
    from paper_2608_10824_amd import gvc
    B, L, N, P, mask, valid = case
    rows, counts, epc, epo = _lists(mask, valid, B, L, N, P)
    assert counts.min() < B * P and counts[0] > P   # some rows reused, episode 1 (invalid) recomputes all
    assert _check(B, L, N, P, mask, valid, rows, counts, epc, epo) == gvc.GVC_OK
    # no mask: every row of every layer
    rows0, counts0, epc0, epo0 = _lists(None, valid, B, L, N, P)
    assert (counts0 == B * P).all()
    assert _check(B, L, N, P, None, valid, rows0, counts0, epc0, epo0) == gvc.GVC_OK


@pytest.mark.parametrize("mistake", ["drop_last", "swap", "wrong_episode", "wrong_position", "extra_reused_row",
                                     "episode_offset", "episode_count", "count_too_high"])
def test_planted_mistakes_fail(case, mistake):
    from paper_2608_10824_amd import gvc
    B, L, N, P, mask, valid = case
    rows, counts, epc, epo = _lists(mask, valid, B, L, N, P)
    l = 2
    if mistake == "drop_last":
        counts[l] -= 1
    elif mistake == "swap":
        rows[l, :, [3, 4]] = rows[l, :, [4, 3]]
    elif mistake == "wrong_episode":
        rows[l, 1, counts[l] - 1] = 0
    elif mistake == "wrong_position":
        rows[l, 2, 5] += 1
    elif mistake == "extra_reused_row":
        # episode 0 is valid: recompute one of its reused patches as well
        b, q = 0, 1 + int(np.flatnonzero(mask[0, l])[0])
        lst = [tuple(rows[l, :, i]) for i in range(counts[l])] + [(b * P + q, b, q)]
        lst.sort()
        counts[l] += 1
        rows[l, :, :counts[l]] = np.array(lst, dtype=np.int32).T
        epc[l, 0] += 1
        epo[l, 1:] += 1
    elif mistake == "episode_offset":
        epo[l, 2] += 1
    elif mistake == "episode_count":
        epc[l, 1] -= 1
    elif mistake == "count_too_high":
        counts[l] = B * P + 1
    assert _check(B, L, N, P, mask, valid, rows, counts, epc, epo) == gvc.GVC_EINVAL
    assert ("layer %d" % l) in gvc.last_error()


def test_bad_arguments_rejected():
    from paper_2608_10824_amd import gvc
    z = np.zeros(64, dtype=np.int32)
    assert _check(0, 1, 1, 4, None, z, z, z, z, z) == gvc.GVC_EINVAL
    assert _check(1, 1, 4, 4, None, z, z, z, z, z) == gvc.GVC_EINVAL   # N must be below P
    assert _check(1, 1, 1, 4, None, None, z, z, z, z) == gvc.GVC_EINVAL
