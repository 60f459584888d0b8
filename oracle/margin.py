"""Logit-margin gate: Eq. 1 and the test of Alg. 1.

Eq. 1: m_{t-1} is the mean over the D action tokens of step t-1 of
p1 - p2, the highest and second-highest probabilities of that token's
softmax distribution over the vocabulary (Sec. IV-A).  Alg. 1 invalidates
the whole cache and runs a full pass when m_{t-1} < theta_m.

Readings: the softmax normaliser runs over the full vocabulary, the two
candidates are the action-bin ids (the tokens the policy can emit), ties go
to the lower id; decoding is greedy over the bins; "<" is strict and a NaN
margin fires (invalidation is always safe, Sec. VI); the parallel-decoded
action chunk gates on the minimum over positions instead of the mean.
"""
import math
import numpy as np


def top2_bins(z: np.ndarray, bin_lo: int):
    """(id1, id2) of the two largest bin logits; ties to the lower id."""
    b = z[bin_lo:]
    order = sorted(range(len(b)), key=lambda i: (-b[i], i))
    return bin_lo + order[0], bin_lo + order[1]


def position_margin(z: np.ndarray, bin_lo: int, full_vocab: bool = True):
    """Greedy token and p1 - p2 for one position's logits z [V] (float64)."""
    z = np.asarray(z, dtype=np.float64)
    i1, i2 = top2_bins(z, bin_lo)
    dom = z if full_vocab else z[bin_lo:]
    M = dom.max()
    S = np.exp(dom - M).sum()
    p1 = math.exp(z[i1] - M) / S
    p2 = math.exp(z[i2] - M) / S
    return i1, p1 - p2


def reduce_margin(margins, use_min: bool = False) -> float:
    """Eq. 1's mean over positions, or the minimum."""
    m = np.asarray(margins, dtype=np.float64)
    return float(m.min() if use_min else m.mean())


def gate_fires(m: float, theta: float) -> bool:
    """Alg. 1's test m < theta_m; NaN fires."""
    return not (m >= theta)
