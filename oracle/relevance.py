"""Stage 2 (task-relevant filtering) -- test infrastructure: a plain float64
statement of what the GPU path computes, used only by tests/, smoke() and the
benchmark's CPU baseline.

Sec. III-B, Stage 2: static patches that receive high attention from the
language tokens are taken out of the candidate set, because they matter for
the task and should be recomputed; what is left is the reusable set.  The
paper's setup (Sec. V-A) keeps k = 120 such patches.

Readings (the paper gives no formula):
  * the signal is the previous step's prompt pass: in every layer l and head
    h, each instruction token after the image (prompt positions N+1 ..
    N+n_text-1; position 0 precedes the image and cannot attend to it) has a
    softmax distribution over the keys up to its position; the probability
    it puts on visual key n (position n + 1), summed over those tokens, is
    a[l][h][n];
  * a patch's score is the sum of a[l][h][n] over all layers and heads;
  * the k patches with the highest scores are task-relevant (ties to the
    lower patch index); they leave the static set before Stage 1's per-layer
    ranking, so k_l = floor(q_l |S'| / 1000) counts the filtered set S';
  * with no earlier pass, or no instruction token after the image, there is
    no signal and nothing is filtered.
"""
import numpy as np

from .llama import rmsnorm, rope_row


def text_vision_attention(w_l: dict, h_in: np.ndarray, K: np.ndarray, n_patches: int, n_text: int,
                          n_heads: int, eps: float, base: float) -> np.ndarray:
    """a[h][n] of one layer: h_in [P][d] is the layer input, K [T][H][d_h]
    the layer's keys after this pass (rotated, absolute positions)."""
    d = h_in.shape[-1]
    dh = d // n_heads
    a = np.zeros((n_heads, n_patches))
    for p in range(n_patches + 1, n_patches + n_text):
        q = rope_row((w_l["wq"] @ rmsnorm(h_in[p], w_l["attn_norm"], eps)).reshape(n_heads, dh), p, base)
        s = np.einsum("hd,thd->ht", q, K[: p + 1]) / np.sqrt(dh)
        s = s - s.max(axis=1, keepdims=True)
        prob = np.exp(s)
        prob = prob / prob.sum(axis=1, keepdims=True)
        a += prob[:, 1: n_patches + 1]
    return a


def relevant_patches(score: np.ndarray, k: int) -> np.ndarray:
    """[N] bool: the k highest scores, ties to the lower index."""
    n = len(score)
    order = sorted(range(n), key=lambda i: (-score[i], i))
    out = np.zeros(n, dtype=bool)
    out[order[: max(0, min(k, n))]] = True
    return out
