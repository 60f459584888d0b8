"""Stage 2 (task-relevant filtering) and Stage 3 computed from attention
entropy -- test infrastructure: a plain float64 statement of what the GPU
path computes, used only by tests/, smoke() and the benchmark's CPU baseline.

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

Sec. III-B, Stage 3: each layer's reuse proportion follows its normalized
attention entropy -- low-entropy layers reuse more, high-entropy layers
recompute more -- smoothed so that it does not jump from layer to layer.
Readings (the paper gives neither the entropy nor the smoothing formula):
  * E_l is the mean, over heads and over the same instruction tokens, of the
    entropy of the token's softmax over the keys up to its position, divided
    by the log of the number of those keys (so 0 <= E_l <= 1);
  * the raw reuse fraction of layer l is u_l = 1 - E_l;
  * "weighted growth smoothing": an exponential average over depth with
    weight 1/2, s_0 = u_0, s_l = s_{l-1} + (u_l - s_{l-1}) / 2;
  * layer l reuses q_l = floor(1000 s_l) per mille of the (filtered) static
    set, in place of the fixed proportions;
  * the signal is the previous step's prompt pass, as for Stage 2.
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


def text_attention_entropy(w_l: dict, h_in: np.ndarray, K: np.ndarray, n_patches: int, n_text: int,
                           n_heads: int, eps: float, base: float) -> np.ndarray:
    """[H]: per head, the sum over the instruction tokens after the image of
    their attention entropy over keys 0..p divided by log(p + 1)."""
    d = h_in.shape[-1]
    dh = d // n_heads
    e = np.zeros(n_heads)
    for p in range(n_patches + 1, n_patches + n_text):
        q = rope_row((w_l["wq"] @ rmsnorm(h_in[p], w_l["attn_norm"], eps)).reshape(n_heads, dh), p, base)
        s = np.einsum("hd,thd->ht", q, K[: p + 1]) / np.sqrt(dh)
        s = s - s.max(axis=1, keepdims=True)
        prob = np.exp(s)
        prob = prob / prob.sum(axis=1, keepdims=True)
        ent = -(prob * np.log(np.where(prob > 0, prob, 1.0))).sum(axis=1)
        e += ent / np.log(p + 1)
    return e


def entropy_permille(ent: np.ndarray, n_instr: int) -> list:
    """Per-layer reuse proportions (per mille) from ent [L][H], the per-head
    sums over the n_instr instruction tokens of normalized entropy."""
    L, H = ent.shape
    q, s = [], 0.0
    for l in range(L):
        u = 1.0 - ent[l].sum() / (H * n_instr)
        s = u if l == 0 else s + (u - s) / 2
        q.append(int(np.floor(1000.0 * min(max(s, 0.0), 1.0))))
    return q


def relevant_patches(score: np.ndarray, k: int) -> np.ndarray:
    """[N] bool: the k highest scores, ties to the lower index."""
    n = len(score)
    order = sorted(range(n), key=lambda i: (-score[i], i))
    out = np.zeros(n, dtype=bool)
    out[order[: max(0, min(k, n))]] = True
    return out
