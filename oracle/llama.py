"""Llama-2 decoder block in float64, one token row at a time.

Sec. V-A: both evaluated models use a Llama-2 backbone.  The paper gives no
block details, so the standard Llama-2 block is taken:
  pre-norm RMSNorm, x / sqrt(mean(x^2) + eps) * g, eps = 1e-5;
  multi-head attention (no grouped KV), scale 1/sqrt(d_h), causal;
  rotary position embedding with base 10000, rotating dimension i together
  with i + d_h/2 by the angle pos * base^(-2i/d_h);
  SwiGLU feed-forward W_d (silu(W_g x) * (W_u x)); no biases.
Sec. III-B, Stage 1 / Alg. 1: a partial pass recomputes only some rows and
attends over keys of which some are fresh and some are carried over; so the
layer here takes an explicit row set and a persistent K/V store.
"""
import numpy as np


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm of one row vector."""
    return x / np.sqrt(np.mean(x * x) + eps) * g


def rope_row(x: np.ndarray, pos: int, base: float) -> np.ndarray:
    """Rotary embedding of one [H][d_h] row at absolute position pos."""
    H, dh = x.shape
    half = dh // 2
    i = np.arange(half, dtype=np.float64)
    ang = pos * base ** (-2.0 * i / dh)
    c, s = np.cos(ang), np.sin(ang)
    a, b = x[:, :half], x[:, half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=1)


def attend_row(q: np.ndarray, last: int, K: np.ndarray, V: np.ndarray) -> np.ndarray:
    """Attention of one query row [H][d_h] over the key slots 0..last of K, V
    ([T][H][d_h]); causal when last is the row's own position."""
    H, dh = q.shape
    k = K[: last + 1]                    # [last+1][H][dh]
    v = V[: last + 1]
    s = np.einsum("hd,thd->ht", q, k) / np.sqrt(dh)
    s = s - s.max(axis=1, keepdims=True)
    p = np.exp(s)
    p = p / p.sum(axis=1, keepdims=True)
    return np.einsum("ht,thd->hd", p, v)


def silu(x):
    return x / (1.0 + np.exp(-x))


def layer_rows(w: dict, h_in: np.ndarray, rows, pos, K: np.ndarray, V: np.ndarray,
               n_heads: int, eps: float, base: float, key_last=None) -> np.ndarray:
    """One decoder layer over the row set `rows` (indices into h_in) at the
    absolute positions `pos`, writing fresh K/V into the slots `pos` of the
    persistent K, V arrays and attending over all slots up to each row's
    position (or up to key_last[i] when given: a bidirectional block).
    Returns the layer outputs [len(rows)][d]."""
    d = h_in.shape[-1]
    dh = d // n_heads
    qs = []
    # K/V of every recomputed row are written before any row attends, so a
    # row sees the fresh values of all recomputed rows before it.
    for r, p in zip(rows, pos):
        xn = rmsnorm(h_in[r], w["attn_norm"], eps)
        q = (w["wq"] @ xn).reshape(n_heads, dh)
        k = (w["wk"] @ xn).reshape(n_heads, dh)
        v = (w["wv"] @ xn).reshape(n_heads, dh)
        qs.append(rope_row(q, p, base))
        K[p] = rope_row(k, p, base)
        V[p] = v
    out = np.empty((len(rows), d))
    for i, (r, p) in enumerate(zip(rows, pos)):
        o = attend_row(qs[i], p if key_last is None else key_last[i], K, V).reshape(d)
        res = h_in[r] + w["wo"] @ o
        rn = rmsnorm(res, w["ffn_norm"], eps)
        out[i] = res + w["wd"] @ (silu(w["wg"] @ rn) * (w["wu"] @ rn))
    return out


def head_row(h: np.ndarray, g: np.ndarray, w_lm: np.ndarray, eps: float) -> np.ndarray:
    """Final RMSNorm then the LM head: logits of one row."""
    return w_lm @ rmsnorm(h, g, eps)


def attend_rows(Q: np.ndarray, last, K: np.ndarray, V: np.ndarray) -> np.ndarray:
    """attend_row for several query rows at once: Q [M][H][d_h], row i sees the
    key slots 0..last[i]; the scores and the weighted sum are taken as batched
    matrix products over the heads (library matmuls as the steps of the same
    formula), keys past a row's last slot masked out."""
    M, H, dh = Q.shape
    last = np.asarray(last)
    T = int(last.max()) + 1
    Qh = Q.transpose(1, 0, 2)                        # [H][M][dh]
    Kh = K[:T].transpose(1, 2, 0)                    # [H][dh][T]
    Vh = V[:T].transpose(1, 0, 2)                    # [H][T][dh]
    s = np.matmul(Qh, Kh) / np.sqrt(dh)              # [H][M][T]
    s = np.where(np.arange(T)[None, None, :] > last[None, :, None], -np.inf, s)
    s = s - s.max(axis=2, keepdims=True)
    p = np.exp(s)
    p = p / p.sum(axis=2, keepdims=True)
    return np.matmul(p, Vh).transpose(1, 0, 2)       # [M][H][dh]


def layer_rows_batched(w: dict, h_in: np.ndarray, rows, pos, K: np.ndarray, V: np.ndarray,
                       n_heads: int, eps: float, base: float, key_last=None) -> np.ndarray:
    """layer_rows with every projection taken as one matrix product over the
    whole row set and the attention as attend_rows; the normalisation and the
    rotation stay per row.  Same block, same arguments and effects (fresh K/V
    written into the slots `pos` before any row attends); the values differ
    from layer_rows only in the summation order inside the library products.
    For the 7B shape, where the row-at-a-time form is too slow."""
    d = h_in.shape[-1]
    dh = d // n_heads
    rows, pos = list(rows), list(pos)
    X = h_in[rows]
    Xn = np.stack([rmsnorm(x, w["attn_norm"], eps) for x in X])
    Qp, Kp, Vp = Xn @ w["wq"].T, Xn @ w["wk"].T, Xn @ w["wv"].T
    Q = np.empty((len(rows), n_heads, dh))
    for i, p in enumerate(pos):
        Q[i] = rope_row(Qp[i].reshape(n_heads, dh), p, base)
        K[p] = rope_row(Kp[i].reshape(n_heads, dh), p, base)
        V[p] = Vp[i].reshape(n_heads, dh)
    last = pos if key_last is None else list(key_last)
    O = attend_rows(Q, last, K, V).reshape(len(rows), d)
    R = X + O @ w["wo"].T
    Rn = np.stack([rmsnorm(r, w["ffn_norm"], eps) for r in R])
    return R + (silu(Rn @ w["wg"].T) * (Rn @ w["wu"].T)) @ w["wd"].T
