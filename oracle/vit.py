"""Vision front end in float64 -- test infrastructure only (tests/, smoke()
and the benchmark's CPU baseline use it; the product path never does).

Sec. III-A: the frame is cut into N = (H/p)(W/p) non-overlapping p x p
patches that are projected into token embeddings before they join the
language tokens.  The paper names no encoder; the evaluated models (Sec. V-A)
put a ViT and a projector in front of the Llama-2 backbone.  Reading taken
here (a ViT without class token, one pass per camera view):
  * patch embedding: the patch's p*p*3 values (H, W, C order) divided by 255,
    times W_patch^T, plus a bias, plus a learned position embedding of the
    patch's raster index within its view;
  * vit_layers pre-norm blocks: h += Attn(LN1(h)), h += MLP(LN2(h)), with
    LayerNorm (gain and bias, eps vit_eps), multi-head attention with biases
    in which every patch of a view attends to every patch of that view, and
    an MLP fc1 -> GELU (tanh form) -> fc2 with biases;
  * a final LayerNorm, then the projector Linear(Dv, d) -> GELU -> Linear(d, d)
    with biases; its output is the visual token's embedding.
Because attention is global, changing one patch changes the embedding of
every patch of that view: a reused token's K/V then really are stale, which
is the error the margin gate guards against (Sec. III-B, Alg. 1).
"""
import numpy as np


def layernorm(x: np.ndarray, g: np.ndarray, b: np.ndarray, eps: float) -> np.ndarray:
    """LayerNorm over the last axis."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * g + b


def gelu_tanh(x: np.ndarray) -> np.ndarray:
    """GELU in its tanh form: x/2 (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3)))."""
    return 0.5 * x * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (x + 0.044715 * x ** 3)))


def view_patches(view: np.ndarray, p: int) -> np.ndarray:
    """[S][p*p*3]: the patches of one [img][img][3] uint8 view in raster
    order, each flattened H, W, C and divided by 255."""
    side = view.shape[0] // p
    out = np.empty((side * side, p * p * 3))
    for r in range(side):
        for c in range(side):
            out[r * side + c] = view[r * p:(r + 1) * p, c * p:(c + 1) * p, :].reshape(-1) / 255.0
    return out


def vit_view(vw: dict, x: np.ndarray, n_heads: int, eps: float) -> np.ndarray:
    """Encoder output [S][Dv] of one view from its patches x [S][p*p*3]."""
    S = x.shape[0]
    h = x @ vw["patch_w"].T + vw["patch_b"] + vw["pos"][:S]
    Dv = h.shape[1]
    dh = Dv // n_heads
    for lw in vw["layers"]:
        a = layernorm(h, lw["ln1_g"], lw["ln1_b"], eps)
        q = (a @ lw["wq"].T + lw["bq"]).reshape(S, n_heads, dh)
        k = (a @ lw["wk"].T + lw["bk"]).reshape(S, n_heads, dh)
        v = (a @ lw["wv"].T + lw["bv"]).reshape(S, n_heads, dh)
        s = np.einsum("qhd,khd->hqk", q, k) / np.sqrt(dh)
        s = s - s.max(axis=2, keepdims=True)
        pr = np.exp(s)
        pr = pr / pr.sum(axis=2, keepdims=True)
        o = np.einsum("hqk,khd->qhd", pr, v).reshape(S, Dv)
        h = h + o @ lw["wo"].T + lw["bo"]
        m = layernorm(h, lw["ln2_g"], lw["ln2_b"], eps)
        h = h + gelu_tanh(m @ lw["w1"].T + lw["b1"]) @ lw["w2"].T + lw["b2"]
    return layernorm(h, vw["post_g"], vw["post_b"], eps)


def project(vw: dict, z: np.ndarray) -> np.ndarray:
    """Projector: [S][Dv] -> [S][d]."""
    return gelu_tanh(z @ vw["proj1"].T + vw["proj1_b"]) @ vw["proj2"].T + vw["proj2_b"]


def visual_embeddings(vw: dict, frame: np.ndarray, p: int, n_heads: int, eps: float) -> np.ndarray:
    """[N][d]: the embeddings of all visual tokens of one frame [views][img][img][3],
    view-major, raster order within a view."""
    return np.concatenate([project(vw, vit_view(vw, view_patches(v, p), n_heads, eps)) for v in frame], axis=0)
