"""Seeded tensors for one workload: weights, frames, text ids and extra rows.

Weight layout is the canonical nn.Linear one, [out_features][in_features],
row-major bf16.  Norm gains are bf16 values 1 + U[-1/16, 1/16).
Frames are uint8 [B][views][H][W][3] (HWC).
"""
import math
import numpy as np
import torch

from .hashgen import uniform_bf16, uniform_f32, uniform_u8, hash_u32
from .configs import VLAConfig


class TensorId:
    """Stream ids of the counter-based generator."""
    EMBED = 1
    PATCH = 2
    LM_HEAD = 3
    LM_HEAD_BINS = 4
    FINAL_NORM = 5
    # per layer: LAYER_BASE + 16*l + kind
    LAYER_BASE = 1000
    WQ, WK, WV, WO, WG, WU, WD, ATTN_NORM, FFN_NORM = range(9)
    # vision front end: VIT_BASE + 32*l + kind per block, VIT_* globals
    VIT_PATCH_W, VIT_PATCH_B, VIT_POS, VIT_POST_G, VIT_POST_B, VIT_PROJ1, VIT_PROJ1_B, VIT_PROJ2, VIT_PROJ2_B = \
        range(20, 29)
    VIT_BASE = 3000
    # inputs
    FRAME = 100000
    CHANGE_ORDER = 110000
    CHANGE_NOISE = 120000
    TEXT = 130000
    EXTRA = 140000
    RECT = 150000


LAYER_KINDS = ("wq", "wk", "wv", "wo", "wg", "wu", "wd", "attn_norm", "ffn_norm")


def _lid(l: int, kind: int) -> int:
    return TensorId.LAYER_BASE + 16 * l + kind


def layer_weights(cfg: VLAConfig, l: int, device="cpu") -> dict:
    """bf16 weights of decoder layer l."""
    d, F, s, a = cfg.d_model, cfg.ffn, cfg.seed, cfg.wscale_log2
    return {
        "wq": uniform_bf16(s, _lid(l, TensorId.WQ), (d, d), a, device),
        "wk": uniform_bf16(s, _lid(l, TensorId.WK), (d, d), a, device),
        "wv": uniform_bf16(s, _lid(l, TensorId.WV), (d, d), a, device),
        "wo": uniform_bf16(s, _lid(l, TensorId.WO), (d, d), a, device),
        "wg": uniform_bf16(s, _lid(l, TensorId.WG), (F, d), a, device),
        "wu": uniform_bf16(s, _lid(l, TensorId.WU), (F, d), a, device),
        "wd": uniform_bf16(s, _lid(l, TensorId.WD), (d, F), a, device),
        "attn_norm": uniform_bf16(s, _lid(l, TensorId.ATTN_NORM), (d,), -4, device, offset=1.0),
        "ffn_norm": uniform_bf16(s, _lid(l, TensorId.FFN_NORM), (d,), -4, device, offset=1.0),
    }


def global_weights(cfg: VLAConfig, device="cpu") -> dict:
    """bf16 embedding table, patch projection, LM head and final-norm gain."""
    d, V, s, a = cfg.d_model, cfg.vocab, cfg.seed, cfg.wscale_log2
    lm = uniform_bf16(s, TensorId.LM_HEAD, (V, d), a, device)
    lm[cfg.bin_lo:] = uniform_bf16(s, TensorId.LM_HEAD_BINS, (cfg.n_bins, d), cfg.bin_scale_log2, device)
    return {
        "embed": uniform_bf16(s, TensorId.EMBED, (V, d), a, device),
        "patch_proj": uniform_bf16(s, TensorId.PATCH, (d, cfg.patch_dim), a, device),
        "lm_head": lm,
        "final_norm": uniform_bf16(s, TensorId.FINAL_NORM, (d,), -4, device, offset=1.0),
    }


VIT_LAYER_KINDS = ("ln1_g", "ln1_b", "wq", "bq", "wk", "bk", "wv", "bv", "wo", "bo", "ln2_g", "ln2_b",
                   "w1", "b1", "w2", "b2")


def vit_weights(cfg: VLAConfig, device="cpu") -> dict:
    """bf16 weights of the vision front end: patch embedding [Dv][p*p*3]
    (input in the H, W, C order of a patch) with bias, a position embedding
    per patch of a view [S][Dv], the blocks, the final LayerNorm and the
    projector [d][Dv], [d][d] with biases.  Matrices U[-2^s, 2^s) with the
    model's s; biases U[-2^-6, 2^-6); LayerNorm gains 1 + U[-1/16, 1/16)."""
    Dv, Fv, d, s, a = cfg.vit_dim, cfg.vit_ffn, cfg.d_model, cfg.seed, cfg.wscale_log2
    S = cfg.patches_per_side ** 2
    T = TensorId
    vid = lambda l, k: T.VIT_BASE + 32 * l + k
    shapes = {"ln1_g": (Dv,), "ln1_b": (Dv,), "wq": (Dv, Dv), "bq": (Dv,), "wk": (Dv, Dv), "bk": (Dv,),
              "wv": (Dv, Dv), "bv": (Dv,), "wo": (Dv, Dv), "bo": (Dv,), "ln2_g": (Dv,), "ln2_b": (Dv,),
              "w1": (Fv, Dv), "b1": (Fv,), "w2": (Dv, Fv), "b2": (Dv,)}

    def gen(tid, name, shape):
        if name.endswith("_g"):
            return uniform_bf16(s, tid, shape, -4, device, offset=1.0)
        if len(shape) == 1 or name.startswith("b") or name.endswith("_b"):
            return uniform_bf16(s, tid, shape, -6, device)
        return uniform_bf16(s, tid, shape, a, device)

    layers = [{k: gen(vid(l, i), k, shapes[k]) for i, k in enumerate(VIT_LAYER_KINDS)}
              for l in range(cfg.vit_layers)]
    return {
        "patch_w": gen(T.VIT_PATCH_W, "patch_w", (Dv, cfg.patch_dim)),
        "patch_b": gen(T.VIT_PATCH_B, "patch_b", (Dv,)),
        "pos": uniform_bf16(s, T.VIT_POS, (S, Dv), a, device),
        "post_g": gen(T.VIT_POST_G, "post_g", (Dv,)),
        "post_b": gen(T.VIT_POST_B, "post_b", (Dv,)),
        "proj1": gen(T.VIT_PROJ1, "proj1", (d, Dv)),
        "proj1_b": gen(T.VIT_PROJ1_B, "proj1_b", (d,)),
        "proj2": gen(T.VIT_PROJ2, "proj2", (d, d)),
        "proj2_b": gen(T.VIT_PROJ2_B, "proj2_b", (d,)),
        "layers": layers,
    }


def model_weights(cfg: VLAConfig, device="cpu") -> dict:
    w = global_weights(cfg, device)
    w["layers"] = [layer_weights(cfg, l, device) for l in range(cfg.n_layers)]
    if cfg.vit_layers > 0:
        w["vit"] = vit_weights(cfg, device)
    return w


# ---------------------------------------------------------------- frames

def random_frame(seed: int, stream: int, img: int) -> torch.Tensor:
    """A [img][img][3] uint8 frame of independent uniform bytes."""
    return uniform_u8(seed, TensorId.FRAME + stream, (img, img, 3))


def changed_patch_order(seed: int, stream: int, n_patches: int) -> np.ndarray:
    """A seeded permutation of patch indices (stable argsort of hash values)."""
    h = hash_u32(seed, TensorId.CHANGE_ORDER + stream, 0, n_patches).numpy()
    return np.argsort(h, kind="stable")


def perturb_patches(frame: torch.Tensor, patch_ids, patch: int, seed: int, stream: int) -> torch.Tensor:
    """Copy of a [H][W][3] frame whose listed patches (raster index) hold fresh
    uniform noise."""
    out = frame.clone()
    side = frame.shape[1] // patch
    noise = uniform_u8(seed, TensorId.CHANGE_NOISE + stream, frame.shape)
    for n in patch_ids:
        r, c = divmod(int(n), side)
        sl = (slice(r * patch, (r + 1) * patch), slice(c * patch, (c + 1) * patch))
        out[sl] = noise[sl]
    return out


def text_ids(cfg: VLAConfig, stream: int = 0) -> torch.Tensor:
    """[B][n_text] int32 ids drawn from the non-action part of the vocabulary."""
    n = cfg.batch * cfg.n_text
    h = hash_u32(cfg.seed, TensorId.TEXT + stream, 0, n)
    return (h % cfg.bin_lo).to(torch.int32).view(cfg.batch, cfg.n_text)


def extra_rows(cfg: VLAConfig, stream: int = 0):
    """[B][n_proprio + n_action_q][d] fp32 input rows (proprio then action
    queries), or None when the config has none."""
    if cfg.n_extra == 0:
        return None
    return uniform_f32(cfg.seed, TensorId.EXTRA + stream,
                       (cfg.batch, cfg.n_extra, cfg.d_model), cfg.wscale_log2)


def step_inputs(cfg: VLAConfig, n_static, stream: int = 0) -> dict:
    """Two consecutive frames per batch element where exactly n_static patches
    (per element; an int or a list of B ints) are unchanged and the rest carry
    fresh uniform noise.  Returns frame_prev, frame_t ([B][views][H][W][3] u8),
    the boolean ground-truth unchanged set [B][N], text ids and extra rows."""
    B, V, N = cfg.batch, cfg.n_views, cfg.n_patches
    if isinstance(n_static, int):
        n_static = [n_static] * B
    per_view = N // V
    prev = torch.empty(B, V, cfg.img, cfg.img, 3, dtype=torch.uint8)
    cur = torch.empty_like(prev)
    unchanged = np.ones((B, N), dtype=bool)
    for b in range(B):
        order = changed_patch_order(cfg.seed, 1000 * stream + b, N)
        changed = order[: N - n_static[b]]
        unchanged[b, changed] = False
        for v in range(V):
            base = random_frame(cfg.seed, 1000 * stream + 16 * b + v, cfg.img)
            ids = [n - v * per_view for n in changed if v * per_view <= n < (v + 1) * per_view]
            prev[b, v] = base
            cur[b, v] = perturb_patches(base, ids, cfg.patch, cfg.seed, 1000 * stream + 16 * b + v)
    return {
        "frame_prev": prev,
        "frame_t": cur,
        "unchanged": unchanged,
        "text_ids": text_ids(cfg, stream),
        "extra_rows": extra_rows(cfg, stream),
    }


def reuse_schedule(cfg: VLAConfig):
    return cfg.permille()


def _changed_patches(a: np.ndarray, b: np.ndarray, patch: int) -> int:
    side = a.shape[0] // patch
    d = (a != b).any(axis=2).reshape(side, patch, side, patch).any(axis=(1, 3))
    return int(d.sum())


def c3_episode_frames(cfg: VLAConfig, n_frames: int = 50, lo: float = 0.05, hi: float = 0.40):
    """Frames [n_frames][1][H][W][3] u8 of a moving solid rectangle over a fixed
    uniform-noise background.  Each frame's rectangle size and velocity are
    redrawn (deterministically, from the hash stream) until the share of
    patches whose pixels differ from the previous frame lies in [lo, hi]."""
    img, p = cfg.img, cfg.patch
    N = (img // p) ** 2
    bg = random_frame(cfg.seed, 7777, img).numpy()
    color = (hash_u32(cfg.seed, TensorId.RECT, 0, 3).numpy() >> 24).astype(np.uint8)
    draws = hash_u32(cfg.seed, TensorId.RECT + 1, 0, 1 << 16).numpy()
    di = 0

    def draw(lo_v, hi_v):
        nonlocal di
        v = lo_v + int(draws[di % draws.size]) % (hi_v - lo_v + 1)
        di += 1
        return v

    def render(x, y, w, h):
        f = bg.copy()
        f[y:y + h, x:x + w] = color
        return f

    w, h = 60, 50
    x, y = 20, 30
    frames = [render(x, y, w, h)]
    for t in range(1, n_frames):
        for _attempt in range(10000):
            nw, nh = draw(20, 120), draw(20, 120)
            vx, vy = draw(-30, 30), draw(-30, 30)
            nx = min(max(x + vx, 0), img - nw)
            ny = min(max(y + vy, 0), img - nh)
            f = render(nx, ny, nw, nh)
            frac = _changed_patches(frames[-1], f, p) / N
            if lo <= frac <= hi:
                break
        else:  # pragma: no cover - the draw stream always finds one in practice
            raise RuntimeError("no rectangle move within the changed-patch band")
        frames.append(f)
        x, y, w, h = nx, ny, nw, nh
    return torch.from_numpy(np.stack(frames)[:, None])
