"""Workload descriptions (shapes, seeds, thresholds) for the five synthetic configs.

Shapes follow the paper's setting: a Llama-2-7B backbone (Sec. V-A), 224x224
frames cut into 14x14 patches so N = 256 (Sec. III-A), and the OFT variant with
8-step action chunks of 7 dimensions decoded in parallel (Sec. V-A).
"""
from dataclasses import dataclass, field, replace
from typing import List, Tuple


@dataclass
class VLAConfig:
    name: str
    batch: int = 1
    n_layers: int = 32
    d_model: int = 4096
    n_heads: int = 32
    ffn: int = 11008
    vocab: int = 32000
    n_bins: int = 256
    img: int = 224
    patch: int = 14
    n_views: int = 1
    n_text: int = 20
    n_proprio: int = 0
    n_action_q: int = 0
    n_decode: int = 7           # D action tokens per control step
    parallel_decode: bool = False   # OFT-style: D head rows from one pass
    reduce_min: bool = False    # gate on min over positions instead of mean
    tau: Tuple[int, int] = (249, 250)   # cosine threshold as num/den
    theta: float = 0.1          # margin threshold
    reuse_permille: List[int] = field(default_factory=list)  # per layer, empty = 1000 everywhere
    rms_eps: float = 1e-5
    rope_theta: float = 10000.0
    seed: int = 2
    wscale_log2: int = -5       # linear / embedding weights U[-2^-5, 2^-5)
    # LM-head rows of the action bins: U[-2^s, 2^s).  -3.625 puts the 7B
    # model's mean action margin near theta = 0.1 on the moving-rectangle
    # episode, so the gate fires on part of the steps (measured: 4/49 steps
    # at s = -3.6, 23/49 at -3.65).
    bin_scale_log2: float = -3.625
    norm_full_vocab: bool = True    # softmax normaliser over the full vocabulary
    task_topk: int = 0          # Stage 2: patches with the most instruction attention leave S (0: off)
    entropy_reuse: bool = False # Stage 3: per-layer proportions from the instruction tokens' attention entropy
    action_bidir: bool = False  # OFT action block: the action-query rows attend to each other both ways
    # vision front end: 0 = linear patch projection; else a ViT of vit_layers
    # pre-norm blocks (no class token) and a two-layer GELU projector to d_model
    vit_layers: int = 0
    vit_dim: int = 1024
    vit_heads: int = 16
    vit_ffn: int = 4096
    vit_eps: float = 1e-6

    @property
    def head_dim(self) -> int:
        return self.d_model // self.n_heads

    @property
    def patches_per_side(self) -> int:
        return self.img // self.patch

    @property
    def n_patches(self) -> int:
        return self.n_views * self.patches_per_side ** 2

    @property
    def patch_dim(self) -> int:
        return self.patch * self.patch * 3

    @property
    def n_extra(self) -> int:
        return self.n_proprio + self.n_action_q

    @property
    def prompt_len(self) -> int:
        return self.n_patches + self.n_text + self.n_extra

    @property
    def bin_lo(self) -> int:
        return self.vocab - self.n_bins

    @property
    def n_head_rows(self) -> int:
        """Rows whose logits the prompt pass produces: the last prompt row, or the
        action-query rows when the action chunk is decoded in parallel."""
        return self.n_action_q if self.parallel_decode else 1

    @property
    def kv_len(self) -> int:
        """Key slots per layer: the prompt plus the D-1 fed-back action tokens."""
        if self.parallel_decode:
            return self.prompt_len
        return self.prompt_len + self.n_decode - 1

    def permille(self) -> List[int]:
        if self.reuse_permille:
            assert len(self.reuse_permille) == self.n_layers
            return list(self.reuse_permille)
        return [1000] * self.n_layers

    def with_(self, **kw) -> "VLAConfig":
        return replace(self, **kw)


def config_c1() -> VLAConfig:
    """Tiny decoder: 2 layers, d=256, 4 heads, FFN 688, vocab 1024 (last 256 are
    action bins), 112x112 frame -> 64 patches, 8 text tokens, 7 action tokens,
    tau = 0.99, theta = 0.1."""
    return VLAConfig(name="C1", n_layers=2, d_model=256, n_heads=4, ffn=688, vocab=1024,
                     img=112, n_text=8, tau=(99, 100), theta=0.1, seed=1,
                     wscale_log2=-4, bin_scale_log2=0)


def config_mid() -> VLAConfig:
    """Mid-size decoder for complete (every element) parity checks: 2 layers,
    d=2048, 16 heads of 128, FFN 5504, vocab 4096 (last 256 are action bins),
    two 112x112 views -> 128 patches, 8 text tokens (136 prompt rows), 7
    action tokens."""
    return VLAConfig(name="MID", n_layers=2, d_model=2048, n_heads=16, ffn=5504, vocab=4096,
                     img=112, n_views=2, n_text=8, tau=(99, 100), theta=0.1, seed=11,
                     wscale_log2=-5, bin_scale_log2=-1)


def config_c4_tiny() -> VLAConfig:
    """Tiny parallel-decoded action chunk for complete parity: the C1 decoder
    with two views (128 patches), 8 text tokens, 1 proprio row and 8
    action-query rows decoded in one pass; gate on the minimum margin."""
    return VLAConfig(name="C4T", n_layers=2, d_model=256, n_heads=4, ffn=688, vocab=1024,
                     img=112, n_views=2, n_text=8, n_proprio=1, n_action_q=8, n_decode=8,
                     parallel_decode=True, reduce_min=True, tau=(99, 100), theta=0.1, seed=6,
                     wscale_log2=-4, bin_scale_log2=0)


def config_c2() -> VLAConfig:
    """Llama-2-7B shape, 256 visual + 20 text tokens, one step at 50% reuse,
    then 7-token autoregressive action decode."""
    return VLAConfig(name="C2", seed=2)


def config_c1v() -> VLAConfig:
    """C1 with a tiny ViT front end: 2 blocks of width 128 (2 heads of 64),
    MLP 512, and the GELU projector to d = 256."""
    return config_c1().with_(name="C1V", vit_layers=2, vit_dim=128, vit_heads=2, vit_ffn=512)


def config_c2v() -> VLAConfig:
    """C2 with a ViT-L/14-shaped front end (24 blocks of width 1024, 16 heads
    of 64, MLP 4096) and the GELU projector 1024 -> 4096 -> 4096."""
    return config_c2().with_(name="C2V", vit_layers=24)


def config_c3() -> VLAConfig:
    """7B shape over a 50-frame moving-rectangle episode; per-layer reuse decays
    linearly 80% -> 20%; tau = 0.996 (the paper's default); theta = 0.1."""
    L = 32
    q = [800 - (600 * l) // (L - 1) for l in range(L)]
    return VLAConfig(name="C3", seed=3, reuse_permille=q, tau=(249, 250), theta=0.1)


def config_c4() -> VLAConfig:
    """7B shape with a parallel-decoded action chunk: two views (512 visual
    tokens), 1 proprio row, 20 text tokens, 56 action-query rows (8 steps x 7
    dims) decoded in one pass; gate on the minimum margin."""
    return VLAConfig(name="C4", seed=4, n_views=2, n_proprio=1, n_action_q=56,
                     n_decode=56, parallel_decode=True, reduce_min=True)


def config_c5() -> VLAConfig:
    """7B shape, 256 visual tokens, 16 independent episodes batched per step."""
    return VLAConfig(name="C5", seed=5, batch=16)


ALL_CONFIGS = {"C1": config_c1, "C2": config_c2, "C3": config_c3, "C4": config_c4, "C5": config_c5}
