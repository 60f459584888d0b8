"""Counter-based hash generator (lowbias32) evaluated exactly in int64 torch ops."""
import torch

_M32 = 0xFFFFFFFF
_C1 = 0x7FEB352D
_C2 = 0x846CA68B
_GOLD = 0x9E3779B9


def _mul32(x: torch.Tensor, c: int) -> torch.Tensor:
    """(x * c) mod 2^32 for 0 <= x < 2^32, without int64 overflow."""
    lo = x * (c & 0xFFFF)                      # < 2^48
    hi = ((x * (c >> 16)) & 0xFFFF) << 16      # < 2^32
    return (lo + hi) & _M32


def lowbias32(x: torch.Tensor) -> torch.Tensor:
    """Wellons' lowbias32 mixer on int64 tensors holding values in [0, 2^32)."""
    x = x & _M32
    x = x ^ (x >> 16)
    x = _mul32(x, _C1)
    x = x ^ (x >> 15)
    x = _mul32(x, _C2)
    x = x ^ (x >> 16)
    return x


def _mix_scalar(v: int) -> int:
    return int(lowbias32(torch.tensor([v & _M32], dtype=torch.int64))[0])


def stream_key(seed: int, tensor_id: int) -> int:
    """32-bit key of one (seed, tensor id) stream."""
    return _mix_scalar(seed ^ _mix_scalar((tensor_id + _GOLD) & _M32))


def hash_u32(seed: int, tensor_id: int, start: int, count: int, device="cpu") -> torch.Tensor:
    """32-bit hash values for element indices [start, start+count) of one stream."""
    key = stream_key(seed, tensor_id)
    idx = torch.arange(start, start + count, dtype=torch.int64, device=device)
    return lowbias32(lowbias32(idx ^ key) ^ ((idx >> 32) * _GOLD & _M32))


def uniform_f32(seed: int, tensor_id: int, shape, scale_log2: int, device="cpu",
                offset: float = 0.0, chunk: int = 1 << 26) -> torch.Tensor:
    """Uniform [-2^scale_log2, 2^scale_log2) + offset, exact in fp32."""
    n = 1
    for s in shape:
        n *= int(s)
    out = torch.empty(n, dtype=torch.float32, device=device)
    scale = 2.0 ** (scale_log2 - 23)
    for s0 in range(0, n, chunk):
        c = min(chunk, n - s0)
        h = hash_u32(seed, tensor_id, s0, c, device=device)
        k = (h >> 8) - (1 << 23)
        out[s0:s0 + c] = k.to(torch.float32) * scale + offset
    return out.view(*shape)


def uniform_bf16(seed: int, tensor_id: int, shape, scale_log2: int, device="cpu",
                 offset: float = 0.0, start: int = 0) -> torch.Tensor:
    """uniform_f32 rounded to bf16 (round-to-nearest-even).  `start` is the
    flat element index of the first generated element, so a row slice of a
    larger tensor can be generated on its own."""
    n = 1
    for s in shape:
        n *= int(s)
    out = torch.empty(n, dtype=torch.bfloat16, device=device)
    chunk = 1 << 26
    scale = 2.0 ** (scale_log2 - 23)
    for s0 in range(0, n, chunk):
        c = min(chunk, n - s0)
        h = hash_u32(seed, tensor_id, start + s0, c, device=device)
        k = (h >> 8) - (1 << 23)
        out[s0:s0 + c] = (k.to(torch.float32) * scale + offset).to(torch.bfloat16)
    return out.view(*shape)


def uniform_u8(seed: int, tensor_id: int, shape, device="cpu") -> torch.Tensor:
    """Uniform bytes: the top 8 bits of each hash value."""
    n = 1
    for s in shape:
        n *= int(s)
    h = hash_u32(seed, tensor_id, 0, n, device=device)
    return (h >> 24).to(torch.uint8).view(*shape)
