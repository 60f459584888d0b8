"""ctypes binding of libgvc (include/gvc.h): argument marshalling only.

Functions keep the C names without the `gvc_` prefix.  Device buffers are
passed as integer addresses (e.g. torch's tensor.data_ptr()); every step of
the computation runs in the HIP kernels of libgvc.  Loading fails loudly when
the library has not been built.
"""
import ctypes
import os

# GVC_LIBRARY selects another build of the same library (the host-code
# AddressSanitizer build, libgvc_asan.so); there is no other implementation.
_LIB_PATH = os.environ.get("GVC_LIBRARY") or os.path.join(os.path.dirname(os.path.abspath(__file__)), "libgvc.so")

GVC_OK, GVC_EINVAL, GVC_ESTATE, GVC_ENOMEM, GVC_EDEVICE = 0, 1, 2, 3, 4
REDUCE_MEAN, REDUCE_MIN = 0, 1
(STATE_H, STATE_K, STATE_V, STATE_HEAD_LOGITS, STATE_VALID, STATE_ROWS, STATE_MARGINS, STATE_TV, STATE_ENTROPY,
 STATE_LAYER_Q) = range(10)

(K_DECODE_QKV, K_DECODE_ATTN, K_DECODE_O, K_DECODE_GU, K_DECODE_DOWN, K_DECODE_HEAD, K_PREFILL_QKV,
 K_PREFILL_ATTN, K_PREFILL_O, K_PREFILL_GU, K_PREFILL_DOWN, K_PREFILL_HEAD, K_EMBED, K_NORM, K_SELECT,
 K_DECODE_PASS, K_STAGE2, K_VIT) = range(18)

EXPORTED = ("gvc_sizes", "gvc_init_cache", "gvc_select_static", "gvc_select_static_noalloc", "gvc_step_prefill",
            "gvc_decode_actions",
            "gvc_margin_gate", "gvc_invalidate", "gvc_read_state", "gvc_state_item_bytes", "gvc_profile_begin",
            "gvc_profile_end", "gvc_destroy", "gvc_last_error", "gvc_check_rows")


class GvcError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__("libgvc error %d: %s" % (code, msg))
        self.code = code


class Desc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "batch", "n_layers", "d_model", "n_heads", "ffn", "vocab", "n_bins", "img", "patch", "n_views",
        "n_text", "n_proprio", "n_action_q", "n_decode", "parallel_decode", "norm_full_vocab")] + [
        ("rms_eps", ctypes.c_float), ("rope_theta", ctypes.c_float), ("task_topk", ctypes.c_int32),
        ("entropy_reuse", ctypes.c_int32), ("action_bidir", ctypes.c_int32), ("vit_layers", ctypes.c_int32),
        ("vit_dim", ctypes.c_int32), ("vit_heads", ctypes.c_int32), ("vit_ffn", ctypes.c_int32),
        ("vit_eps", ctypes.c_float)]


class LayerWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("wq", "wk", "wv", "wo", "wg", "wu", "wd", "attn_norm", "ffn_norm")]


VIT_LAYER_FIELDS = ("ln1_g", "ln1_b", "wq", "bq", "wk", "bk", "wv", "bv", "wo", "bo", "ln2_g", "ln2_b", "w1", "b1",
                    "w2", "b2")
VIT_FIELDS = ("patch_w", "patch_b", "pos", "post_g", "post_b", "proj1", "proj1_b", "proj2", "proj2_b")


class VitLayerWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in VIT_LAYER_FIELDS]


class VitWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in VIT_FIELDS] + [("layers", ctypes.POINTER(VitLayerWeights))]


class Weights(ctypes.Structure):
    _fields_ = [("embed", ctypes.c_void_p), ("patch_proj", ctypes.c_void_p), ("lm_head", ctypes.c_void_p),
                ("final_norm", ctypes.c_void_p), ("layers", ctypes.POINTER(LayerWeights)),
                ("vit", ctypes.POINTER(VitWeights))]


_lib = None


def lib():
    """The loaded libgvc; raises if it is missing (no fallback path exists)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise ImportError("libgvc.so is not built; run `python -m paper_2608_10824_amd.build` "
                              "(the HIP library is the only implementation)")
        L = ctypes.CDLL(_LIB_PATH)
        vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        L.gvc_sizes.argtypes = [ctypes.POINTER(Desc), ctypes.POINTER(sz), ctypes.POINTER(sz), ctypes.POINTER(sz)]
        L.gvc_init_cache.argtypes = [ctypes.POINTER(Desc), ctypes.POINTER(Weights), vp, sz, vp, sz, vp, sz, vp,
                                     ctypes.POINTER(vp)]
        L.gvc_select_static.argtypes = [vp, vp, vp, i32, i32, ctypes.POINTER(i32), vp, vp]
        L.gvc_select_static_noalloc.argtypes = [ctypes.POINTER(Desc), vp, vp, i32, i32, ctypes.POINTER(i32), vp, vp,
                                                vp]
        L.gvc_step_prefill.argtypes = [vp, vp, vp, vp, vp]
        L.gvc_decode_actions.argtypes = [vp, vp, vp, vp, vp]
        L.gvc_margin_gate.argtypes = [vp, ctypes.c_float, i32, ctypes.POINTER(ctypes.c_float),
                                      ctypes.POINTER(ctypes.c_uint8), ctypes.POINTER(ctypes.c_int8)]
        L.gvc_invalidate.argtypes = [vp, i32]
        L.gvc_read_state.argtypes = [vp, i32, i32, vp, sz]
        L.gvc_state_item_bytes.argtypes = [vp, i32]
        L.gvc_state_item_bytes.restype = sz
        L.gvc_profile_begin.argtypes = [vp, i32, i32]
        L.gvc_profile_end.argtypes = [vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(i32)]
        L.gvc_destroy.argtypes = [vp]
        L.gvc_check_rows.argtypes = [i32, i32, i32, i32, vp, vp, vp, vp, vp, vp]
        L.gvc_last_error.restype = ctypes.c_char_p
        for n in EXPORTED:
            if n not in ("gvc_state_item_bytes", "gvc_last_error"):
                getattr(L, n).restype = i32
        _lib = L
    return _lib


def _check(code):
    if code != GVC_OK:
        raise GvcError(code, lib().gvc_last_error().decode())


def last_error() -> str:
    return lib().gvc_last_error().decode()


def sizes(desc: Desc):
    w, s, k = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_size_t()
    _check(lib().gvc_sizes(ctypes.byref(desc), ctypes.byref(w), ctypes.byref(s), ctypes.byref(k)))
    return w.value, s.value, k.value


def init_cache(desc: Desc, weights: Weights, weight_arena: int, weight_bytes: int, state: int, state_bytes: int,
               workspace: int, workspace_bytes: int, stream: int) -> int:
    ctx = ctypes.c_void_p()
    _check(lib().gvc_init_cache(ctypes.byref(desc), ctypes.byref(weights), weight_arena, weight_bytes, state,
                                state_bytes, workspace, workspace_bytes, stream, ctypes.byref(ctx)))
    return ctx.value


def check_rows(B: int, L: int, N: int, P: int, mask: int, valid: int, rows: int, counts: int, ep_counts: int,
               ep_offsets: int) -> int:
    """Host-side row-list check (all arguments host addresses, mask may be 0);
    returns the status code (GVC_OK or GVC_EINVAL, message in last_error())."""
    return lib().gvc_check_rows(B, L, N, P, mask or None, valid, rows, counts, ep_counts, ep_offsets)


def select_static(ctx: int, frame_t: int, frame_prev: int, tau_num: int, tau_den: int, reuse_permille,
                  reuse_mask: int, n_static: int):
    q = None
    if reuse_permille is not None:
        q = (ctypes.c_int32 * len(reuse_permille))(*[int(v) for v in reuse_permille])
    _check(lib().gvc_select_static(ctx, frame_t, frame_prev, tau_num, tau_den, q, reuse_mask, n_static))


def select_static_noalloc(desc: Desc, frame_t: int, frame_prev: int, tau_num: int, tau_den: int, reuse_permille,
                          reuse_mask: int, n_static: int, stream: int):
    q = None
    if reuse_permille is not None:
        q = (ctypes.c_int32 * len(reuse_permille))(*[int(v) for v in reuse_permille])
    _check(lib().gvc_select_static_noalloc(ctypes.byref(desc), frame_t, frame_prev, tau_num, tau_den, q, reuse_mask,
                                           n_static, stream))


def step_prefill(ctx: int, frame_t: int, text_ids: int, extra_rows, reuse_mask):
    _check(lib().gvc_step_prefill(ctx, frame_t, text_ids, extra_rows, reuse_mask))


def decode_actions(ctx: int, tokens_out: int, margins_out: int, logits_out=None, forced_tokens=None):
    _check(lib().gvc_decode_actions(ctx, tokens_out, margins_out, logits_out, forced_tokens))


def margin_gate(ctx: int, theta: float, reduce: int, batch: int, force=None):
    m = (ctypes.c_float * batch)()
    f = (ctypes.c_uint8 * batch)()
    fr = None
    if force is not None:
        fr = (ctypes.c_int8 * batch)(*[int(v) for v in force])
    _check(lib().gvc_margin_gate(ctx, theta, reduce, m, f, fr))
    return list(m), [bool(v) for v in f]


def invalidate(ctx: int, b: int = -1):
    _check(lib().gvc_invalidate(ctx, b))


def state_item_bytes(ctx: int, item: int) -> int:
    return lib().gvc_state_item_bytes(ctx, item)


def read_state(ctx: int, item: int, layer: int, dst: int, dst_bytes: int):
    _check(lib().gvc_read_state(ctx, item, layer, dst, dst_bytes))


def profile_begin(ctx: int, cls: int, max_launches: int):
    _check(lib().gvc_profile_begin(ctx, cls, max_launches))


def profile_end(ctx: int):
    """(total milliseconds, launches) of the profiled kernel class."""
    ms, n = ctypes.c_double(), ctypes.c_int32()
    _check(lib().gvc_profile_end(ctx, ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value


def destroy(ctx: int):
    _check(lib().gvc_destroy(ctx))
