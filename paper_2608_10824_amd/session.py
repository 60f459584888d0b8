"""A control-step session over libgvc with PyTorch as the device allocator.

PyTorch provides device memory and the stream; every computation is a call
into libgvc.  The session owns the arenas the library asks for, the output
buffers of each call and the context handle.
"""
import ctypes

import torch

from . import gvc


def desc_from(cfg) -> gvc.Desc:
    """C descriptor from a workload description with the synth.VLAConfig fields."""
    return gvc.Desc(batch=cfg.batch, n_layers=cfg.n_layers, d_model=cfg.d_model, n_heads=cfg.n_heads,
                    ffn=cfg.ffn, vocab=cfg.vocab, n_bins=cfg.n_bins, img=cfg.img, patch=cfg.patch,
                    n_views=cfg.n_views, n_text=cfg.n_text, n_proprio=cfg.n_proprio, n_action_q=cfg.n_action_q,
                    n_decode=cfg.n_decode, parallel_decode=int(cfg.parallel_decode),
                    norm_full_vocab=int(cfg.norm_full_vocab), rms_eps=cfg.rms_eps, rope_theta=cfg.rope_theta,
                    task_topk=cfg.task_topk, entropy_reuse=int(cfg.entropy_reuse),
                    action_bidir=int(cfg.action_bidir), vit_layers=cfg.vit_layers, vit_dim=cfg.vit_dim,
                    vit_heads=cfg.vit_heads, vit_ffn=cfg.vit_ffn, vit_eps=cfg.vit_eps)


def _ptr(t):
    return None if t is None else t.data_ptr()


def _bf16_ptr(t):
    assert t.is_cuda and t.dtype == torch.bfloat16 and t.is_contiguous()
    return t.data_ptr()


class Session:
    """Holds one libgvc context.  `weights` is a dict of CUDA bf16 tensors in
    the canonical layout (embed, patch_proj, lm_head, final_norm, layers[l]
    with wq..wd, attn_norm, ffn_norm); they may be dropped after init."""

    def __init__(self, cfg, weights, device="cuda"):
        if not torch.cuda.is_available():
            raise RuntimeError("libgvc needs a GPU")
        self.cfg = cfg
        self.device = torch.device(device)
        self.desc = desc_from(cfg)
        wb, sb, kb = gvc.sizes(self.desc)
        self.weight_arena = torch.empty(wb, dtype=torch.uint8, device=self.device)
        self.state = torch.empty(sb, dtype=torch.uint8, device=self.device)
        self.workspace = torch.empty(kb, dtype=torch.uint8, device=self.device)
        layers = (gvc.LayerWeights * cfg.n_layers)()
        for l, lw in enumerate(weights["layers"]):
            for k in ("wq", "wk", "wv", "wo", "wg", "wu", "wd", "attn_norm", "ffn_norm"):
                t = lw[k]
                assert t.is_cuda and t.dtype == torch.bfloat16 and t.is_contiguous()
                setattr(layers[l], k, t.data_ptr())
        w = gvc.Weights(embed=weights["embed"].data_ptr(), patch_proj=weights["patch_proj"].data_ptr(),
                        lm_head=weights["lm_head"].data_ptr(), final_norm=weights["final_norm"].data_ptr(),
                        layers=layers)
        if cfg.vit_layers > 0:
            vw = weights["vit"]
            vl = (gvc.VitLayerWeights * cfg.vit_layers)()
            for l, lw in enumerate(vw["layers"]):
                for k in gvc.VIT_LAYER_FIELDS:
                    setattr(vl[l], k, _bf16_ptr(lw[k]))
            self._vit = gvc.VitWeights(layers=vl, **{k: _bf16_ptr(vw[k]) for k in gvc.VIT_FIELDS})
            self._vit_layers = vl
            w.vit = ctypes.pointer(self._vit)
        self.stream = torch.cuda.current_stream(self.device)
        self.ctx = gvc.init_cache(self.desc, w, self.weight_arena.data_ptr(), wb, self.state.data_ptr(), sb,
                                  self.workspace.data_ptr(), kb, self.stream.cuda_stream)
        B, L, N, D = cfg.batch, cfg.n_layers, cfg.n_patches, cfg.n_decode
        self.mask = torch.zeros(B, L, N, dtype=torch.uint8, device=self.device)
        self.n_static = torch.zeros(B, dtype=torch.int32, device=self.device)
        self.tokens = torch.zeros(B, D, dtype=torch.int32, device=self.device)
        self.margins = torch.zeros(B, D, dtype=torch.float32, device=self.device)

    def close(self):
        if self.ctx:
            gvc.destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ---- the five calls of a control step
    def select_static(self, frame_t, frame_prev, tau=None, permille=None):
        tau = tau or self.cfg.tau
        permille = self.cfg.permille() if permille is None else permille
        gvc.select_static(self.ctx, frame_t.data_ptr(), frame_prev.data_ptr(), tau[0], tau[1], permille,
                          self.mask.data_ptr(), self.n_static.data_ptr())
        return self.mask, self.n_static

    def step_prefill(self, frame_t, text_ids, extra_rows=None, mask=None):
        gvc.step_prefill(self.ctx, frame_t.data_ptr(), text_ids.data_ptr(), _ptr(extra_rows), _ptr(mask))

    def decode_actions(self, logits=False, forced_tokens=None):
        out = None
        if logits:
            out = torch.empty(self.cfg.batch, self.cfg.n_decode, self.cfg.vocab, dtype=torch.float32,
                              device=self.device)
        gvc.decode_actions(self.ctx, self.tokens.data_ptr(), self.margins.data_ptr(), _ptr(out),
                           _ptr(forced_tokens))
        return self.tokens, self.margins, out

    def margin_gate(self, theta=None, use_min=None, force=None):
        theta = self.cfg.theta if theta is None else theta
        use_min = self.cfg.reduce_min if use_min is None else use_min
        return gvc.margin_gate(self.ctx, float(theta), gvc.REDUCE_MIN if use_min else gvc.REDUCE_MEAN,
                               self.cfg.batch, force)

    def invalidate(self, b=-1):
        gvc.invalidate(self.ctx, b)

    # ---- state inspection
    def read(self, item, layer=0):
        n = gvc.state_item_bytes(self.ctx, item)
        buf = torch.empty(n, dtype=torch.uint8, device=self.device)
        gvc.read_state(self.ctx, item, layer, buf.data_ptr(), n)
        cfg = self.cfg
        B, P, d, H, dh = cfg.batch, cfg.prompt_len, cfg.d_model, cfg.n_heads, cfg.head_dim
        kv_pad = (cfg.kv_len + 31) // 32 * 32
        if item == gvc.STATE_H:
            return buf.view(torch.float32).view(B, P, d)
        if item == gvc.STATE_K:
            return buf.view(torch.bfloat16).view(B, H, kv_pad, dh)
        if item == gvc.STATE_V:
            return buf.view(torch.bfloat16).view(B, H, dh, kv_pad)
        if item == gvc.STATE_HEAD_LOGITS:
            return buf.view(torch.float32).view(B, cfg.n_head_rows, cfg.vocab)
        if item in (gvc.STATE_VALID, gvc.STATE_ROWS):
            return buf.view(torch.int32)
        if item == gvc.STATE_MARGINS:
            return buf.view(torch.float32).view(B, cfg.n_decode)
        if item == gvc.STATE_TV:
            return buf.view(torch.float32).view(B, cfg.n_layers, H, cfg.n_patches)
        if item == gvc.STATE_ENTROPY:
            return buf.view(torch.float32).view(B, cfg.n_layers, H)
        if item == gvc.STATE_LAYER_Q:
            return buf.view(torch.int32).view(B, cfg.n_layers)
        return buf
