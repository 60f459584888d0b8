"""Pins of the vision front end in the oracle (Sec. III-A patch embedding;
reading: a class-token-free ViT and a GELU projector) -- CPU only: the
encoder against Hugging Face's SigLIP vision tower given the same weights,
GELU and LayerNorm closed forms, and the global-attention property."""
import numpy as np
import torch

import synth
from oracle.vit import layernorm, gelu_tanh, view_patches, vit_view, project, visual_embeddings
from oracle.vla import OracleVLA, convert_weights


def _hf_siglip(cfg, vw):
    from transformers import SiglipVisionConfig, SiglipVisionModel
    hc = SiglipVisionConfig(hidden_size=cfg.vit_dim, intermediate_size=cfg.vit_ffn,
                            num_hidden_layers=cfg.vit_layers, num_attention_heads=cfg.vit_heads, num_channels=3,
                            image_size=cfg.img, patch_size=cfg.patch, hidden_act="gelu_pytorch_tanh",
                            layer_norm_eps=cfg.vit_eps, vision_use_head=False)
    hc._attn_implementation = "eager"
    m = SiglipVisionModel(hc).double().eval()
    f = lambda t: torch.nn.Parameter(torch.from_numpy(np.ascontiguousarray(t)).double())
    p, Dv = cfg.patch, cfg.vit_dim
    vm = getattr(m, "vision_model", m)
    emb = vm.embeddings
    # the patch weights are stored H, W, C per output row; the convolution wants C, H, W
    emb.patch_embedding.weight = f(vw["patch_w"].reshape(Dv, p, p, 3).transpose(0, 3, 1, 2))
    emb.patch_embedding.bias = f(vw["patch_b"])
    emb.position_embedding.weight = f(vw["pos"])
    for lw, L in zip(vw["layers"], vm.encoder.layers):
        L.layer_norm1.weight, L.layer_norm1.bias = f(lw["ln1_g"]), f(lw["ln1_b"])
        L.layer_norm2.weight, L.layer_norm2.bias = f(lw["ln2_g"]), f(lw["ln2_b"])
        a = L.self_attn
        a.q_proj.weight, a.q_proj.bias = f(lw["wq"]), f(lw["bq"])
        a.k_proj.weight, a.k_proj.bias = f(lw["wk"]), f(lw["bk"])
        a.v_proj.weight, a.v_proj.bias = f(lw["wv"]), f(lw["bv"])
        a.out_proj.weight, a.out_proj.bias = f(lw["wo"]), f(lw["bo"])
        L.mlp.fc1.weight, L.mlp.fc1.bias = f(lw["w1"]), f(lw["b1"])
        L.mlp.fc2.weight, L.mlp.fc2.bias = f(lw["w2"]), f(lw["b2"])
    vm.post_layernorm.weight = f(vw["post_g"])
    vm.post_layernorm.bias = f(vw["post_b"])
    return m


def test_encoder_matches_hf_siglip_vision_tower():
    cfg = synth.config_c1v().with_(n_views=2)
    w = synth.model_weights(cfg)
    vw = convert_weights(w)["vit"]
    frame = synth.step_inputs(cfg, 30)["frame_t"].numpy()[0]       # [views][img][img][3]
    m = _hf_siglip(cfg, vw)
    with torch.no_grad():
        px = torch.from_numpy(frame.transpose(0, 3, 1, 2) / 255.0)  # [views][3][img][img]
        ref = m(pixel_values=px).last_hidden_state.numpy()
    # HF's eager attention takes its softmax in fp32, hence 1e-6 (a dropped
    # bias, a transposed patch or a wrong scale is > 1e-3)
    for v in range(cfg.n_views):
        mine = vit_view(vw, view_patches(frame[v], cfg.patch), cfg.vit_heads, cfg.vit_eps)
        assert np.abs(mine - ref[v]).max() / np.abs(ref[v]).max() < 1e-6


def test_gelu_and_layernorm_closed_forms():
    x = np.linspace(-6, 6, 101)
    ref = torch.nn.functional.gelu(torch.from_numpy(x), approximate="tanh").numpy()
    assert np.allclose(gelu_tanh(x), ref, atol=1e-15)
    assert gelu_tanh(np.array([0.0]))[0] == 0.0
    assert abs(gelu_tanh(np.array([20.0]))[0] - 20.0) < 1e-12 and abs(gelu_tanh(np.array([-20.0]))[0]) < 1e-12
    g, b = np.array([2.0, 3.0]), np.array([0.5, -1.0])
    # [a, -a] normalises to [1, -1] (up to eps); a constant row to the bias
    assert np.allclose(layernorm(np.array([3.0, -3.0]), g, b, 0.0), [2.5, -4.0])
    assert np.allclose(layernorm(np.array([7.0, 7.0]), g, b, 1e-6), b)
    y = layernorm(np.random.default_rng(0).standard_normal((5, 64)), np.ones(64), np.zeros(64), 0.0)
    assert np.allclose(y.mean(axis=1), 0, atol=1e-12) and np.allclose((y ** 2).mean(axis=1), 1, atol=1e-12)


def test_one_patch_moves_every_embedding_of_its_view_only():
    """Global attention: a change to one patch changes every visual
    embedding of that view; other views are untouched.  With no blocks the
    change stays in its own patch."""
    for layers in (2, 0):
        cfg = synth.config_c1v().with_(n_views=2, vit_layers=layers)
        vw = convert_weights({"vit": synth.vit_weights(cfg)})["vit"]
        frame = synth.step_inputs(cfg, 30)["frame_t"].numpy()[0].copy()
        e0 = visual_embeddings(vw, frame, cfg.patch, cfg.vit_heads, cfg.vit_eps)
        frame[0, :cfg.patch, :cfg.patch, :] = 255 - frame[0, :cfg.patch, :cfg.patch, :]
        e1 = visual_embeddings(vw, frame, cfg.patch, cfg.vit_heads, cfg.vit_eps)
        S = cfg.patches_per_side ** 2
        moved = np.abs(e1 - e0).max(axis=1)
        assert moved[0] > 1e-3 and np.all(moved[S:] == 0.0)
        if layers:
            assert np.all(moved[1:S] > 1e-9)
        else:
            assert np.all(moved[1:S] == 0.0)


def test_prompt_pass_uses_the_front_end():
    cfg = synth.config_c1v()
    w = synth.model_weights(cfg)
    si = synth.step_inputs(cfg, 45)
    o = OracleVLA(cfg, w)
    o.step_prefill(si["frame_t"].numpy(), si["text_ids"].numpy())
    vw = o.w["vit"]
    vis = visual_embeddings(vw, si["frame_t"].numpy()[0], cfg.patch, cfg.vit_heads, cfg.vit_eps)
    N = cfg.n_patches
    assert np.array_equal(o.H[0, 0, 1:N + 1], vis)
    assert vis.shape == (N, cfg.d_model)
    # the projector is the last step: its input is the encoder output; it
    # equals torch's Linear -> GELU(tanh) -> Linear with the same weights
    z = vit_view(vw, view_patches(si["frame_t"].numpy()[0, 0], cfg.patch), cfg.vit_heads, cfg.vit_eps)
    assert np.array_equal(project(vw, z), vis[: cfg.patches_per_side ** 2])
    mlp = torch.nn.Sequential(torch.nn.Linear(cfg.vit_dim, cfg.d_model), torch.nn.GELU(approximate="tanh"),
                              torch.nn.Linear(cfg.d_model, cfg.d_model)).double()
    with torch.no_grad():
        mlp[0].weight.copy_(torch.from_numpy(vw["proj1"])); mlp[0].bias.copy_(torch.from_numpy(vw["proj1_b"]))
        mlp[2].weight.copy_(torch.from_numpy(vw["proj2"])); mlp[2].bias.copy_(torch.from_numpy(vw["proj2_b"]))
        ref = mlp(torch.from_numpy(z)).numpy()
    assert np.abs(project(vw, z) - ref).max() < 1e-12
