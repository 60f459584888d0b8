"""Every-element parity at the 7B shape (32 layers, d 4096, 32 heads, FFN
11008, vocab 32000): the oracle runs Alg. 1 with its own state from the
first frame on, the HIP path runs the same calls through the C ABI, and
after every step every element of the hidden state entering each layer
H[0..L], of every layer's K and V over the prompt, of the head logits and of
every decode pass's logits is compared.

The oracle runs in its batched float64 mode (each projection one library
matrix product over the recomputed rows; pinned on the CPU against its
row-at-a-time form and the Hugging Face forward).  Where several results are
correct the oracle decides and the GPU follows: the GPU decode is fed the
oracle's greedy tokens (forced_tokens) and the GPU gate is forced to the
oracle's decision, so both sides walk the same path; the GPU's own argmax
tokens and its own gate decisions on its own margins are then checked
against the oracle's, each equal unless the oracle's own gap lies inside
the band the measured logit error allows.

Tolerances: 2e-2 of the tensor's largest magnitude for H, K, V and logits
(bf16 operands against the float64 oracle); per slice (a row of H, a (row,
head) of K or V, a position of the logits) 5e-2 of that slice's own largest
magnitude.  Through 32 layers the bf16 roundings of every GEMM operand
and of the K/V cache build up to ~1.5e-2 of the tensor maximum in the last
layers, and a slice whose own maximum is half the tensor's shows twice
that; a wrong row or head is off by its own magnitude, 20x the bound.
"""
import numpy as np
import pytest
import torch

import synth
from oracle.vla import OracleVLA
from oracle.margin import gate_fires
from tests._parity import TOL, TOL_SLICE, rel_err, rel_err_slices, check_tokens, check_margins, state64

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def _pair(cfg, oracle_cfg=None):
    """Oracle (float64 CPU copy of the weights) and GPU session on the same
    seeded weights; the GPU's bf16 canonical copies are dropped after init."""
    from paper_2608_10824_amd.session import Session
    w = synth.model_weights(cfg, device=DEV)
    o = OracleVLA(oracle_cfg or cfg, w, batched=True)
    s = Session(cfg, w, device=DEV)
    torch.cuda.synchronize()
    del w
    torch.cuda.empty_cache()
    return o, s


def _compare_state(s, o, b, label):
    """Every prompt element of H[0..L], K and V of every layer, and the head
    logits of GPU episode b against the oracle's episode 0."""
    from paper_2608_10824_amd import gvc
    cfg = o.cfg
    P, L = cfg.prompt_len, cfg.n_layers
    worst = {"H": 0.0, "K": 0.0, "V": 0.0, "H/row": 0.0, "K/head": 0.0, "V/head": 0.0}
    trend = []
    for l in range(L + 1):
        Hg, Ho = state64(s, gvc.STATE_H, l, b, P), o.H[l, 0]
        trend.append(rel_err(Hg, Ho))
        worst["H"] = max(worst["H"], trend[-1])
        worst["H/row"] = max(worst["H/row"], rel_err_slices(Hg, Ho, 1))
        if l == L:
            break
        for item, name in ((gvc.STATE_K, "K"), (gvc.STATE_V, "V")):
            g = state64(s, item, l, b, P)
            ref = (o.K if name == "K" else o.V)[l, 0, :P]
            worst[name] = max(worst[name], rel_err(g, ref))
            worst[name + "/head"] = max(worst[name + "/head"], rel_err_slices(g, ref, 2))
    head = s.read(gvc.STATE_HEAD_LOGITS).cpu().numpy()[b]
    worst["head"] = rel_err(head, o.head_logits[0])
    worst["head/pos"] = rel_err_slices(head, o.head_logits[0], 1)
    print("%s: %s" % (label, " ".join("%s %.2e" % kv for kv in worst.items())))
    print("%s: H error entering layers 0, 1, 2, 4, 8, 16, %d: %s"
          % (label, L, " ".join("%.1e" % trend[l] for l in (0, 1, 2, 4, 8, 16, L))))
    for k, v in worst.items():
        assert v <= (TOL_SLICE if "/" in k else TOL), (label, k, v)
    return worst


def _decode_lockstep(s, o, b, label):
    """Oracle decode with its own greedy tokens; GPU decode of episode b fed
    the same tokens; logits, tokens (near-tie band) and margins compared.
    Returns the oracle's margins and the GPU's, and the per-position bound."""
    cfg = o.cfg
    tok_o, m_o, z_o = o.decode_actions()
    # every GPU episode is fed the oracle's tokens; only episode b is compared
    forced = torch.from_numpy(np.repeat(tok_o[:1], s.cfg.batch, axis=0).astype(np.int32)).to(DEV)
    tok_g, mg_g, lg_g = s.decode_actions(logits=True, forced_tokens=forced)
    torch.cuda.synchronize()
    lg, tg, mg = lg_g.cpu().numpy()[b], tok_g.cpu().numpy()[b], mg_g.cpu().numpy()[b]
    e, es = rel_err(lg, z_o[0]), rel_err_slices(lg, z_o[0], 1)
    ties = check_tokens(tg, lg, tok_o[0], z_o[0], cfg.bin_lo)
    bound = check_margins(mg, m_o[0], lg, z_o[0], cfg.bin_lo, cfg.norm_full_vocab)
    print("%s decode: logits %.2e (per position %.2e), near-tie tokens %d, margins %s vs %s"
          % (label, e, es, ties, np.round(mg, 4).tolist(), np.round(m_o[0], 4).tolist()))
    assert e <= TOL and es <= TOL_SLICE
    return m_o[0], mg, bound


def _masks(o, frame_t, frame_prev):
    """The oracle's own masks (Stage 1 on its inputs) as the GPU's reuse mask."""
    masks, n_static = o.select_static(frame_t, frame_prev)
    return masks, n_static


def test_c2_full_and_partial_step_every_element():
    """C2 (the benchmark's workload): a full step on frame t-1, then the 50%
    reuse step on frame t (128 static patches, gate kept), each with its
    6-pass decode."""
    cfg = synth.config_c2()
    o, s = _pair(cfg)
    si = synth.step_inputs(cfg, 128)
    fp, ft, ids = si["frame_prev"].numpy(), si["frame_t"].numpy(), si["text_ids"].numpy()
    o.step_prefill(fp, ids)
    s.step_prefill(si["frame_prev"].to(DEV), si["text_ids"].to(DEV))
    _compare_state(s, o, 0, "C2 full step")
    _decode_lockstep(s, o, 0, "C2 full step")
    o.margin_gate(force=[0])
    s.margin_gate(force=[0])
    masks, n_static = _masks(o, ft, fp)
    mask_g, n_g = s.select_static(si["frame_t"].to(DEV), si["frame_prev"].to(DEV))
    assert np.array_equal(mask_g.cpu().numpy().astype(bool), masks) and n_g.cpu().tolist() == [128]
    o.step_prefill(ft, ids, None, masks)
    s.step_prefill(si["frame_t"].to(DEV), si["text_ids"].to(DEV), None, s.mask)
    assert o.recomputed[0].tolist() == [148] * cfg.n_layers
    _compare_state(s, o, 0, "C2 partial step")
    _decode_lockstep(s, o, 0, "C2 partial step")
    s.close()


def test_c5_episode_at_half_reuse_every_element():
    """C5 at 128 static patches per episode (the many-row GEMMs with their
    192-row tiles): one episode of the 16 followed through a full and a
    partial step, every element, and its batched decode."""
    cfg = synth.config_c5()
    b = 5
    o, s = _pair(cfg, cfg.with_(batch=1))
    si = synth.step_inputs(cfg, 128, stream=129)
    one = lambda t: t[b:b + 1].numpy()
    o.step_prefill(one(si["frame_prev"]), one(si["text_ids"]))
    s.step_prefill(si["frame_prev"].to(DEV), si["text_ids"].to(DEV))
    _decode_lockstep(s, o, b, "C5 episode %d full step" % b)
    o.margin_gate(force=[0])
    s.margin_gate(force=[0] * cfg.batch)
    masks, _ = _masks(o, one(si["frame_t"]), one(si["frame_prev"]))
    mask_g, n_g = s.select_static(si["frame_t"].to(DEV), si["frame_prev"].to(DEV))
    assert np.array_equal(mask_g.cpu().numpy()[b:b + 1].astype(bool), masks)
    assert n_g.cpu().tolist() == [128] * cfg.batch
    o.step_prefill(one(si["frame_t"]), one(si["text_ids"]), None, masks)
    s.step_prefill(si["frame_t"].to(DEV), si["text_ids"].to(DEV), None, s.mask)
    _compare_state(s, o, b, "C5 episode %d partial step" % b)
    _decode_lockstep(s, o, b, "C5 episode %d partial step" % b)
    s.close()


@pytest.mark.parametrize("mode", ["causal", "bidir"])
def test_c4_parallel_chunk_every_element(mode):
    """C4: two views, proprio row, 56 parallel-decoded action rows (causal,
    or with the action block: the action rows see each other both ways),
    307 of 512 patches reused; the head's 56 rows, their tokens, margins and
    the minimum gate."""
    cfg = synth.config_c4().with_(action_bidir=mode == "bidir")
    o, s = _pair(cfg)
    si = synth.step_inputs(cfg, 307)
    fp, ft, ids = si["frame_prev"].numpy(), si["frame_t"].numpy(), si["text_ids"].numpy()
    ex = si["extra_rows"].numpy()
    exd = si["extra_rows"].to(DEV)
    o.step_prefill(fp, ids, ex)
    s.step_prefill(si["frame_prev"].to(DEV), si["text_ids"].to(DEV), exd)
    o.decode_actions()
    s.decode_actions()
    o.margin_gate(force=[0])
    s.margin_gate(force=[0])
    masks, _ = _masks(o, ft, fp)
    mask_g, n_g = s.select_static(si["frame_t"].to(DEV), si["frame_prev"].to(DEV))
    assert np.array_equal(mask_g.cpu().numpy().astype(bool), masks) and n_g.cpu().tolist() == [307]
    o.step_prefill(ft, ids, ex, masks)
    s.step_prefill(si["frame_t"].to(DEV), si["text_ids"].to(DEV), exd, s.mask)
    _compare_state(s, o, 0, "C4 %s partial step" % mode)
    m_o, m_g, bound = _decode_lockstep(s, o, 0, "C4 %s partial step" % mode)
    mo, fire_o = o.margin_gate()
    mg, fire_g = s.margin_gate(force=[int(fire_o[0])])
    assert abs(mg[0] - m_g.min()) <= 1e-6 and abs(mo[0] - m_o.min()) <= 1e-12
    assert abs(mg[0] - mo[0]) <= bound.max()
    assert gate_fires(float(mg[0]), cfg.theta) == bool(fire_o[0]) or abs(mo[0] - cfg.theta) < bound.max()
    s.close()


def test_c2v_front_end_full_and_partial_step_every_element():
    """C2 with the ViT-L/14-shaped front end (24 blocks of width 1024): the
    front end runs over every patch at each pass, so a reused token's K/V
    are stale against the oracle's full recompute only through the reuse
    itself; every element after a full and after the 50% reuse step."""
    cfg = synth.config_c2v()
    o, s = _pair(cfg)
    si = synth.step_inputs(cfg, 128)
    fp, ft, ids = si["frame_prev"].numpy(), si["frame_t"].numpy(), si["text_ids"].numpy()
    o.step_prefill(fp, ids)
    s.step_prefill(si["frame_prev"].to(DEV), si["text_ids"].to(DEV))
    _compare_state(s, o, 0, "C2V full step")
    o.decode_actions()
    s.decode_actions()
    o.margin_gate(force=[0])
    s.margin_gate(force=[0])
    masks, _ = _masks(o, ft, fp)
    mask_g, _ = s.select_static(si["frame_t"].to(DEV), si["frame_prev"].to(DEV))
    assert np.array_equal(mask_g.cpu().numpy().astype(bool), masks)
    o.step_prefill(ft, ids, None, masks)
    s.step_prefill(si["frame_t"].to(DEV), si["text_ids"].to(DEV), None, s.mask)
    _compare_state(s, o, 0, "C2V partial step")
    _decode_lockstep(s, o, 0, "C2V partial step")
    s.close()


def test_c2_stage2_stage3_every_element():
    """The benchmark's Stage 2 (k = 120) + Stage 3 (entropy) configuration:
    after the full step, the recorded signals of every layer and head
    against the oracle's own; each side's selection on its own signal
    (decided in fp32 on both sides; equal except for near ties); then the
    partial step on the (equal) masks, every element."""
    from paper_2608_10824_amd import gvc
    from oracle.relevance import relevant_patches
    from tests._parity import fp32_scores, fp32_layer_q, layer_q_near_ties, relevant_near_ties
    cfg = synth.config_c2().with_(task_topk=120, entropy_reuse=True)
    o, s = _pair(cfg)
    si = synth.step_inputs(cfg, 128)
    fp, ft, ids = si["frame_prev"].numpy(), si["frame_t"].numpy(), si["text_ids"].numpy()
    o.step_prefill(fp, ids)
    s.step_prefill(si["frame_prev"].to(DEV), si["text_ids"].to(DEV))
    tv, ent = s.read(gvc.STATE_TV).cpu().numpy(), s.read(gvc.STATE_ENTROPY).cpu().numpy()
    e_tv, e_ent = rel_err(tv, o.tv), rel_err(ent, o.ent)
    e_tv_s = rel_err_slices(tv, o.tv, 3)   # per (layer, head)
    print("signals: attention %.2e (per layer and head %.2e), entropy %.2e" % (e_tv, e_tv_s, e_ent))
    print("attention signal error per layer 0, 1, 2, 4, 8, 16, 31: %s; layer-input error: %s" % (
        " ".join("%.1e" % rel_err(tv[0, l], o.tv[0, l]) for l in (0, 1, 2, 4, 8, 16, 31)),
        " ".join("%.1e" % rel_err(s.read(gvc.STATE_H, l).cpu().numpy()[0], o.H[l, 0]) for l in (0, 1, 2, 4, 8, 16, 31))))
    # The attention signal is a softmax over products of two projections of
    # the layer input, so its relative error is about twice that input's:
    # 3e-3 at layer 0 (exact input) and up to ~2.7e-2 where the 32-layer bf16
    # error of the input is ~1.5e-2; hence twice the state tolerances.
    assert e_tv <= 2 * TOL and e_ent <= TOL and e_tv_s <= 2 * TOL_SLICE
    n_instr = cfg.n_text - 1
    mask_g, n_g = s.select_static(si["frame_t"].to(DEV), si["frame_prev"].to(DEV))
    q_g = s.read(gvc.STATE_LAYER_Q).cpu().numpy()[0].tolist()
    q_o = fp32_layer_q(o.ent[0], n_instr)
    q_ties = layer_q_near_ties(o.ent[0], ent[0], n_instr, q_o, q_g)
    sc_o, sc_g = fp32_scores(o.tv)[0].astype(np.float64), fp32_scores(tv)[0].astype(np.float64)
    r_ties = relevant_near_ties(sc_o, sc_g, 120, relevant_patches(sc_o, 120), relevant_patches(sc_g, 120))
    masks, n_o = o.select_static(ft, fp, scores=sc_o[None], layer_q=[q_o])
    print("proportions %s..., static after Stage 2: %d; near ties: %d layers, %d patches"
          % (q_o[:4], n_o[0], len(q_ties), len(r_ties)))
    if not (q_ties or r_ties):
        assert np.array_equal(mask_g.cpu().numpy().astype(bool), masks) and n_g.cpu().tolist() == n_o.tolist()
    # the oracle's selection decides; the GPU's partial step takes its masks
    o.step_prefill(ft, ids, None, masks)
    s.step_prefill(si["frame_t"].to(DEV), si["text_ids"].to(DEV), None,
                   torch.from_numpy(masks.astype(np.uint8)).to(DEV))
    assert s.read(gvc.STATE_ROWS).cpu().tolist() == o.recomputed[0].tolist()
    _compare_state(s, o, 0, "C2 Stage 2+3 partial step")
    s.close()


# Steps 1..C3_STEPS of the moving-rectangle episode; the gate decisions on
# them include a fired and a kept step.
C3_STEPS = 6


def test_c3_gate_decisions_every_element():
    """C3 (per-layer reuse 80% -> 20%, tau 0.996, theta 0.1) with the gate
    applied: the oracle walks the episode with its own margins and gate;
    every GPU gate decision taken on its own margins must equal the
    oracle's (unless the oracle's margin lies within the error band of the
    threshold), the episode must contain a fired and a kept step, and every
    element of the state is compared after the first partial step and after
    the first step that follows a fired gate."""
    from paper_2608_10824_amd import gvc
    cfg = synth.config_c3()
    o, s = _pair(cfg)
    frames = synth.c3_episode_frames(cfg, n_frames=C3_STEPS + 1)
    fdev = frames.to(DEV)
    ids = synth.text_ids(cfg)
    ids_np, ids_dev = ids.numpy(), ids.to(DEV)
    o.step_prefill(frames[0:1].numpy(), ids_np)
    s.step_prefill(fdev[0:1], ids_dev)
    _, _, bound = _decode_lockstep(s, o, 0, "C3 step 0")
    decisions, compared_after_fire, compared_partial = [], False, False
    for t in range(1, C3_STEPS + 1):
        m_o, fire_o = o.margin_gate()
        m_g, _ = s.margin_gate(force=[int(fire_o[0])])
        own = gate_fires(float(m_g[0]), cfg.theta)
        band = float(np.mean(bound))
        print("C3 step %d gate: oracle m %.5f fire %d, GPU m %.5f own decision %d (band %.1e)"
              % (t, m_o[0], fire_o[0], m_g[0], own, band))
        assert abs(m_g[0] - m_o[0]) <= band
        assert own == bool(fire_o[0]) or abs(m_o[0] - cfg.theta) < band
        decisions.append(bool(fire_o[0]))
        masks, _ = o.select_static(frames[t:t + 1].numpy(), frames[t - 1:t].numpy())
        mask_g, _ = s.select_static(fdev[t:t + 1], fdev[t - 1:t])
        assert np.array_equal(mask_g.cpu().numpy().astype(bool), masks)
        o.step_prefill(frames[t:t + 1].numpy(), ids_np, None, masks)
        s.step_prefill(fdev[t:t + 1], ids_dev, None, s.mask)
        assert s.read(gvc.STATE_ROWS).cpu().tolist() == o.recomputed[0].tolist()
        if (fire_o[0] and not compared_after_fire) or (not fire_o[0] and not compared_partial):
            _compare_state(s, o, 0, "C3 step %d (%s)" % (t, "fired: full" if fire_o[0] else "partial"))
            compared_after_fire |= bool(fire_o[0])
            compared_partial |= not fire_o[0]
        _, _, bound = _decode_lockstep(s, o, 0, "C3 step %d" % t)
    assert any(decisions) and not all(decisions), decisions
    s.close()


def test_decode_pass_is_bit_reproducible():
    """The single-launch decode pass sums the heads' output-projection
    contributions in fixed point, so two decodes of the same prompt state give
    bit-identical logits, tokens and margins (the next step's gate depends on
    them)."""
    from paper_2608_10824_amd import gvc
    from paper_2608_10824_amd.session import Session
    cfg = synth.config_c2()
    w = synth.model_weights(cfg, device=DEV)
    s = Session(cfg, w, device=DEV)
    del w
    si = synth.step_inputs(cfg, 128)
    runs = []
    for _ in range(3):   # a full prompt pass (itself deterministic) before each decode
        s.step_prefill(si["frame_prev"].to(DEV), si["text_ids"].to(DEV))
        tok, mg, lg = s.decode_actions(logits=True)
        torch.cuda.synchronize()
        runs.append((tok.cpu().clone(), mg.cpu().clone(), lg.cpu().clone()))
    for r in runs[1:]:
        assert torch.equal(r[0], runs[0][0]) and torch.equal(r[1], runs[0][1]) and torch.equal(r[2], runs[0][2])
    s.close()
