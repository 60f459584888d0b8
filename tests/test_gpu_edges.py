"""Edge cases of the HIP path, every element checked against the oracle (or
bit-exactly against another GPU run where the method fixes the result):
parallel-decoded action chunk, identical frames, no static patch, all-zero
frames, a single action token, per-episode static counts, the largest
frame the library accepts.  Every call goes through the C ABI."""
import numpy as np
import pytest
import torch

import synth
from oracle.vla import OracleVLA
from oracle import patches as op
from oracle.margin import gate_fires
from tests._parity import TOL, rel_err, to_dev, check_tokens, check_margins

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def _session(cfg, w):
    from paper_2608_10824_amd.session import Session
    return Session(cfg, to_dev(w, DEV), device=DEV)


def _state(s, cfg):
    from paper_2608_10824_amd import gvc
    H = [s.read(gvc.STATE_H, l).cpu().numpy() for l in range(cfg.n_layers + 1)]
    K = [s.read(gvc.STATE_K, l).float().cpu().numpy() for l in range(cfg.n_layers)]
    V = [s.read(gvc.STATE_V, l).float().cpu().numpy() for l in range(cfg.n_layers)]
    return H, K, V, s.read(gvc.STATE_HEAD_LOGITS).cpu().numpy()


def _chunk_cfg(name):
    if name == "C4T":
        return synth.config_c4_tiny()
    if name == "C4T-bidir":
        return synth.config_c4_tiny().with_(action_bidir=True)
    # heads of 128 and a 56-row block that starts inside a 16-row tile
    return synth.config_mid().with_(n_proprio=1, n_action_q=56, n_decode=56, parallel_decode=True,
                                    reduce_min=True, action_bidir=True)


@pytest.mark.parametrize("name", ["C4T", "C4T-bidir", "MID-bidir", "MID-bidir-big"])
def test_parallel_action_chunk_complete_parity(name, monkeypatch):
    """Two views, a proprio row and the action-query rows decoded in one pass
    (the OFT variant, Sec. V-A), causal or with the action rows attending to
    each other both ways: state, every position's logits, tokens, margins
    and the minimum-margin gate.  MID-bidir-big runs the many-row kernels
    (projections, 16-row norm, grouped attention) on the same case."""
    from paper_2608_10824_amd import gvc
    cfg = _chunk_cfg(name)
    w = synth.model_weights(cfg)
    si = synth.step_inputs(cfg, 90)
    if name.endswith("-big"):
        monkeypatch.setenv("GVC_GEMM", "big")
    s = _session(cfg, w)
    o = OracleVLA(cfg, w)
    fp, ft, ids, ex = si["frame_prev"], si["frame_t"], si["text_ids"], si["extra_rows"]
    s.step_prefill(fp.to(DEV), ids.to(DEV), ex.to(DEV))
    o.step_prefill(fp.numpy(), ids.numpy(), ex.numpy())
    s.decode_actions()
    o.decode_actions()
    s.margin_gate(force=[0])
    o.margin_gate(force=[0])
    mask, _ = s.select_static(ft.to(DEV), fp.to(DEV))
    mo, _ = o.select_static(ft.numpy(), fp.numpy())
    assert np.array_equal(mask.cpu().numpy().astype(bool), mo)
    s.step_prefill(ft.to(DEV), ids.to(DEV), ex.to(DEV), mask)
    o.step_prefill(ft.numpy(), ids.numpy(), ex.numpy(), mo)
    H, K, V, z = _state(s, cfg)
    P = cfg.prompt_len
    for l in range(cfg.n_layers + 1):
        assert rel_err(H[l], o.H[l]) <= TOL
    for l in range(cfg.n_layers):
        assert rel_err(K[l][:, :, :P], o.K[l].transpose(0, 2, 1, 3)[:, :, :P]) <= TOL
    assert rel_err(z, o.head_logits) <= TOL
    if cfg.action_bidir:
        # the block is really applied: the action rows sit much closer to the
        # oracle with the block than to the oracle without it
        oc = OracleVLA(cfg.with_(action_bidir=False), w)
        oc.step_prefill(fp.numpy(), ids.numpy(), ex.numpy())
        oc.step_prefill(ft.numpy(), ids.numpy(), ex.numpy(), mo)
        a0, L = P - cfg.n_action_q, cfg.n_layers
        e_block = rel_err(H[L][:, a0:], o.H[L][:, a0:])
        e_causal = rel_err(o.H[L][:, a0:], oc.H[L][:, a0:])
        print("%s action rows: err %.2e, causal distance %.2e" % (name, e_block, e_causal))
        assert e_block < e_causal / 4
    tok, mg, lg = s.decode_actions(logits=True)
    tok_o, mg_o, lg_o = o.decode_actions()
    torch.cuda.synchronize()
    assert rel_err(lg.cpu().numpy(), lg_o) <= TOL
    check_tokens(tok.cpu().numpy(), lg.cpu().numpy(), tok_o, lg_o, cfg.bin_lo)
    check_margins(mg.cpu().numpy(), mg_o, lg.cpu().numpy(), lg_o, cfg.bin_lo)
    m, fire = s.margin_gate()
    assert abs(m[0] - float(mg.cpu().numpy()[0].min())) <= 1e-6
    assert fire[0] == gate_fires(m[0], cfg.theta)
    s.close()


@pytest.mark.parametrize("gemm", ["small", "big"])
def test_identical_frame_full_reuse_is_bit_identical(gemm):
    """After a full step, the same frame with every patch reused recomputes
    only the text rows; with deterministic, row-independent kernels the
    whole state must equal the previous step bit for bit (with either
    prompt-pass GEMM kernel)."""
    import os
    cfg = synth.config_c1()
    w = synth.model_weights(cfg)
    si = synth.step_inputs(cfg, 45)
    os.environ["GVC_GEMM"] = gemm
    try:
        s = _session(cfg, w)
    finally:
        os.environ.pop("GVC_GEMM", None)
    fp, ids = si["frame_prev"].to(DEV), si["text_ids"].to(DEV)
    s.step_prefill(fp, ids)
    ref = _state(s, cfg)
    mask, n_static = s.select_static(fp, fp)
    assert n_static.item() == cfg.n_patches and bool(mask.all())
    s.step_prefill(fp, ids, None, mask)
    got = _state(s, cfg)
    from paper_2608_10824_amd import gvc
    assert s.read(gvc.STATE_ROWS).cpu().tolist() == [cfg.n_text] * cfg.n_layers
    for a, b in zip(got[0] + got[1] + got[2] + [got[3]], ref[0] + ref[1] + ref[2] + [ref[3]]):
        assert np.array_equal(a, b)
    s.close()


def test_no_static_patch_equals_fresh_full_pass():
    cfg = synth.config_c1()
    w = synth.model_weights(cfg)
    si = synth.step_inputs(cfg, 0)
    s = _session(cfg, w)
    fp, ft, ids = si["frame_prev"].to(DEV), si["frame_t"].to(DEV), si["text_ids"].to(DEV)
    s.step_prefill(fp, ids)
    mask, n_static = s.select_static(ft, fp)
    assert n_static.item() == 0 and not bool(mask.any())
    s.step_prefill(ft, ids, None, mask)
    got = _state(s, cfg)
    s2 = _session(cfg, w)
    s2.step_prefill(ft, ids)
    ref = _state(s2, cfg)
    for a, b in zip(got[0] + [got[3]], ref[0] + [ref[3]]):
        assert np.array_equal(a, b)
    s.close()
    s2.close()


def test_zero_frames_and_per_episode_counts():
    """All-zero patches are static against all-zero patches and dynamic
    against anything else; episodes of one batch keep their own counts."""
    cfg = synth.config_c1().with_(batch=3)
    w = synth.model_weights(cfg)
    s = _session(cfg, w)
    si = synth.step_inputs(cfg, [0, 17, 64])
    fp, ft = si["frame_prev"].clone(), si["frame_t"].clone()
    fp[2] = 0
    ft[2] = 0
    ft[1, 0, :14, :14, :] = 0          # patch 0 of episode 1: zero vs non-zero
    mask, n_static = s.select_static(ft.to(DEV), fp.to(DEV))
    exp = []
    for b in range(cfg.batch):
        m, n, st, _ = op.select_static(ft[b].numpy(), fp[b].numpy(), cfg.patch, cfg.tau, cfg.permille())
        exp.append(m)
        assert n_static[b].item() == n
    assert np.array_equal(mask.cpu().numpy().astype(bool), np.stack(exp))
    assert n_static.cpu().tolist()[2] == cfg.n_patches
    ids = si["text_ids"].to(DEV)
    s.step_prefill(fp.to(DEV), ids)
    s.decode_actions()
    s.margin_gate(force=[0, 0, 0])
    s.step_prefill(ft.to(DEV), ids, None, mask)
    from paper_2608_10824_amd import gvc
    rows = s.read(gvc.STATE_ROWS).cpu().tolist()
    assert rows == [sum(cfg.prompt_len - int(e[l].sum()) for e in exp) for l in range(cfg.n_layers)]
    s.close()


def test_single_action_token():
    """D = 1: the prompt pass's head row gives the only token; no decode pass."""
    cfg = synth.config_c1().with_(n_decode=1)
    w = synth.model_weights(cfg)
    si = synth.step_inputs(cfg, 45)
    s = _session(cfg, w)
    o = OracleVLA(cfg, w)
    s.step_prefill(si["frame_prev"].to(DEV), si["text_ids"].to(DEV))
    o.step_prefill(si["frame_prev"].numpy(), si["text_ids"].numpy())
    tok, mg, lg = s.decode_actions(logits=True)
    tok_o, mg_o, lg_o = o.decode_actions()
    torch.cuda.synchronize()
    assert rel_err(lg.cpu().numpy(), lg_o) <= TOL
    check_tokens(tok.cpu().numpy(), lg.cpu().numpy(), tok_o, lg_o, cfg.bin_lo)
    check_margins(mg.cpu().numpy(), mg_o, lg.cpu().numpy(), lg_o, cfg.bin_lo)
    s.close()


def test_largest_frame_selection():
    """1024 patches (448 x 448, p = 14), the most the library accepts:
    exact masks and ranking-dependent per-layer counts against the oracle."""
    cfg = synth.config_c1().with_(img=448, reuse_permille=[700, 300])
    w = synth.model_weights(cfg)
    s = _session(cfg, w)
    si = synth.step_inputs(cfg, 600)
    mask, n_static = s.select_static(si["frame_t"].to(DEV), si["frame_prev"].to(DEV))
    m, n, _, _ = op.select_static(si["frame_t"][0].numpy(), si["frame_prev"][0].numpy(), cfg.patch, cfg.tau,
                                  cfg.permille())
    assert n == 600 and n_static.item() == 600
    assert np.array_equal(mask[0].cpu().numpy().astype(bool), m)
    assert mask[0].sum(dim=1).cpu().tolist() == [420, 180]
    s.close()


def _mid_bins_normaliser():
    return synth.config_mid().with_(norm_full_vocab=False)


def _c1_odd_head_blocks():
    # 1008 logits: 63 LM-head blocks (an odd count), the bins starting at id
    # 808, inside a block
    return synth.config_c1().with_(vocab=1008, n_bins=200)


@pytest.mark.parametrize("cfg_fn", [synth.config_c1, synth.config_mid, _mid_bins_normaliser, _c1_odd_head_blocks])
def test_decode_pass_matches_per_step_launches(cfg_fn, monkeypatch):
    """The single-launch decode pass (one episode) and the per-step launches
    compute the same passes: with the same fed-back tokens their logits agree
    to the bf16 tolerance, and the single-launch path is the one that ran.
    The pass runs with the LM head and the token choice inside it (the
    default) and with them as separate launches (decode flags 3): both give
    the oracle's tokens and margins to the bound their logit error implies,
    and each token is the argmax of that run's own logits."""
    from paper_2608_10824_amd import gvc
    cfg = cfg_fn()
    w = synth.model_weights(cfg)
    si = synth.step_inputs(cfg, cfg.n_patches // 2)
    o = OracleVLA(cfg, w)
    o.step_prefill(si["frame_prev"].numpy(), si["text_ids"].numpy())
    tok_o, m_o, lg_o = o.decode_actions()
    forced = torch.from_numpy(tok_o.astype(np.int32)).to(DEV)
    got = {}
    for mode in ("legacy", "split", "fused"):
        monkeypatch.delenv("GVC_DECODE", raising=False)
        monkeypatch.delenv("GVC_DECODE_FLAGS", raising=False)
        if mode == "legacy":
            monkeypatch.setenv("GVC_DECODE", "legacy")
        elif mode == "split":
            monkeypatch.setenv("GVC_DECODE_FLAGS", "3")
        s = _session(cfg, w)
        s.step_prefill(si["frame_prev"].to(DEV), si["text_ids"].to(DEV))
        gvc.profile_begin(s.ctx, gvc.K_DECODE_PASS, 64)
        tok, mg, lg = s.decode_actions(logits=True, forced_tokens=forced)
        _, n = gvc.profile_end(s.ctx)
        assert n == (0 if mode == "legacy" else cfg.n_decode - 1)
        s.margin_gate()   # surfaces a barrier timeout of the single-launch path
        got[mode] = (tok.cpu().numpy(), mg.cpu().numpy(), lg.cpu().numpy())
        s.close()
    for mode, (tok, mg, lg) in got.items():
        assert rel_err(lg, lg_o) <= TOL, mode
        check_tokens(tok, lg, tok_o.reshape(tok.shape), lg_o.reshape(lg.shape), cfg.bin_lo)
        check_margins(mg, m_o.reshape(mg.shape), lg, lg_o.reshape(lg.shape), cfg.bin_lo, cfg.norm_full_vocab)
    assert rel_err(got["fused"][2], got["legacy"][2]) <= TOL
    assert rel_err(got["fused"][2], got["split"][2]) <= TOL


@pytest.mark.parametrize("mode", ["single", "legacy"])
def test_forced_tokens_outside_the_vocabulary_are_clamped(mode, monkeypatch):
    """A fed-back id below 0 or at or above V reads the embedding row of 0 or
    V - 1: the decode equals, bit for bit, the one fed those ids (single-launch
    pass and per-step launches)."""
    cfg = synth.config_c1()
    w = synth.model_weights(cfg)
    si = synth.step_inputs(cfg, 0)
    if mode == "legacy":
        monkeypatch.setenv("GVC_DECODE", "legacy")
    V, D = cfg.vocab, cfg.n_decode
    wild = [V + 7, -3, V, 5, -1, 2 * V, 0][:D]
    tame = [min(max(t, 0), V - 1) for t in wild]
    got = []
    for ids in (wild, tame):
        s = _session(cfg, w)
        s.step_prefill(si["frame_prev"].to(DEV), si["text_ids"].to(DEV))
        forced = torch.tensor([ids], dtype=torch.int32, device=DEV)
        tok, mg, lg = s.decode_actions(logits=True, forced_tokens=forced)
        s.margin_gate()
        got.append((tok.cpu().numpy(), mg.cpu().numpy(), lg.cpu().numpy()))
        s.close()
    for a, b in zip(*got):
        assert np.array_equal(a, b)


def test_text_ids_outside_the_vocabulary_are_clamped():
    """Prompt text ids below 0 or at or above V embed as 0 or V - 1: the
    prompt pass gives the same state, bit for bit."""
    cfg = synth.config_c1()
    w = synth.model_weights(cfg)
    si = synth.step_inputs(cfg, 0)
    V = cfg.vocab
    wild = si["text_ids"].clone()
    wild[0, 1], wild[0, 2], wild[0, 3] = V + 3, -7, 2 * V
    tame = wild.clamp(0, V - 1)
    states = []
    for ids in (wild, tame):
        s = _session(cfg, w)
        s.step_prefill(si["frame_prev"].to(DEV), ids.to(DEV))
        states.append(_state(s, cfg))
        s.close()
    a, b = states
    for x, y in zip(a[0] + a[1] + a[2] + [a[3]], b[0] + b[1] + b[2] + [b[3]]):
        assert np.array_equal(x, y)


@pytest.mark.parametrize("name", ["C1V-B2", "C4T-bidir-B2"])
def test_batched_front_end_and_action_block(name):
    """Two episodes at once: the ViT front end (two views, so four view
    passes) and the action block each run per episode; every state element
    of both episodes after a full and a partial step, against the oracle."""
    from paper_2608_10824_amd import gvc
    if name == "C1V-B2":
        cfg = synth.config_c1v().with_(batch=2, n_views=2)
    else:
        cfg = synth.config_c4_tiny().with_(batch=2, action_bidir=True)
    w = synth.model_weights(cfg)
    si = synth.step_inputs(cfg, [40, 70])
    s = _session(cfg, w)
    o = OracleVLA(cfg, w)
    fp, ft, ids, ex = si["frame_prev"], si["frame_t"], si["text_ids"], si["extra_rows"]
    exd = None if ex is None else ex.to(DEV)
    exn = None if ex is None else ex.numpy()
    s.step_prefill(fp.to(DEV), ids.to(DEV), exd)
    o.step_prefill(fp.numpy(), ids.numpy(), exn)
    H, K, V, z = _state(s, cfg)
    for l in range(cfg.n_layers + 1):
        assert rel_err(H[l], o.H[l]) <= TOL, ("full", l)
    assert rel_err(z, o.head_logits) <= TOL
    s.decode_actions()
    o.decode_actions()
    s.margin_gate(force=[0, 0])
    o.margin_gate(force=[0, 0])
    mask, n_static = s.select_static(ft.to(DEV), fp.to(DEV))
    mo, no = o.select_static(ft.numpy(), fp.numpy())
    assert np.array_equal(mask.cpu().numpy().astype(bool), mo) and n_static.cpu().tolist() == no.tolist()
    s.step_prefill(ft.to(DEV), ids.to(DEV), exd, mask)
    o.step_prefill(ft.numpy(), ids.numpy(), exn, mo)
    assert s.read(gvc.STATE_ROWS).cpu().tolist() == [int(x) for x in o.recomputed.sum(axis=0)]
    H, K, V, z = _state(s, cfg)
    P = cfg.prompt_len
    errs = {"H%d" % l: rel_err(H[l], o.H[l]) for l in range(cfg.n_layers + 1)}
    for l in range(cfg.n_layers):
        errs["K%d" % l] = rel_err(K[l][:, :, :P], o.K[l].transpose(0, 2, 1, 3)[:, :, :P])
    errs["logits"] = rel_err(z, o.head_logits)
    print(name, {k: "%.2e" % v for k, v in errs.items()})
    assert all(v <= TOL for v in errs.values()), errs
    s.close()


def test_sixteen_episodes_prompt_and_decode():
    """16 episodes of the mid-size decoder (16 heads of 128, two views):
    2176 prompt rows (the many-row projection kernel) and a batched decode
    whose attention takes one value slice per (head, episode) (16 x 16 = 256
    pairs).  Episodes are independent, so episodes 0 and 15 are checked
    against a one-episode oracle each: the prompt state, and the decode with
    every GPU episode fed the oracle's greedy tokens (episode 0's where the
    episode is not checked); the GPU's own argmax tokens and margins against
    the oracle's."""
    from paper_2608_10824_amd import gvc
    cfg = synth.config_mid().with_(batch=16)
    w = synth.model_weights(cfg)
    si = synth.step_inputs(cfg, 90)
    s = _session(cfg, w)
    fp, ids = si["frame_prev"], si["text_ids"]
    s.step_prefill(fp.to(DEV), ids.to(DEV))
    H, K, V, z = _state(s, cfg)
    one = cfg.with_(batch=1)
    oracles = {}
    for b in (0, cfg.batch - 1):
        o = OracleVLA(one, w)
        o.step_prefill(fp.numpy()[b:b + 1], ids.numpy()[b:b + 1])
        for l in range(cfg.n_layers + 1):
            assert rel_err(H[l][b:b + 1], o.H[l]) <= TOL, (b, l)
        oracles[b] = o.decode_actions()
    forced = np.repeat(oracles[0][0], cfg.batch, axis=0)
    forced[cfg.batch - 1] = oracles[cfg.batch - 1][0][0]
    tok, mg, lg = s.decode_actions(logits=True, forced_tokens=torch.from_numpy(forced.astype(np.int32)).to(DEV))
    torch.cuda.synchronize()
    tok, mg, lgn = tok.cpu().numpy(), mg.cpu().numpy(), lg.cpu().numpy()
    for b, (tok_o, m_o, lg_o) in oracles.items():
        err = rel_err(lgn[b:b + 1], lg_o)
        print("episode %d decode logits rel err %.2e" % (b, err))
        assert err <= TOL
        check_tokens(tok[b:b + 1], lgn[b:b + 1], tok_o, lg_o, cfg.bin_lo)
        check_margins(mg[b:b + 1], m_o, lgn[b:b + 1], lg_o, cfg.bin_lo)
    s.close()


def test_many_row_tile_height_does_not_change_a_row():
    """The many-row kernel sums each row over k in the same order whatever
    its tile height (128-, 192- or 256-row tiles), so the same 16-episode
    full and partial steps run with each height forced give bit-identical
    hidden states, K/V caches and head logits."""
    import os
    cfg = synth.config_mid().with_(batch=16)
    w = synth.model_weights(cfg)
    si = synth.step_inputs(cfg, 90)
    ref = None
    for tw in ("2", "3", "4"):
        os.environ["GVC_BIG_TW"] = tw
        try:
            s = _session(cfg, w)
        finally:
            os.environ.pop("GVC_BIG_TW", None)
        fp, ft, ids = si["frame_prev"].to(DEV), si["frame_t"].to(DEV), si["text_ids"].to(DEV)
        s.step_prefill(fp, ids)
        s.decode_actions()
        s.margin_gate(force=[0] * cfg.batch)
        mask, _ = s.select_static(ft, fp)
        s.step_prefill(ft, ids, None, mask)
        got = _state(s, cfg)
        s.close()
        flat = got[0] + got[1] + got[2] + [got[3]]
        if ref is None:
            ref = flat
        else:
            assert all(np.array_equal(a, b) for a, b in zip(flat, ref)), "tile height %s" % tw


@pytest.mark.parametrize("views,text,batch", [(2, 33, 1), (4, 8, 1), (4, 32, 1), (2, 8, 2)],
                         ids=["161-rows", "264-rows", "288-rows", "2x136-rows"])
def test_tall_split_k_tiles_agree_bit_for_bit(views, text, batch, monkeypatch):
    """At 161-288 rows the split-k projections run one tile of 18 token
    blocks per k slice instead of two tiles of 10, and the output projection
    runs on the split-k core in 8 k slices instead of the per-pair kernel's
    8 k shares (GVC_SK_TALL=0 turns both off).  Each slice's partial sums are
    the same MFMA sequence either way and are added in the same order, so a
    full step and a partial step give the same state bit for bit.  MID
    with 161, 264 and 288 prompt rows: 11, 17 and 18 token blocks, the
    lowest and highest heights that take a tall tile; and two episodes of
    136 rows in one launch."""
    cfg = synth.config_mid().with_(n_views=views, n_text=text, batch=batch)
    assert 160 < cfg.batch * cfg.prompt_len <= 288
    w = synth.model_weights(cfg)
    si = synth.step_inputs(cfg, 96)
    states = []
    for tall in ("1", "0"):
        monkeypatch.setenv("GVC_SK_TALL", tall)
        s = _session(cfg, w)
        monkeypatch.delenv("GVC_SK_TALL")
        fp, ft, ids = si["frame_prev"].to(DEV), si["frame_t"].to(DEV), si["text_ids"].to(DEV)
        s.step_prefill(fp, ids)
        s.decode_actions()
        s.margin_gate(force=[0] * cfg.batch)
        mask, _ = s.select_static(ft, fp)
        s.step_prefill(ft, ids, None, mask)
        states.append(_state(s, cfg))
        s.close()
    a, b = states
    for x, y in zip(a[0] + a[1] + a[2] + [a[3]], b[0] + b[1] + b[2] + [b[3]]):
        assert np.array_equal(x, y)


def test_split_k_cores_agree_bit_for_bit(monkeypatch):
    """The two split-k cores of the gate/up projection (decoupled weight and
    token streams in 12-block groups, the default, and the register-fed one
    in 16-block groups, GVC_SK_CORE=0) sum each k slice in the same order, so
    a full and a partial step give the same state bit for bit (MID: 136 rows,
    2 k slices; QKV and down on the per-pair kernel in both runs)."""
    cfg = synth.config_mid()
    w = synth.model_weights(cfg)
    si = synth.step_inputs(cfg, 64)
    states = []
    monkeypatch.setenv("GVC_SK_QKV", "0")
    monkeypatch.setenv("GVC_SK_DOWN", "0")
    for core in ("1", "0"):
        monkeypatch.setenv("GVC_SK_CORE", core)
        s = _session(cfg, w)
        monkeypatch.delenv("GVC_SK_CORE")
        fp, ft, ids = si["frame_prev"].to(DEV), si["frame_t"].to(DEV), si["text_ids"].to(DEV)
        s.step_prefill(fp, ids)
        s.decode_actions()
        s.margin_gate(force=[0])
        mask, _ = s.select_static(ft, fp)
        s.step_prefill(ft, ids, None, mask)
        states.append(_state(s, cfg))
        s.close()
    a, b = states
    for x, y in zip(a[0] + a[1] + a[2] + [a[3]], b[0] + b[1] + b[2] + [b[3]]):
        assert np.array_equal(x, y)
