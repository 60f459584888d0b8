"""Stage 3 computed from attention entropy (Sec. III-B) on the HIP path
against the oracle, through the C ABI: the per-layer, per-head entropy sums a
prompt pass records; the per-layer proportions the selection derives from
them (an integer decision taken in fp32, checked exactly against the same
fp32 steps applied to the GPU's signal and within the signal's error of the
oracle's fp64 proportions); the masks; and the partial step that follows.
C1 (heads of 64) and MID (heads of 128, two views, with Stage 2 on too)."""
import numpy as np
import pytest
import torch

import synth
from oracle.vla import OracleVLA
from oracle.relevance import entropy_permille
from oracle.patches import select_static as select_one
from tests._parity import TOL, rel_err, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", params=["C1", "MID"])
def run(request):
    from paper_2608_10824_amd.session import Session
    if request.param == "C1":
        cfg = synth.config_c1().with_(entropy_reuse=True)
    else:
        cfg = synth.config_mid().with_(entropy_reuse=True, task_topk=16)
    w = synth.model_weights(cfg)
    si = synth.step_inputs(cfg, 45 * cfg.n_views)
    dev = torch.device("cuda:0")
    s = Session(cfg, to_dev(w, dev), device=dev)
    o = OracleVLA(cfg, w)
    yield cfg, w, si, s, o, dev
    s.close()


def _q_fp32(ent, n_instr):
    """The selection's per-layer proportions from ent [L][H] (fp32), taking
    the same fp32 steps in the same order."""
    f = np.float32
    L, H = ent.shape
    out, sl = [], f(0)
    for l in range(L):
        e = f(0)
        for h in range(H):
            e = f(e + f(ent[l, h]))
        u = f(f(1) - f(e / f(H * n_instr)))
        sl = u if l == 0 else f(sl + f(f(u - sl) * f(0.5)))
        c = min(max(sl, f(0)), f(1))
        out.append(int(np.floor(f(f(1000) * c))))
    return out


def _gpu_scores(tv):
    B, L, H, N = tv.shape
    flat = tv.reshape(B, L * H, N).astype(np.float32)
    acc = np.zeros((B, N), dtype=np.float32)
    for c in range(L * H):
        acc = (acc + flat[:, c, :]).astype(np.float32)
    return acc


def test_stage3_signal_proportions_and_step(run):
    from paper_2608_10824_amd import gvc
    cfg, w, si, s, o, dev = run
    fp, ft, ids = si["frame_prev"], si["frame_t"], si["text_ids"]
    n_instr = cfg.n_text - 1

    # before any prompt pass the fixed proportions apply
    mask0, n0 = s.select_static(ft.to(dev), fp.to(dev))
    m1, n1, _, _ = select_one(ft.numpy()[0], fp.numpy()[0], cfg.patch, cfg.tau, cfg.permille())
    assert np.array_equal(mask0.cpu().numpy()[0].astype(bool), m1) and n0[0].item() == n1

    s.step_prefill(fp.to(dev), ids.to(dev))
    o.step_prefill(fp.numpy(), ids.numpy())
    ent = s.read(gvc.STATE_ENTROPY).cpu().numpy()
    assert ent.shape == o.ent.shape == (cfg.batch, cfg.n_layers, cfg.n_heads)
    err = rel_err(ent, o.ent)
    print("Stage 3 signal rel err %.2e" % err)
    assert err <= TOL
    assert np.all(ent > 0) and np.all(ent <= n_instr * (1 + 1e-5))

    mask, n_static = s.select_static(ft.to(dev), fp.to(dev))
    q_gpu = s.read(gvc.STATE_LAYER_Q).cpu().numpy()
    for b in range(cfg.batch):
        # exact: the same fp32 steps on the GPU's own signal
        assert q_gpu[b].tolist() == _q_fp32(ent[b], n_instr)
        # close to the oracle's fp64 proportions: s_l is a convex mix of the
        # u_j, so |dq| <= 1000 max_l |dE_l| + 1
        q_o = entropy_permille(o.ent[b], n_instr)
        dE = np.abs(ent[b].astype(np.float64).sum(axis=1) - o.ent[b].sum(axis=1)).max() / (cfg.n_heads * n_instr)
        assert np.all(np.abs(np.array(q_o) - q_gpu[b]) <= 1000 * dE + 1), (q_o, q_gpu[b].tolist())
        print("layer proportions gpu", q_gpu[b].tolist(), "oracle", q_o)

    # masks: exact against the oracle's selection on the GPU's proportions
    # (and, with Stage 2, on the GPU's scores)
    sc = _gpu_scores(s.read(gvc.STATE_TV).cpu().numpy()).astype(np.float64) if cfg.task_topk else None
    m_o, n_o = o.select_static(ft.numpy(), fp.numpy(), scores=sc, layer_q=q_gpu)
    assert np.array_equal(mask.cpu().numpy().astype(bool), m_o)
    assert n_static.cpu().numpy().tolist() == n_o.tolist()
    for l in range(cfg.n_layers):
        assert int(m_o[0, l].sum()) == (int(q_gpu[0, l]) * int(n_o[0])) // 1000

    # the partial step on that mask
    s.step_prefill(ft.to(dev), ids.to(dev), None, s.mask)
    o.step_prefill(ft.numpy(), ids.numpy(), None, m_o)
    rows = s.read(gvc.STATE_ROWS).cpu().numpy().tolist()
    assert rows == [int(x) for x in o.recomputed[0]]
    errs = {"H%d" % l: rel_err(s.read(gvc.STATE_H, l).cpu().numpy(), o.H[l]) for l in range(cfg.n_layers + 1)}
    errs["logits"] = rel_err(s.read(gvc.STATE_HEAD_LOGITS).cpu().numpy(), o.head_logits)
    errs["ent"] = rel_err(s.read(gvc.STATE_ENTROPY).cpu().numpy(), o.ent)
    print({k: "%.2e" % v for k, v in errs.items()})
    assert all(v <= TOL for v in errs.values()), errs


def test_stage3_off_has_no_signal():
    from paper_2608_10824_amd.session import Session
    from paper_2608_10824_amd import gvc
    cfg = synth.config_c1()
    w = synth.model_weights(cfg)
    dev = torch.device("cuda:0")
    s = Session(cfg, to_dev(w, dev), device=dev)
    assert gvc.state_item_bytes(s.ctx, gvc.STATE_ENTROPY) == 0
    assert gvc.state_item_bytes(s.ctx, gvc.STATE_LAYER_Q) == 0
    s.close()
