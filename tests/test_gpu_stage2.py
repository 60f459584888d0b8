"""Stage 2 (task-relevant filtering, Sec. III-B) on the HIP path against the
oracle, through the C ABI: the per-layer, per-head instruction-to-vision
attention recorded by a prompt pass; the selection that removes the top-k
patches from the static set (each side on its own signal, decided in fp32;
equal except for near ties); and the partial step that follows.  C1 (heads
of 64) and MID (heads of 128, two views)."""
import numpy as np
import pytest
import torch

import synth
from oracle.vla import OracleVLA
from oracle.relevance import relevant_patches
from oracle.patches import select_static as select_one
from tests._parity import TOL, rel_err, to_dev, fp32_scores, relevant_near_ties

pytestmark = pytest.mark.gpu

TOPK = 20


@pytest.fixture(scope="module", params=["C1", "MID"])
def run(request):
    from paper_2608_10824_amd.session import Session
    cfg = synth.config_c1() if request.param == "C1" else synth.config_mid()
    cfg = cfg.with_(task_topk=TOPK)
    w = synth.model_weights(cfg)
    si = synth.step_inputs(cfg, 45 * cfg.n_views)
    dev = torch.device("cuda:0")
    s = Session(cfg, to_dev(w, dev), device=dev)
    o = OracleVLA(cfg, w)
    yield cfg, w, si, s, o, dev
    s.close()


def test_stage2_signal_selection_and_step(run):
    """The recorded signal against the oracle's own; each side's selection on
    its own signal (decided in fp32 on both sides), equal unless a patch's
    oracle score sits within the signal error of the k-th boundary; then the
    partial step on those (equal) masks, every state element."""
    from paper_2608_10824_amd import gvc
    cfg, w, si, s, o, dev = run
    fp, ft, ids = si["frame_prev"], si["frame_t"], si["text_ids"]
    s.step_prefill(fp.to(dev), ids.to(dev))
    o.step_prefill(fp.numpy(), ids.numpy())
    tv = s.read(gvc.STATE_TV).cpu().numpy()
    assert tv.shape == o.tv.shape
    err = rel_err(tv, o.tv)
    print("Stage 2 signal rel err %.2e" % err)
    assert err <= TOL
    assert np.all(tv >= 0) and np.all(tv.sum(axis=3) <= cfg.n_text - 1 + 1e-3)

    mask, n_static = s.select_static(ft.to(dev), fp.to(dev))
    sc_o, sc_g = fp32_scores(o.tv), fp32_scores(tv)
    m_o, n_o = o.select_static(ft.numpy(), fp.numpy(), scores=sc_o.astype(np.float64))
    rel_o = relevant_patches(sc_o[0].astype(np.float64), TOPK)
    rel_g = relevant_patches(sc_g[0].astype(np.float64), TOPK)
    ties = relevant_near_ties(sc_o[0], sc_g[0], TOPK, rel_o, rel_g)
    _, n1, static1, _ = select_one(ft.numpy()[0], fp.numpy()[0], cfg.patch, cfg.tau, cfg.permille())
    assert n_o[0] == int((static1 & ~rel_o).sum()) and n_o[0] < n1   # the filter removed the top-k of S
    print("Stage 2 relevant set: %d near-tie patches" % len(ties))
    if ties:   # both selections are valid
        assert n_static.cpu().numpy()[0] == int((static1 & ~rel_g).sum())
    else:
        assert np.array_equal(mask.cpu().numpy().astype(bool), m_o)
        assert n_static.cpu().numpy().tolist() == n_o.tolist()

    # the oracle's selection decides; the GPU's partial step takes its masks
    s.step_prefill(ft.to(dev), ids.to(dev), None, torch.from_numpy(m_o.astype(np.uint8)).to(dev))
    o.step_prefill(ft.numpy(), ids.numpy(), None, m_o)
    rows = s.read(gvc.STATE_ROWS).cpu().numpy().tolist()
    assert rows == [int(x) for x in o.recomputed[0]]
    errs = {"H%d" % l: rel_err(s.read(gvc.STATE_H, l).cpu().numpy(), o.H[l]) for l in range(cfg.n_layers + 1)}
    errs["logits"] = rel_err(s.read(gvc.STATE_HEAD_LOGITS).cpu().numpy(), o.head_logits)
    errs["tv"] = rel_err(s.read(gvc.STATE_TV).cpu().numpy(), o.tv)
    print({k: "%.2e" % v for k, v in errs.items()})
    assert all(v <= TOL for v in errs.values()), errs


def test_stage2_k0_is_stage1():
    """task_topk = 0: no signal is recorded and the masks equal Stage 1's."""
    from paper_2608_10824_amd.session import Session
    from paper_2608_10824_amd import gvc
    cfg = synth.config_c1()
    w = synth.model_weights(cfg)
    si = synth.step_inputs(cfg, 45)
    dev = torch.device("cuda:0")
    s = Session(cfg, to_dev(w, dev), device=dev)
    fp, ft, ids = si["frame_prev"], si["frame_t"], si["text_ids"]
    s.step_prefill(fp.to(dev), ids.to(dev))
    assert gvc.state_item_bytes(s.ctx, gvc.STATE_TV) == 0
    mask, n_static = s.select_static(ft.to(dev), fp.to(dev))
    m1, n1, _, _ = select_one(ft.numpy()[0], fp.numpy()[0], cfg.patch, cfg.tau, cfg.permille())
    assert np.array_equal(mask.cpu().numpy()[0].astype(bool), m1) and n_static.item() == n1
    s.close()
