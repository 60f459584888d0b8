"""Stage 3 computed from attention entropy (Sec. III-B) on the HIP path
against the oracle, through the C ABI: the per-layer, per-head entropy sums a
prompt pass records; the per-layer proportions the selection derives from
them (an integer decision each side takes in fp32 from its own signal,
equal except for near ties); the masks; and the partial step that follows.
C1 (heads of 64) and MID (heads of 128, two views, with Stage 2 on too)."""
import numpy as np
import pytest
import torch

import synth
from oracle.vla import OracleVLA
from oracle.relevance import entropy_permille, relevant_patches
from oracle.patches import select_static as select_one
from tests._parity import TOL, rel_err, to_dev, fp32_scores, fp32_layer_q, layer_q_near_ties, relevant_near_ties

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


def test_stage3_signal_proportions_and_step(run):
    """The recorded entropy signal against the oracle's own; the per-layer
    proportions of each side from its own signal, taken in fp32 on both
    sides (equal except for layers whose oracle value is within the signal
    error of an integer boundary); the masks; the partial step that follows,
    every state element."""
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
    ties = 0
    q_o = []
    for b in range(cfg.batch):
        q_o.append(fp32_layer_q(o.ent[b], n_instr))
        ties += len(layer_q_near_ties(o.ent[b], ent[b], n_instr, q_o[b], q_gpu[b].tolist()))
        # the fp64 proportions of the reading itself are within one of the fp32 ones
        assert np.all(np.abs(np.array(entropy_permille(o.ent[b], n_instr)) - np.array(q_o[b])) <= 1)
        print("layer proportions gpu", q_gpu[b].tolist(), "oracle", q_o[b])
    sc_o = fp32_scores(o.tv).astype(np.float64) if cfg.task_topk else None
    ties_rel = []
    if cfg.task_topk:
        tv = s.read(gvc.STATE_TV).cpu().numpy()
        sc_g = fp32_scores(tv)
        ties_rel = relevant_near_ties(sc_o[0], sc_g[0], cfg.task_topk,
                                      relevant_patches(sc_o[0], cfg.task_topk),
                                      relevant_patches(sc_g[0].astype(np.float64), cfg.task_topk))
    m_o, n_o = o.select_static(ft.numpy(), fp.numpy(), scores=sc_o, layer_q=q_o)
    print("near ties: %d layer proportions, %d relevant patches" % (ties, len(ties_rel)))
    if not (ties or ties_rel):
        assert np.array_equal(mask.cpu().numpy().astype(bool), m_o)
        assert n_static.cpu().numpy().tolist() == n_o.tolist()
    for l in range(cfg.n_layers):
        assert int(m_o[0, l].sum()) == (int(q_o[0][l]) * int(n_o[0])) // 1000

    # the oracle's selection decides; the GPU's partial step takes its masks
    s.step_prefill(ft.to(dev), ids.to(dev), None, torch.from_numpy(m_o.astype(np.uint8)).to(dev))
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
