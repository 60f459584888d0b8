"""Robustness modes of the HIP path, through the C ABI.

* Poisoned arenas (GVC_POISON=1): the state and workspace start as 0xFF
  bytes (NaN in fp32 and bf16) instead of zeros, apart from the few words the
  library documents as starting at zero.  A full step, a decode, a partial
  step and a second decode must then give bit-identical results to a session
  whose arenas start at zero, so no kernel reads memory before writing it.
* Validated row lists (GVC_VALIDATE=1): every prompt pass copies its
  compacted row lists to the host and checks them against the rule of the
  partial forward pass (gvc_check_rows); the same sequence must pass the
  check and give the same results."""
import numpy as np
import pytest
import torch

import synth
from tests._parity import to_dev

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")

CONFIGS = {
    "C1": lambda: synth.config_c1(),
    "MID": lambda: synth.config_mid(),
    "C4T-bidir": lambda: synth.config_c4_tiny().with_(action_bidir=True),
    "C1V": lambda: synth.config_c1v(),
    "MID-big": lambda: synth.config_mid(),
}


def _run(cfg, w, si, env, monkeypatch):
    """Full step on the previous frame, decode, kept gate, selection, partial
    step on the current frame, decode; every result as host arrays."""
    from paper_2608_10824_amd import gvc
    from paper_2608_10824_amd.session import Session
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    try:
        s = Session(cfg, to_dev(w, DEV), device=DEV)
    finally:
        for k in env:
            monkeypatch.delenv(k, raising=False)
    ex = si["extra_rows"].to(DEV) if si.get("extra_rows") is not None else None
    fp, ft, ids = si["frame_prev"].to(DEV), si["frame_t"].to(DEV), si["text_ids"].to(DEV)
    # written only by a decode: shows what the arenas started as
    init_margins = s.read(gvc.STATE_MARGINS).cpu().numpy()
    out = {}
    s.step_prefill(fp, ids, ex)
    t0, m0, l0 = s.decode_actions(logits=True)
    out.update(tok0=t0.cpu().numpy(), mg0=m0.cpu().numpy(), lg0=l0.cpu().numpy())
    s.margin_gate(force=[0] * cfg.batch)
    mask, n_static = s.select_static(ft, fp)
    out.update(mask=mask.cpu().numpy(), n_static=n_static.cpu().numpy())
    s.step_prefill(ft, ids, ex, mask)
    for l in range(cfg.n_layers + 1):
        out["H%d" % l] = s.read(gvc.STATE_H, l).cpu().numpy()
    for l in range(cfg.n_layers):
        out["K%d" % l] = s.read(gvc.STATE_K, l).float().cpu().numpy()[..., :cfg.prompt_len, :]
        out["V%d" % l] = s.read(gvc.STATE_V, l).float().cpu().numpy()[..., :cfg.prompt_len]
    out["head"] = s.read(gvc.STATE_HEAD_LOGITS).cpu().numpy()
    out["rows"] = s.read(gvc.STATE_ROWS).cpu().numpy()
    t1, m1, l1 = s.decode_actions(logits=True)
    out.update(tok1=t1.cpu().numpy(), mg1=m1.cpu().numpy(), lg1=l1.cpu().numpy())
    m, fire = s.margin_gate()
    out.update(gate_m=np.asarray(m), gate_f=np.asarray(fire))
    s.close()
    return out, init_margins


def _inputs(name):
    cfg = CONFIGS[name]()
    return cfg, synth.model_weights(cfg), synth.step_inputs(cfg, cfg.n_patches // 2, stream=7)


@pytest.mark.parametrize("name", list(CONFIGS))
def test_poisoned_arenas_give_the_same_step(name, monkeypatch):
    cfg, w, si = _inputs(name)
    big = {"GVC_GEMM": "big"} if name.endswith("-big") else {}
    ref, init_ref = _run(cfg, w, si, big, monkeypatch)
    got, init_got = _run(cfg, w, si, dict(big, GVC_POISON="1"), monkeypatch)
    assert (init_ref == 0).all() and np.isnan(init_got).all()      # the poison is really there
    assert 0 < int(ref["rows"].min()) < cfg.batch * cfg.prompt_len   # a real partial step
    for k, a in ref.items():
        b = got[k]
        if a.dtype.kind == "f":
            assert np.isfinite(b).all(), (name, k)
        assert np.array_equal(a, b), (name, k)


@pytest.mark.parametrize("name", ["C1", "C4T-bidir", "MID-big"])
def test_validated_row_lists_pass_and_change_nothing(name, monkeypatch):
    cfg, w, si = _inputs(name)
    big = {"GVC_GEMM": "big"} if name.endswith("-big") else {}
    ref, _ = _run(cfg, w, si, big, monkeypatch)
    got, _ = _run(cfg, w, si, dict(big, GVC_VALIDATE="1"), monkeypatch)
    for k, a in ref.items():
        assert np.array_equal(a, got[k]), (name, k)


def test_validation_hook_reports_a_bad_list(monkeypatch):
    """GVC_VALIDATE=2 alters the host copy of the lists before the check, so
    the prompt pass must stop with GVC_EDEVICE and the check's message."""
    from paper_2608_10824_amd import gvc
    from paper_2608_10824_amd.session import Session
    cfg, w, si = _inputs("C1")
    monkeypatch.setenv("GVC_VALIDATE", "2")
    s = Session(cfg, to_dev(w, DEV), device=DEV)
    monkeypatch.delenv("GVC_VALIDATE")
    with pytest.raises(gvc.GvcError) as e:
        s.step_prefill(si["frame_prev"].to(DEV), si["text_ids"].to(DEV))
    assert e.value.code == gvc.GVC_EDEVICE and "row lists fail the host check" in str(e.value)
    assert "layer 0" in str(e.value)
    s.close()
