"""The C ABI library loads and exports every function include/gvc.h declares,
and its host-only calls validate shapes (CPU only, no compute calls)."""
import os
import re

import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "gvc.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(gvc_[a-z_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported():
    from paper_2608_10824_amd import gvc
    L = gvc.lib()
    names = _declared()
    assert "gvc_step_prefill" in names and len(names) >= 10
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(gvc.EXPORTED)


def test_sizes_for_every_config():
    from paper_2608_10824_amd import gvc
    from paper_2608_10824_amd.session import desc_from
    for name, f in synth.ALL_CONFIGS.items():
        w, s, k = gvc.sizes(desc_from(f()))
        assert w > 0 and s > 0 and k > 0 and w % 256 == 0
    c2 = synth.config_c2()
    w, s, k = gvc.sizes(desc_from(c2))
    # packed weights: the 7B backbone plus the patch projection, bf16
    params = 32 * (4 * 4096 ** 2 + 3 * 4096 * 11008) + 2 * 32000 * 4096
    assert params * 2 <= w <= params * 2 * 1.01


@pytest.mark.parametrize("field,value", [("n_heads", 48), ("d_model", 100), ("batch", 0), ("batch", 65),
                                         ("ffn", 30), ("img", 100), ("n_text", 0)])
def test_bad_shapes_rejected(field, value):
    from paper_2608_10824_amd import gvc
    from paper_2608_10824_amd.session import desc_from
    d = desc_from(synth.config_c1())
    setattr(d, field, value)
    with pytest.raises(gvc.GvcError) as e:
        gvc.sizes(d)
    assert e.value.code == gvc.GVC_EINVAL
    assert gvc.last_error()


def test_null_context_calls_fail_cleanly():
    from paper_2608_10824_amd import gvc
    with pytest.raises(gvc.GvcError):
        gvc.invalidate(None, -1)
    with pytest.raises(gvc.GvcError):
        gvc.step_prefill(None, 0, 0, None, None)
