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


@pytest.mark.parametrize("field,value", [("n_heads", 48), ("d_model", 100), ("batch", 0), ("batch", 17),
                                         ("ffn", 30), ("img", 100), ("n_text", 0), ("task_topk", -1),
                                         ("task_topk", 65), ("entropy_reuse", 2), ("action_bidir", 1),
                                         ("vit_layers", 65), ("vit_layers", -1)])
def test_bad_shapes_rejected(field, value):
    from paper_2608_10824_amd import gvc
    from paper_2608_10824_amd.session import desc_from
    d = desc_from(synth.config_c1())
    setattr(d, field, value)
    with pytest.raises(gvc.GvcError) as e:
        gvc.sizes(d)
    assert e.value.code == gvc.GVC_EINVAL
    assert gvc.last_error()


@pytest.mark.parametrize("field,value", [("vit_dim", 96), ("vit_heads", 3), ("vit_heads", 16), ("vit_ffn", 40),
                                         ("vit_eps", 0.0)])
def test_bad_front_end_rejected(field, value):
    """With the ViT front end on, its shape limits are checked (width a
    multiple of 64, heads of 64 or 128, MLP width a multiple of 32, eps > 0)."""
    from paper_2608_10824_amd import gvc
    from paper_2608_10824_amd.session import desc_from
    d = desc_from(synth.config_c1v())
    gvc.sizes(d)
    setattr(d, field, value)
    with pytest.raises(gvc.GvcError) as e:
        gvc.sizes(d)
    assert e.value.code == gvc.GVC_EINVAL


def test_stage_limits_and_action_block_need_their_shapes():
    """Stages 2/3 need at most 32 instruction tokens after the image; the
    action block needs parallel decode; both accepted on their configs."""
    from paper_2608_10824_amd import gvc
    from paper_2608_10824_amd.session import desc_from
    gvc.sizes(desc_from(synth.config_c1().with_(task_topk=10, entropy_reuse=True)))
    gvc.sizes(desc_from(synth.config_c4_tiny().with_(action_bidir=True)))
    for cfg in (synth.config_c1().with_(n_text=40, task_topk=10), synth.config_c1().with_(n_text=40, entropy_reuse=True)):
        with pytest.raises(gvc.GvcError):
            gvc.sizes(desc_from(cfg))


def test_null_context_calls_fail_cleanly():
    from paper_2608_10824_amd import gvc
    with pytest.raises(gvc.GvcError):
        gvc.invalidate(None, -1)
    with pytest.raises(gvc.GvcError):
        gvc.step_prefill(None, 0, 0, None, None)


@pytest.mark.parametrize("field,value", [("img", 462), ("batch", 17), ("batch", 0), ("n_views", 2),
                                         ("task_topk", 1), ("entropy_reuse", 1), ("patch", 15)])
def test_noalloc_selection_rejects_sizes_beyond_its_scratch(field, value):
    """The allocation-free selection validates its sizes on the host before
    any device work: at most 16 episodes of 1024 patches (here 33^2 = 1089
    patches, or two views of 1024), no Stage 2 or 3; bad pointers fail the
    same way (nothing is launched, so this runs without a GPU)."""
    from paper_2608_10824_amd import gvc
    from paper_2608_10824_amd.session import desc_from
    d = desc_from(synth.config_c1().with_(img=448))
    setattr(d, field, value)
    with pytest.raises(gvc.GvcError) as e:
        gvc.select_static_noalloc(d, 256, 256, 99, 100, None, 256, 256, None)
    assert e.value.code == gvc.GVC_EINVAL and gvc.last_error()
    d = desc_from(synth.config_c1())
    with pytest.raises(gvc.GvcError) as e:
        gvc.select_static_noalloc(d, 256, 256, 99, 100, None, None, 256, None)
    assert e.value.code == gvc.GVC_EINVAL
    with pytest.raises(gvc.GvcError) as e:
        gvc.select_static_noalloc(d, 256, 256, 101, 100, None, 256, 256, None)
    assert e.value.code == gvc.GVC_EINVAL
