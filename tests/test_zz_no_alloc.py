"""The allocation-free attention entry point (pcpp_partial_attention_noalloc)
against pcpp_partial_attention, through the C ABI: the same kernels and
plan on the same inputs, so the outputs must be identical; two calls in a
row, the second with a smaller input, then a geometry too large for the
fixed device array."""

import numpy as np
import pytest

from paper_2412_02962_amd import synth
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu


def _say(*a):
    print("[case]", *a, flush=True)


def _both(cfg):
    import torch
    from paper_2412_02962_amd import pcpp
    inp = synth.attention_inputs(cfg)
    ref = gu.run_attention(cfg, inp)
    d = {k: gu.to_dev(v, cfg.dtype) for k, v in inp.items()}
    out = torch.full_like(d["q"], float("nan"))
    pcpp.pcpp_partial_attention_noalloc(gu.geom(cfg), d["q"], d["k_fresh"], d["v_fresh"], d["k_up"], d["v_up"],
                                        d["k_dn"], d["v_dn"], out)
    torch.cuda.synchronize()
    return ref, out


def test_noalloc_matches_the_workspace_entry_point_on_two_calls():
    import torch
    for name in ("sdxl2048_l1_p25", "sdxl2048_l2_edge"):   # the second call is the smaller input
        cfg = synth.ATTN_CONFIGS[name]
        _say("noalloc", name)
        ref, out = _both(cfg)
        gu.assert_close(cfg, gu.to_f64(out), gu.to_f64(ref), f"noalloc {name}")
        assert torch.equal(out, ref), name
    # ragged shape, unsplit launch, f32 path
    for cfg in (synth.AttnConfig(name="r", H=12, W=20, n=3, i=1, p=0.5, heads=2, d=64, dtype="bf16", seed_id=91),
                synth.ATTN_CONFIGS["tiny_f32"]):
        _say("noalloc", cfg.name)
        ref, out = _both(cfg)
        assert torch.equal(out, ref), cfg.name


def test_noalloc_refuses_a_geometry_beyond_its_array():
    from paper_2412_02962_amd import pcpp
    cfg = synth.AttnConfig(name="3840", H=240, W=240, n=2, i=0, p=0.3, heads=10, d=64, dtype="bf16", seed_id=42)
    _say("noalloc too large")
    import torch
    q = torch.zeros((1, cfg.n_q, cfg.C), dtype=torch.bfloat16, device=gu.DEV)
    with pytest.raises(pcpp.PcppError) as e:
        pcpp.pcpp_partial_attention_noalloc(gu.geom(cfg), q, q, q, None, None, q, q, q)
    assert e.value.status == pcpp.PCPP_EWORKSPACE
