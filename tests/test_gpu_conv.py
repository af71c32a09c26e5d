"""GPU parity of pcpp_conv3x3 (the U-Net's stride-1, stride-2 and
upsampling 3x3 convolutions on a band) against the float64 oracle, through
the C ABI.

Tolerance: the inputs are bf16 and exact in both; the library accumulates
in float32 and rounds y to bf16 once: |dy| <= 2^-8 |y| + 2^-12 rms(y) per
element (the second term covers float32 accumulation over 9 c_in terms),
mean-abs <= 2^-9 rms(y).
"""

import numpy as np
import pytest

import oracle
from paper_2412_02962_amd import synth
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

MODES = {0: "same", 1: "down", 2: "up"}
CASES = [
    (12, 20, 3, 1, 64, 128, 2, 0), (12, 20, 3, 0, 64, 64, 1, 0), (12, 20, 3, 2, 128, 64, 1, 0),
    (8, 24, 1, 0, 64, 64, 1, 0),
    (16, 20, 4, 2, 64, 64, 2, 1), (16, 20, 4, 0, 128, 64, 1, 1), (8, 6, 2, 1, 64, 128, 3, 1),
    (6, 10, 3, 1, 128, 64, 1, 2), (6, 10, 3, 2, 64, 64, 2, 2), (4, 3, 1, 0, 64, 128, 1, 2),
]
FULL = list(synth.CONV_CONFIGS.items())


def _say(*a):
    print("[case]", *a, flush=True)


def _run(H, W, n, i, ci, co, B, mode, seed):
    import torch
    from paper_2412_02962_amd import pcpp
    inp = synth.conv_inputs(H, W, n, i, ci, co, B, seed)
    d = {k: gu.to_dev(v, "bf16") for k, v in inp.items()}
    g = pcpp.make_conv_geom(H, W, n, i, ci, co, B, mode)
    h = H // n
    tokens = {0: h * W, 1: (h // 2) * (W // 2), 2: 4 * h * W}[mode]
    y = torch.full((B, tokens, co), float("nan"), dtype=torch.bfloat16, device=gu.DEV)
    wsb = pcpp.pcpp_conv3x3_workspace_size(g)
    assert wsb > 0
    ws = torch.full((wsb,), 0x7F, dtype=torch.uint8, device=gu.DEV)      # no clearing needed
    pcpp.pcpp_conv3x3(g, d["x"], d["row_up"], d["row_dn"], d["w"], d["b"], y, ws, wsb)
    torch.cuda.synchronize()
    f = {k: (None if v is None else oracle.from_bf16_bits(v)) for k, v in inp.items()}
    want = oracle.conv3x3_band_mode(f["x"], W, f["w"], f["b"], f["row_up"], f["row_dn"], MODES[mode])
    return gu.to_f64(y), want


def _check(got, want, tag):
    err = np.abs(got - want)
    rms = float(np.sqrt(np.mean(want ** 2)))
    bound = 2.0 ** -8 * np.abs(want) + 2.0 ** -12 * rms
    worst = float((err / bound).max())
    print(f"{tag}: max-abs {err.max():.3e}, worst err/bound {worst:.3f}, mean-abs {err.mean():.3e}")
    assert not np.isnan(got).any()
    assert worst <= 1.0, f"{tag}: max error exceeds bound by {worst:.2f}x"
    assert err.mean() <= 2.0 ** -9 * rms


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{MODES[c[7]]}-H{c[0]}W{c[1]}n{c[2]}i{c[3]}-{c[4]}to{c[5]}-B{c[6]}")
def test_conv3x3_matches_oracle(case):
    _say("conv", case)
    got, want = _run(*case, seed=40 + CASES.index(case))
    _check(got, want, str(case))


@pytest.mark.parametrize("name,cfg", FULL, ids=[k for k, _ in FULL])
def test_sdxl_resolution_change_convs(name, cfg):
    _say("conv", name)
    got, want = _run(*cfg[:6], 1, cfg[6], seed=60)
    _check(got, want, name)


def test_down_ignores_the_row_below():
    import torch
    from paper_2412_02962_amd import pcpp
    _say("down without the row below")
    H, W, n, i, ci, co, B = 16, 20, 4, 1, 64, 64, 1
    inp = synth.conv_inputs(H, W, n, i, ci, co, B, 70)
    d = {k: gu.to_dev(v, "bf16") for k, v in inp.items()}
    g = pcpp.make_conv_geom(H, W, n, i, ci, co, B, pcpp.PCPP_CONV_DOWN)
    wsb = pcpp.pcpp_conv3x3_workspace_size(g)
    ws = torch.zeros(wsb, dtype=torch.uint8, device=gu.DEV)
    outs = []
    for dn in (d["row_dn"], None):
        y = torch.empty((B, (H // n // 2) * (W // 2), co), dtype=torch.bfloat16, device=gu.DEV)
        pcpp.pcpp_conv3x3(g, d["x"], d["row_up"], dn, d["w"], d["b"], y, ws, wsb)
        outs.append(y)
    torch.cuda.synchronize()
    assert torch.equal(outs[0], outs[1])


@pytest.mark.parametrize("mode", [0, 1, 2], ids=["same", "down", "up"])
def test_conv_exports_first_and_last_rows(mode):
    """pcpp_conv3x3_export: the same output as pcpp_conv3x3, and the band's
    first and last input rows (before upsampling) bit for bit."""
    import torch
    from paper_2412_02962_amd import pcpp
    H, W, n, i, ci, co, B = 12, 10, 3, 1, 64, 128, 2
    _say("conv export", mode)
    d = {k: gu.to_dev(v, "bf16") for k, v in synth.conv_inputs(H, W, n, i, ci, co, B, 61).items()}
    g = pcpp.make_conv_geom(H, W, n, i, ci, co, B, mode)
    h = H // n
    tok = {0: h * W, 1: (h // 2) * (W // 2), 2: 4 * h * W}[mode]
    wsb = pcpp.pcpp_conv3x3_workspace_size(g)
    ws = torch.empty(wsb, dtype=torch.uint8, device=gu.DEV)
    y0 = torch.empty((B, tok, co), dtype=torch.bfloat16, device=gu.DEV)
    y1 = torch.empty_like(y0)
    first = torch.empty((B, W, ci), dtype=torch.bfloat16, device=gu.DEV)
    last = torch.empty_like(first)
    pcpp.pcpp_conv3x3(g, d["x"], d["row_up"], d["row_dn"], d["w"], d["b"], y0, ws, wsb)
    pcpp.pcpp_conv3x3_export(g, d["x"], d["row_up"], d["row_dn"], d["w"], d["b"], y1, first, last, ws, wsb)
    torch.cuda.synchronize()
    x = d["x"].view(B, h, W, ci)
    assert torch.equal(y0, y1)
    assert torch.equal(first, x[:, 0]) and torch.equal(last, x[:, h - 1])
