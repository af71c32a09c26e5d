"""GPU parity of pcpp_resnet_block and pcpp_guided_step against the float64
oracle, through the C ABI.

ResNet tolerance: the library stores the two convolution inputs (GroupNorm
then SiLU) and conv1's output in bf16, computes the second GroupNorm's
statistics from that bf16 output, keeps the shortcut in float32 and rounds
y to bf16.  Each rounding is a relative error of at most 2^-8 of its tensor,
so the bound is |dy| <= 2^-8 |y| + 4 * 2^-8 * rms(y) per element, with a
mean absolute error below 2^-8 * rms(y).  The exported edge rows are SiLU
of GroupNorm outputs and sit behind one rounding (the first) or three (the
second).  Their errors scale with the GroupNorm output, whose rms is
sqrt(mean(gamma^2) + mean(beta^2)), times SiLU's slope (at most 1.1), not
with the smaller rms of the SiLU output, so that product stands for rms in
their bound.  The rounding of conv1's output h1 (2^-9 |h1| at most) enters
the second GroupNorm divided by its group's standard deviation and scaled
by gamma, then by SiLU's slope, so for the second edge rows that stage is
the per-element term 2^-9 |h1| / std_group |gamma| 1.1 instead of a share
of the rms: it grows where a group's values sit far from zero compared with
their spread (few tokens per group, a large per-channel bias).

Latent update tolerance: float32 arithmetic on float32 inputs, with the two
coefficients rounded to float32: |d| <= 2^-20 (|a x| + |b| |e| + |sigma z|)
per element, e being the guided noise.
"""

import dataclasses
import math

import numpy as np
import pytest

import oracle
from paper_2412_02962_amd import synth
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

SMALL = [
    synth.ResnetConfig("r_mid", 12, 20, 3, 1, 64, 128, temb_dim=64, groups=8, batch=2, seed_id=82),
    synth.ResnetConfig("r_top", 12, 20, 3, 0, 64, 128, temb_dim=64, groups=8, batch=2, seed_id=83),
    synth.ResnetConfig("r_bot", 12, 20, 3, 2, 128, 128, temb_dim=64, groups=8, batch=1, seed_id=84),
    synth.ResnetConfig("r_one", 8, 24, 1, 0, 128, 64, temb_dim=128, groups=32, batch=1, seed_id=85),
    synth.ResnetConfig("r_tiny", 4, 3, 2, 1, 64, 64, temb_dim=8, groups=32, batch=3, seed_id=86),
    # conv1 (K = 9 * 1024) splits K eight ways over 32 tiles: the whole device
    synth.ResnetConfig("r_split", 32, 128, 2, 1, 1024, 256, temb_dim=64, groups=32, batch=1, seed_id=88),
]
FULL = [synth.RESNET_CONFIGS["sdxl2048_l1_res640"], synth.RESNET_CONFIGS["sdxl2048_l1_res320_640"],
        synth.RESNET_CONFIGS["sdxl2048_l0_res320"], synth.RESNET_CONFIGS["sdxl2048_l2_res1280"],
        synth.RESNET_CONFIGS["sdxl2048_l2_res640_1280"], synth.RESNET_CONFIGS["sdxl2048_l2_res2560_1280"],
        synth.RESNET_CONFIGS["sdxl2048_l1_res1920_640"], synth.RESNET_CONFIGS["sdxl2048_l0_res960_320"]]


def _say(*a):
    print("[case]", *a, flush=True)


def _check(got, want, stages, tag, scale=None, extra=0.0):
    err = np.abs(got - want)
    rms = float(np.sqrt(np.mean(want ** 2))) if scale is None else scale
    bound = 2.0 ** -8 * np.abs(want) + stages * 2.0 ** -8 * rms + extra
    worst = float((err / bound).max())
    mean = float(err.mean())
    print(f"{tag}: max-abs {err.max():.3e}, worst err/bound {worst:.3f}, mean-abs {mean:.3e}, rms {rms:.3f}")
    assert worst <= 1.0, f"{tag}: max error exceeds bound by {worst:.2f}x"
    assert mean <= 2.0 ** -8 * rms, f"{tag}: mean-abs {mean:.3e} > {2.0 ** -8 * rms:.3e}"


def _geom(rc, i=None):
    from paper_2412_02962_amd import pcpp
    return pcpp.make_resnet_geom(rc.H, rc.W, rc.n, rc.i if i is None else i, rc.c_in, rc.c_out, rc.temb_dim,
                                 rc.groups, rc.batch, 1e-5)


def _run(rc, d, i=None, edges=None, gn1_bands=None, gn2_bands=None, want_own=False):
    """One call on band i; d holds device tensors.  Returns (y, e1, e2, own1, own2)."""
    import torch
    from paper_2412_02962_amd import pcpp
    g = _geom(rc, i)
    w = pcpp.make_resnet_weights(d)
    B, h, W = rc.batch, rc.h, rc.W
    y = torch.empty((B, h * W, rc.c_out), dtype=torch.bfloat16, device=gu.DEV)
    e1 = torch.empty((B, 2, W, rc.c_in), dtype=torch.bfloat16, device=gu.DEV)
    e2 = torch.empty((B, 2, W, rc.c_out), dtype=torch.bfloat16, device=gu.DEV)
    own1 = torch.empty((B, rc.groups, 3), dtype=torch.float32, device=gu.DEV) if want_own else None
    own2 = torch.empty((B, rc.groups, 3), dtype=torch.float32, device=gu.DEV) if want_own else None
    ed = edges if edges is not None else {k: d.get(k) for k in ("edges1_up", "edges1_dn", "edges2_up", "edges2_dn")}
    wsb = pcpp.pcpp_resnet_block_workspace_size(g)
    assert wsb > 0
    ws = torch.empty(wsb, dtype=torch.uint8, device=gu.DEV)
    pcpp.pcpp_resnet_block(g, w, d["x"], d["temb"], ed["edges1_up"], ed["edges1_dn"], ed["edges2_up"],
                           ed["edges2_dn"], gn1_bands, own1, gn2_bands, own2, y, e1, e2, ws, wsb)
    torch.cuda.synchronize()
    return y, e1, e2, own1, own2


def _oracle(rc, inp, **kw):
    f = {k: (None if v is None else oracle.from_bf16_bits(v)) for k, v in inp.items()}
    wts = {k: f[k] for k in synth.resnet_weight_shapes(rc)}
    return oracle.resnet_block(rc.W, wts, f["x"], f["temb"], f["edges1_up"], f["edges1_dn"], f["edges2_up"],
                               f["edges2_dn"], groups=rc.groups, i=rc.i, **kw)


@pytest.mark.parametrize("rc", SMALL + FULL, ids=lambda r: r.name)
def test_resnet_matches_oracle(rc):
    _say("resnet", rc)
    inp = synth.resnet_inputs(rc)
    d = {k: gu.to_dev(v, "bf16") for k, v in inp.items()}
    y, e1, e2, _, _ = _run(rc, d)
    want, w1, w2 = _oracle(rc, inp)
    _check(gu.to_f64(y), want, 4, f"resnet {rc.name}")
    _check(gu.to_f64(e1), w1, 1, f"edges1 {rc.name}", _silu_gn_scale(inp, "gn1"))
    _check(gu.to_f64(e2), w2, 2, f"edges2 {rc.name}", _silu_gn_scale(inp, "gn2"), _h1_rounding_term(rc, inp))


def _h1_rounding_term(rc, inp):
    """2^-9 |h1| / std_group |gamma2| 1.1 at the band's first and last rows,
    [B, 2, W, C_out], h1 being conv1's output (with the time embedding)."""
    f = {k: (None if v is None else oracle.from_bf16_bits(v)) for k, v in inp.items()}
    a1 = oracle.silu(oracle.group_norm(f["x"], rc.groups, f["gn1_gamma"], f["gn1_beta"], eps=1e-5))
    h1 = oracle.conv3x3_band(a1, rc.W, f["conv1_w"], f["conv1_b"],
                             None if f["edges1_up"] is None else f["edges1_up"][:, 1],
                             None if f["edges1_dn"] is None else f["edges1_dn"][:, 0])
    h1 = h1 + oracle.linear(oracle.silu(f["temb"]), f["temb_w"], f["temb_b"])[:, None, :]
    cg = rc.c_out // rc.groups
    std = np.empty((rc.batch, rc.c_out))
    for b in range(rc.batch):
        for g in range(rc.groups):
            std[b, g * cg:(g + 1) * cg] = h1[b, :, g * cg:(g + 1) * cg].std()
    rows = h1.reshape(rc.batch, rc.h, rc.W, rc.c_out)[:, [0, rc.h - 1]]
    return 2.0 ** -9 * np.abs(rows) / std[:, None, None, :] * np.abs(f["gn2_gamma"]) * 1.1


def _silu_gn_scale(inp, which):
    g = oracle.from_bf16_bits(inp[which + "_gamma"])
    b = oracle.from_bf16_bits(inp[which + "_beta"])
    return 1.1 * float(np.sqrt(np.mean(g ** 2) + np.mean(b ** 2)))


def _other_band_stats(rc, G, C, seed):
    """[n, B, G, 3] (count, mean, M2) of synthetic GroupNorm inputs of every band."""
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(rc.n):
        t = 0.2 * rng.standard_normal() + (1.0 + 0.3 * rng.random()) * rng.standard_normal((rc.batch, rc.h * rc.W, C))
        out.append(oracle.group_stats(t, G))
    return np.stack(out)


# FULL[2] (8192 tokens of 320 channels) applies 32 tokens per workgroup
@pytest.mark.parametrize("rc", [SMALL[0], SMALL[2], FULL[1], FULL[2]], ids=lambda r: r.name)
def test_resnet_synchronized_group_norm(rc):
    import torch
    _say("resnet sync GN", rc)
    inp = synth.resnet_inputs(rc)
    d = {k: gu.to_dev(v, "bf16") for k, v in inp.items()}
    st1 = _other_band_stats(rc, rc.groups, rc.c_in, 1)
    st2 = _other_band_stats(rc, rc.groups, rc.c_out, 2)
    b1 = torch.from_numpy(st1.astype(np.float32)).to(gu.DEV)
    b2 = torch.from_numpy(st2.astype(np.float32)).to(gu.DEV)
    y, _, _, own1, _ = _run(rc, d, gn1_bands=b1, gn2_bands=b2, want_own=True)
    want, _, _ = _oracle(rc, inp, gn1_band_stats=st1, gn2_band_stats=st2)
    _check(gu.to_f64(y), want, 4, f"resnet sync {rc.name}")
    want_own = oracle.group_stats(oracle.from_bf16_bits(inp["x"]), rc.groups)
    got_own = own1.double().cpu().numpy()
    assert np.array_equal(got_own[..., 0], want_own[..., 0])
    assert np.allclose(got_own[..., 1], want_own[..., 1], rtol=0, atol=1e-5)
    assert np.allclose(got_own[..., 2], want_own[..., 2], rtol=1e-4, atol=0)


@pytest.mark.parametrize("n", [3, 4])
def test_bands_exchanging_edges_and_statistics_rebuild_the_whole_image(n):
    """Every band runs on the GPU, each pass taking the previous pass's
    exported edge rows and GroupNorm statistics of the other bands (stale =
    fresh: the input does not change between passes).  Five passes carry the
    exact values through both GroupNorms and both convolutions; the result
    is then the whole image's ResNet block, computed by the oracle with one
    band."""
    import torch
    rc = synth.ResnetConfig("chain", 4 * n, 12, n, 0, 64, 128, temb_dim=64, groups=8, batch=2, seed_id=87)
    whole = dataclasses.replace(rc, H=rc.H, n=1, i=0)
    _say("exchange chain", n)
    inp_whole = synth.resnet_inputs(whole)      # the whole image's x and the shared weights
    want, _, _ = _oracle(whole, inp_whole)
    d_w = {k: gu.to_dev(v, "bf16") for k, v in inp_whole.items() if v is not None}
    x_all = d_w["x"].view(rc.batch, rc.n, rc.h * rc.W, rc.c_in)
    B = rc.batch
    zeros1 = torch.zeros((B, 2, rc.W, rc.c_in), dtype=torch.bfloat16, device=gu.DEV)
    zeros2 = torch.zeros((B, 2, rc.W, rc.c_out), dtype=torch.bfloat16, device=gu.DEV)
    exp1, exp2 = [zeros1] * n, [zeros2] * n
    st1 = torch.zeros((n, B, rc.groups, 3), dtype=torch.float32, device=gu.DEV)
    st2 = torch.zeros((n, B, rc.groups, 3), dtype=torch.float32, device=gu.DEV)
    st1[..., 0] = 1.0
    st2[..., 0] = 1.0
    for _ in range(5):
        outs = []
        new1, new2, own1s, own2s = [], [], [], []
        for i in range(n):
            d = dict(d_w)
            d["x"] = x_all[:, i].contiguous()
            edges = {"edges1_up": exp1[i - 1] if i > 0 else None, "edges1_dn": exp1[i + 1] if i < n - 1 else None,
                     "edges2_up": exp2[i - 1] if i > 0 else None, "edges2_dn": exp2[i + 1] if i < n - 1 else None}
            y, e1, e2, o1, o2 = _run(rc, d, i=i, edges=edges, gn1_bands=st1, gn2_bands=st2, want_own=True)
            outs.append(y)
            new1.append(e1)
            new2.append(e2)
            own1s.append(o1)
            own2s.append(o2)
        exp1, exp2 = new1, new2
        st1 = torch.stack(own1s)
        st2 = torch.stack(own2s)
    got = torch.cat(outs, dim=1)                  # bands in order = the whole image's tokens
    _check(gu.to_f64(got), want, 4, f"exchange chain n={n}")


@pytest.mark.parametrize("rc", [SMALL[5], FULL[0]], ids=lambda r: r.name)
def test_resnet_is_deterministic(rc):
    """The split convolutions add their pieces in a fixed order: repeated
    calls give the same bits."""
    import torch
    _say("resnet determinism", rc.name)
    inp = synth.resnet_inputs(rc)
    d = {k: gu.to_dev(v, "bf16") for k, v in inp.items()}
    ref = _run(rc, d)[0]
    for _ in range(3):
        assert torch.equal(_run(rc, d)[0], ref)


def test_resnet_workspace_needs_no_clearing():
    import torch
    from paper_2412_02962_amd import pcpp
    rc = SMALL[0]
    _say("resnet dirty workspace")
    inp = synth.resnet_inputs(rc)
    d = {k: gu.to_dev(v, "bf16") for k, v in inp.items()}
    ref = _run(rc, d)[0]
    g = _geom(rc)
    wsb = pcpp.pcpp_resnet_block_workspace_size(g)
    ws = torch.full((wsb,), 0x7F, dtype=torch.uint8, device=gu.DEV)     # NaN-like bf16 garbage everywhere
    y = torch.empty_like(ref)
    pcpp.pcpp_resnet_block(g, pcpp.make_resnet_weights(d), d["x"], d["temb"], d["edges1_up"], d["edges1_dn"],
                           d["edges2_up"], d["edges2_dn"], None, None, None, None, y, None, None, ws, wsb)
    torch.cuda.synchronize()
    assert torch.equal(y, ref)


# ---------------------------------------------------------------------------
# pcpp_guided_step
# ---------------------------------------------------------------------------

def _coef(mode, p):
    if mode == "ddpm":
        return 1 / math.sqrt(p["alpha_t"]), -(1 - p["alpha_t"]) / (math.sqrt(1 - p["alphabar_t"]) * math.sqrt(p["alpha_t"]))
    return (math.sqrt(p["alphabar_prev"] / p["alphabar_t"]),
            math.sqrt(1 - p["alphabar_prev"]) - math.sqrt(p["alphabar_prev"] * (1 - p["alphabar_t"]) / p["alphabar_t"]))


@pytest.mark.parametrize("mode,t,prev,noise", [("ddpm", 999, 998, True), ("ddpm", 500, 499, False),
                                               ("ddpm", 1, 0, True), ("ddim", 999, 979, False),
                                               ("ddim", 21, 1, False), ("ddim", 500, 500, False)])
@pytest.mark.parametrize("n,offset", [(32768, 0), (1001, 1), (4, 0)])
def test_guided_step_matches_oracle(mode, t, prev, noise, n, offset):
    import torch
    from paper_2412_02962_amd import pcpp
    _say("guided step", mode, t, prev, noise, n, offset)
    abar = oracle.scaled_linear_alphabar()
    alpha_t = float(abar[t] / abar[t - 1]) if t > 0 else float(abar[0])
    p = dict(alpha_t=np.float32(alpha_t).item(), alphabar_t=np.float32(abar[t]).item(),
             alphabar_prev=np.float32(abar[prev]).item(), sigma_t=np.float32(0.37).item())
    s = 5.0
    inp = synth.step_inputs(n, seed=31 + t, with_noise=noise)
    dev = {}
    for k, v in inp.items():   # an element offset makes the pointers unaligned
        dev[k] = None if v is None else torch.from_numpy(np.concatenate([np.zeros(offset, np.float32), v])).to(gu.DEV)[offset:]
    out = torch.full_like(dev["x_t"], float("nan"))
    if mode == "ddpm":
        sp = pcpp.make_step_params(pcpp.PCPP_STEP_DDPM, s, alpha_t=p["alpha_t"], alphabar_t=p["alphabar_t"],
                                   sigma_t=p["sigma_t"])
    else:
        sp = pcpp.make_step_params(pcpp.PCPP_STEP_DDIM, s, alphabar_t=p["alphabar_t"], alphabar_prev=p["alphabar_prev"])
    pcpp.pcpp_guided_step(sp, n, dev["x_t"], dev["eps_uncond"], dev["eps_cond"], dev["z"], out)
    # in place as well
    xin = dev["x_t"].clone()
    pcpp.pcpp_guided_step(sp, n, xin, dev["eps_uncond"], dev["eps_cond"], dev["z"], xin)
    torch.cuda.synchronize()
    f = {k: (None if v is None else v.astype(np.float64)) for k, v in inp.items()}
    if mode == "ddpm":
        want = oracle.reverse_step_ddpm(f["x_t"], f["eps_uncond"], f["eps_cond"], s, p["alpha_t"], p["alphabar_t"],
                                        p["sigma_t"], f["z"])
    else:
        want = oracle.reverse_step_ddim(f["x_t"], f["eps_uncond"], f["eps_cond"], s, p["alphabar_t"],
                                        p["alphabar_prev"])
    a, b = _coef(mode, p)
    e = oracle.guided_noise(f["eps_uncond"], f["eps_cond"], s)
    scale = np.abs(a * f["x_t"]) + abs(b) * (np.abs(f["eps_uncond"]) + s * np.abs(f["eps_cond"] - f["eps_uncond"]))
    if mode == "ddpm" and f["z"] is not None:
        scale = scale + abs(p["sigma_t"] * f["z"])
    bound = 2.0 ** -20 * (scale + np.abs(b * e)) + 1e-30
    for got in (out, xin):
        err = np.abs(got.double().cpu().numpy() - want)
        assert (err <= bound).all(), f"worst err/bound {(err / bound).max():.2f}"
