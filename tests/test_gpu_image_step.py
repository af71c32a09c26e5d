"""GPU parity of whole-image PCPP steps on one device (ImageStep: every band's
U-Net forward, each with its neighbours' exports of the previous step)
against the float64 oracle's image step, over consecutive steps on a small
U-Net of the SDXL topology.

Tolerance: element-wise, tests.gpu_util.check_composition.  The first step
(the bands computed separately) is one band step per band, S =
unet_stages(layers).  From the second step on, the stale inputs are the
GPU's own bf16 exports of the previous step, whose errors (from the same
number of roundings, independent of this step's) enter each band through
the exchange: S doubles.
"""

import dataclasses

import numpy as np
import pytest

import oracle
from oracle import unet_oracle as uo
from paper_2412_02962_amd import synth
from tests import gpu_util as gu
from tests.test_gpu_unet import _dev_tree, _f64_tree, unet_stages

pytestmark = pytest.mark.gpu

CASES = [
    (dataclasses.replace(synth.UNET_TINY, n=2, i=0, p=0.5), True, 3),
    (dataclasses.replace(synth.UNET_TINY, H0=48, n=3, i=0, p=0.5, seed_id=124), True, 2),
    (dataclasses.replace(synth.UNET_TINY, n=2, i=0, p=1.0, batch=2, seed_id=125), False, 2),
]


def _say(*a):
    print("[case]", *a, flush=True)


@pytest.mark.parametrize("case", CASES, ids=["n2_p05_sync_3steps", "n3_p05_sync", "n2_p1_local_b2"])
def test_image_steps_match_oracle(case):
    import torch
    from paper_2412_02962_amd.image_step import ImageStep
    sp, sync_gn, steps = case
    _say("image step", sp.n, sp.p, sp.batch, sync_gn, steps)
    layers = synth.unet_layers(sp)
    weights, _, latent, temb, text = synth.unet_band_inputs(dataclasses.replace(sp, n=1, i=0))
    h0 = sp.H0 // sp.n
    tok = h0 * sp.W0
    lat_f = oracle.from_bf16_bits(latent)
    lat_d = gu.to_dev(latent, "bf16")
    bands_f = [lat_f[:, i * tok:(i + 1) * tok] for i in range(sp.n)]
    bands_d = [lat_d[:, i * tok:(i + 1) * tok].contiguous() for i in range(sp.n)]
    fw = _f64_tree(weights)
    net = ImageStep(sp, layers, _dev_tree(weights), gu.DEV, sync_gn=sync_gn)
    temb_d, text_d = gu.to_dev(temb, "bf16"), gu.to_dev(text, "bf16")
    prev = None
    for t in range(steps):
        want, prev = uo.image_step(layers, sp.n, sp.p, sp.groups, fw, prev, bands_f, oracle.from_bf16_bits(temb),
                                   oracle.from_bf16_bits(text), sync_gn=sync_gn)
        got = net.step(bands_d, temb_d, text_d)
        torch.cuda.synchronize()
        stages = unet_stages(layers) * (1 if t == 0 else 2)
        for i in range(sp.n):
            g = gu.to_f64(got[i])
            gu.check_composition(g[..., :4], want[i][..., :4], stages, f"step {t} band {i}")
            assert np.abs(g[..., 4:]).max() == 0.0


def test_image_steps_settle_on_the_whole_image_unet():
    """On constant inputs the exchange hands every band the neighbours' data
    of the step before; once those stop changing they equal the fresh data.
    With n = 2, p = 1 and synchronized GroupNorm the bands then compute the
    whole-image U-Net (the oracle's pin U8).  After 100 steps the bands'
    outputs, side by side, must match the oracle's whole-image forward (its
    band step with n = 1) within one band step's bound, while the first step
    (the bands computed separately) must not."""
    import torch
    from paper_2412_02962_amd.image_step import ImageStep
    sp = dataclasses.replace(synth.UNET_TINY, n=2, i=0, H0=16, W0=8, p=1.0)
    sp1 = dataclasses.replace(sp, n=1)
    _say("image steps settle", sp.n, sp.p)
    layers = synth.unet_layers(sp)
    weights, stale1, latent, temb, text = synth.unet_band_inputs(sp1, sync_gn=True)
    want = oracle.unet_band_step(layers, 1, 0, sp.p, sp.groups, _f64_tree(weights), _f64_tree(stale1),
                                 oracle.from_bf16_bits(latent), oracle.from_bf16_bits(temb),
                                 oracle.from_bf16_bits(text))[..., :4]
    wd = _dev_tree(weights)
    temb_d, text_d, lat_d = gu.to_dev(temb, "bf16"), gu.to_dev(text, "bf16"), gu.to_dev(latent, "bf16")
    tok = (sp.H0 // sp.n) * sp.W0
    bands = [lat_d[:, i * tok:(i + 1) * tok].contiguous() for i in range(sp.n)]
    net = ImageStep(sp, layers, wd, gu.DEV, sync_gn=True)
    got = {}
    for t in range(100):  # the oracle's image step reaches its fixed point after 93 here
        outs = net.step(bands, temb_d, text_d)
        if t in (0, 99):
            got[t] = np.concatenate([gu.to_f64(o) for o in outs], axis=1)[..., :4]
    torch.cuda.synchronize()
    gu.check_composition(got[99], want, unet_stages(layers), "after 100 steps")
    with pytest.raises(AssertionError):
        gu.check_composition(got[0], want, unet_stages(layers), "first step")
