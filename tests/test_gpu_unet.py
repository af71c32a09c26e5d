"""GPU parity of one band's SDXL-shaped U-Net step (paper_2412_02962_amd.unet,
every layer a C-ABI call) against the float64 oracle composition, on a small
U-Net of the same topology and on one of SDXL's widths and depths on a
reduced latent grid, with seeded random weights and stale neighbour data.

Tolerance: element-wise, tests.gpu_util.check_composition with S the
number of bf16 roundings on the way to the output (unet_stages: every
convolution input, three per ResNet, two per module plus six per basic
block, the output head); the padding channels are exactly zero.  The
layers' shared workspace is filled with garbage first: no call may rely on
it being clear.
"""

import dataclasses

import numpy as np
import pytest

import oracle
from paper_2412_02962_amd import synth
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

SPECS = [
    synth.UNET_TINY,                                                   # bottom band of 2
    dataclasses.replace(synth.UNET_TINY, i=0),                         # top band of 2
    dataclasses.replace(synth.UNET_TINY, H0=48, n=3, i=1, seed_id=122),  # middle band of 3
    dataclasses.replace(synth.UNET_TINY, batch=2, seed_id=123),        # two images
]


def _say(*a):
    print("[case]", *a, flush=True)


def _dev_tree(t):
    if t is None:
        return None
    if isinstance(t, np.ndarray):
        if t.dtype == np.float32:       # GroupNorm statistics
            import torch
            return torch.from_numpy(t).to(gu.DEV)
        return gu.to_dev(t, "bf16")
    if isinstance(t, dict):
        return {k: _dev_tree(v) for k, v in t.items()}
    if isinstance(t, (list, tuple)):
        return type(t)(_dev_tree(v) for v in t)
    return t


def unet_stages(layers):
    """bf16 roundings along the U-Net's forward: a convolution rounds its
    input (and output), a ResNet its two convolution inputs and conv1's
    output, a module its GroupNorm output and proj_out's input plus six per
    basic block (three LayerNorm outputs, Q/K/V, two attention outputs,
    the GEGLU state, less the ones that stay float32), the head its
    GroupNorm output."""
    s = 0
    for ly in layers:
        s += {"conv": 1, "resnet": 3, "gn": 1}.get(ly["kind"], 0)
        if ly["kind"] == "module":
            s += 2 + 6 * ly["depth"]
    return s


def _f64_tree(t):
    if t is None:
        return None
    if isinstance(t, np.ndarray):
        return t.astype(np.float64) if t.dtype == np.float32 else oracle.from_bf16_bits(t)
    if isinstance(t, dict):
        return {k: _f64_tree(v) for k, v in t.items()}
    if isinstance(t, (list, tuple)):
        return type(t)(_f64_tree(v) for v in t)
    return t


@pytest.mark.parametrize("sync_gn", [False, True], ids=["local_gn", "sync_gn"])
@pytest.mark.parametrize("sp", SPECS, ids=["n2_i1", "n2_i0", "n3_i1", "n2_i1_b2"])
def test_unet_band_step_matches_oracle(sp, sync_gn):
    import torch
    from paper_2412_02962_amd.unet import BandUNet
    _say("unet", sp, "sync_gn" if sync_gn else "local_gn")
    layers = synth.unet_layers(sp)
    weights, stale, latent, temb, text = synth.unet_band_inputs(sp, sync_gn=sync_gn)
    net = BandUNet(sp, layers, _dev_tree(weights), _dev_tree(stale), sync_gn=sync_gn)
    net.ws.fill_(0xA5)
    got = net.forward(gu.to_dev(latent, "bf16"), gu.to_dev(temb, "bf16"), gu.to_dev(text, "bf16"))
    torch.cuda.synchronize()
    got = gu.to_f64(got)
    want = oracle.unet_band_step(layers, sp.n, sp.i, sp.p, sp.groups, _f64_tree(weights), _f64_tree(stale),
                                 oracle.from_bf16_bits(latent), oracle.from_bf16_bits(temb),
                                 oracle.from_bf16_bits(text), sync_gn=sync_gn)
    assert np.abs(got[..., 4:]).max() == 0.0
    gu.check_composition(got[..., :4], want[..., :4], unet_stages(layers), f"unet {sp.n}/{sp.i} b{sp.batch}")


def _first_rows_as_last(t, W, r):
    """The mistake of reading a band's first r rows where its last r rows
    belong: [B, h*W, C] with rows h-r .. h-1 replaced by rows 0 .. r-1."""
    t = t.copy()
    t[:, t.shape[1] - r * W:] = t[:, :r * W]
    return t


class _LazyF64(dict):
    """A layer-name -> float64 tree mapping that converts one layer's bf16
    data when the oracle reaches it (the SDXL-width weights are 5 GB as bf16,
    20 GB as float64)."""

    def __getitem__(self, k):
        return _f64_tree(dict.__getitem__(self, k))


# SDXL's widths and depths (320 / 640 / 1280 channels, 0 / 2 / 10 basic blocks)
# on a 96 x 128 latent in two bands: a band holds 1536 tokens at level 1 and
# 384 at level 2, so the library takes the same kernel paths as on the 2048 px
# grid in eight bands: the 3x3 convolutions with K = 9 * 640 and 9 * 1280 split
# over 128 x 128 tiles (60 and 30 tiles), the level-2 GEGLU and Q/K/V products
# on XCD-contiguous tile ranges (their weight rows are more than four times the
# tokens), the split FF-out product at level 2 (K = 5120 over 64 x 64 tiles),
# the grouped text K/V product of a depth-10 module, and GroupNorm over the
# 2560 channels of the first level-2 up ResNet.
SDXL_REDUCED = dataclasses.replace(synth.UNET_SDXL_2048, H0=96, W0=128, n=2, i=1, p=0.5, seed_id=124)


def test_unet_band_step_at_sdxl_widths():
    import torch
    from paper_2412_02962_amd.unet import BandUNet
    sp = SDXL_REDUCED
    _say("unet at SDXL widths", sp)
    layers = synth.unet_layers(sp)
    weights, stale, latent, temb, text = synth.unet_band_inputs(sp, sync_gn=True)
    _say("inputs drawn")
    net = BandUNet(sp, layers, _dev_tree(weights), _dev_tree(stale), sync_gn=True)
    net.ws.fill_(0xA5)
    got = net.forward(gu.to_dev(latent, "bf16"), gu.to_dev(temb, "bf16"), gu.to_dev(text, "bf16"))
    torch.cuda.synchronize()
    got = gu.to_f64(got)
    del net
    torch.cuda.empty_cache()
    _say("GPU forward done; oracle")
    want = oracle.unet_band_step(layers, sp.n, sp.i, sp.p, sp.groups, _LazyF64(weights), _LazyF64(stale),
                                 oracle.from_bf16_bits(latent), oracle.from_bf16_bits(temb),
                                 oracle.from_bf16_bits(text), sync_gn=True)
    assert np.abs(got[..., 4:]).max() == 0.0
    gu.check_composition(got[..., :4], want[..., :4], unet_stages(layers), "unet SDXL widths 96x128 n2 i1")
    # Negative control, planted in the oracle: every module reads the first r
    # rows of the band above where its last r rows belong; the same bound
    # rejects that composition.
    _say("oracle with a planted mistake")
    bad = dict(stale)
    for ly in layers:
        if ly["kind"] == "module":
            r = oracle.context_rows(ly["H"], sp.n, sp.i, sp.p)[1]
            bad[ly["name"]] = [(_first_rows_as_last(ku, ly["W"], r), _first_rows_as_last(vu, ly["W"], r), kd, vd)
                               for ku, vu, kd, vd in stale[ly["name"]]]
    want_bad = oracle.unet_band_step(layers, sp.n, sp.i, sp.p, sp.groups, _LazyF64(weights), _LazyF64(bad),
                                     oracle.from_bf16_bits(latent), oracle.from_bf16_bits(temb),
                                     oracle.from_bf16_bits(text), sync_gn=True)
    with pytest.raises(AssertionError):
        gu.check_composition(got[..., :4], want_bad[..., :4], unet_stages(layers), "planted mistake, SDXL widths")


def test_unet_band_step_is_deterministic():
    import torch
    from paper_2412_02962_amd.unet import BandUNet
    sp = synth.UNET_TINY
    _say("unet determinism")
    layers = synth.unet_layers(sp)
    weights, stale, latent, temb, text = synth.unet_band_inputs(sp)
    net = BandUNet(sp, layers, _dev_tree(weights), _dev_tree(stale))
    args = (gu.to_dev(latent, "bf16"), gu.to_dev(temb, "bf16"), gu.to_dev(text, "bf16"))
    ref = net.forward(*args).clone()
    for _ in range(2):
        assert torch.equal(net.forward(*args), ref)


def test_unet_bound_rejects_a_planted_mistake():
    """Negative control, planted in the oracle on the CPU: every attention
    reads the first r rows of the band above where its last r rows belong
    (an indexing mistake in the stale context).  That oracle is further from
    the GPU result than the bound allows."""
    import torch
    from paper_2412_02962_amd.unet import BandUNet
    sp = synth.UNET_TINY                                  # bottom band: only a band above
    _say("unet negative control")
    layers = synth.unet_layers(sp)
    weights, stale, latent, temb, text = synth.unet_band_inputs(sp)
    net = BandUNet(sp, layers, _dev_tree(weights), _dev_tree(stale))
    got = gu.to_f64(net.forward(gu.to_dev(latent, "bf16"), gu.to_dev(temb, "bf16"), gu.to_dev(text, "bf16")))
    torch.cuda.synchronize()
    fs = _f64_tree(stale)
    for ly in layers:
        if ly["kind"] == "module":
            r = oracle.context_rows(ly["H"], sp.n, sp.i, sp.p)[1]
            fs[ly["name"]] = [(_first_rows_as_last(ku, ly["W"], r), _first_rows_as_last(vu, ly["W"], r), kd, vd)
                              for ku, vu, kd, vd in fs[ly["name"]]]
    want_bad = oracle.unet_band_step(layers, sp.n, sp.i, sp.p, sp.groups, _f64_tree(weights), fs,
                                     oracle.from_bf16_bits(latent), oracle.from_bf16_bits(temb),
                                     oracle.from_bf16_bits(text))
    with pytest.raises(AssertionError):
        gu.check_composition(got[..., :4], want_bad[..., :4], unet_stages(layers), "planted mistake")
