"""Pins of the oracle's per-band U-Net step pieces (unet_oracle), CPU only.

  U1  conv3x3_band of every band, given the true neighbour rows as its halo,
      reproduces torch's conv2d (padding 1, NCHW) of the whole image
  U2  with n = 1 the ResNet block equals a composition of torch's
      group_norm, silu, conv2d and linear on the whole image (NCHW)
  U3  every band's ResNet block, given the true neighbour edge rows and the
      true per-band statistics (synchronized GroupNorm), reproduces the
      whole image's block, and its edge exports are the whole image's rows
  U4  Eq. 3 with the true noise equals the DDPM posterior mean written from
      x0 and x_t (a different closed form); DDIM with the true noise moves
      x_t exactly to the previous noise level; Eq. 2 at s = 0 / 1 gives the
      unconditional / conditional prediction
  U5  planted mistakes (tap order, halo sides, temb SiLU, shortcut, Eq. 3
      coefficient, DDIM re-noising, stride-2 grid, upsampled grid) fail the pins
  U6  the stride-2 (downsampling) and nearest-2x-then-conv (upsampling)
      convolutions of every band, given the true neighbour rows, reproduce
      torch's whole-image conv2d (stride 2) and interpolate + conv2d; the
      stride-2 band never reads the row below
"""

import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import oracle.unet_oracle as uo


def _torch_conv(img, w, b):
    """img [B, H, W, C] -> [B, H, W, C_out] by torch conv2d (padding 1); w [Co, 3, 3, Ci]."""
    x = torch.from_numpy(img).permute(0, 3, 1, 2)
    k = torch.from_numpy(np.ascontiguousarray(w.transpose(0, 3, 1, 2)))
    y = F.conv2d(x, k, None if b is None else torch.from_numpy(b), padding=1)
    return y.permute(0, 2, 3, 1).numpy()


def _bands(img, n):
    B, H, W, C = img.shape
    h = H // n
    return [img[:, j * h:(j + 1) * h].reshape(B, h * W, C) for j in range(n)]


@pytest.mark.parametrize("B,H,W,ci,co,n", [(1, 12, 7, 3, 5, 3), (2, 8, 5, 4, 4, 4), (1, 6, 9, 2, 3, 1),
                                           (1, 10, 4, 5, 2, 5)])
def test_u1_band_conv_with_true_halos_is_the_whole_image_conv(B, H, W, ci, co, n):
    rng = np.random.default_rng(1)
    img = rng.standard_normal((B, H, W, ci))
    w = rng.standard_normal((co, 3, 3, ci))
    b = rng.standard_normal(co)
    want = _torch_conv(img, w, b)
    h = H // n
    for i, xb in enumerate(_bands(img, n)):
        up = img[:, i * h - 1] if i > 0 else None
        dn = img[:, (i + 1) * h] if i < n - 1 else None
        got = uo.conv3x3_band(xb, W, w, b, up, dn)
        assert np.allclose(got.reshape(B, h, W, co), want[:, i * h:(i + 1) * h], rtol=1e-12, atol=1e-12), i


def _wts(ci, co, T, seed=2):
    rng = np.random.default_rng(seed)
    out = {}
    for k, shp in uo.resnet_weight_shapes(ci, co, T).items():
        if k.endswith("gamma"):
            out[k] = 1.0 + 0.1 * rng.standard_normal(shp)
        elif k.endswith("_w"):
            out[k] = rng.standard_normal(shp) / math.sqrt(np.prod(shp[1:]))
        else:
            out[k] = 0.1 * rng.standard_normal(shp)
    return out


def _torch_resnet(img, temb, wts, groups):
    """Whole image [B, H, W, Ci] -> [B, H, W, Co] by torch ops in NCHW."""
    x = torch.from_numpy(img).permute(0, 3, 1, 2)
    t = {k: torch.from_numpy(np.ascontiguousarray(v)) for k, v in wts.items()}
    k1 = t["conv1_w"].permute(0, 3, 1, 2)
    k2 = t["conv2_w"].permute(0, 3, 1, 2)
    a1 = F.silu(F.group_norm(x, groups, t["gn1_gamma"], t["gn1_beta"], eps=1e-5))
    hid = F.conv2d(a1, k1, t["conv1_b"], padding=1)
    hid = hid + F.linear(F.silu(torch.from_numpy(temb)), t["temb_w"], t["temb_b"])[:, :, None, None]
    a2 = F.silu(F.group_norm(hid, groups, t["gn2_gamma"], t["gn2_beta"], eps=1e-5))
    hid = F.conv2d(a2, k2, t["conv2_b"], padding=1)
    skip = x if "skip_w" not in t else F.conv2d(x, t["skip_w"][:, :, None, None], t["skip_b"])
    return (skip + hid).permute(0, 2, 3, 1).numpy(), a1.permute(0, 2, 3, 1).numpy(), a2.permute(0, 2, 3, 1).numpy()


@pytest.mark.parametrize("ci,co", [(8, 8), (8, 12)])
def test_u2_whole_image_resnet_is_torchs(ci, co):
    B, H, W, T, G = 2, 6, 5, 7, 4
    rng = np.random.default_rng(3)
    img = rng.standard_normal((B, H, W, ci))
    temb = rng.standard_normal((B, T))
    wts = _wts(ci, co, T)
    want, _, _ = _torch_resnet(img, temb, wts, G)
    got, e1, e2 = uo.resnet_block(W, wts, img.reshape(B, H * W, ci), temb, None, None, None, None, groups=G)
    assert np.allclose(got.reshape(B, H, W, co), want, rtol=1e-11, atol=1e-11)
    assert e1.shape == (B, 2, W, ci) and e2.shape == (B, 2, W, co)


@pytest.mark.parametrize("n,ci,co", [(4, 8, 8), (3, 8, 12), (2, 4, 4)])
def test_u3_bands_with_true_edges_and_statistics_rebuild_the_whole_block(n, ci, co):
    B, h, W, T, G = 2, 3, 5, 6, 4
    H = n * h
    rng = np.random.default_rng(4)
    img = rng.standard_normal((B, H, W, ci))
    temb = rng.standard_normal((B, T))
    wts = _wts(ci, co, T)
    want, a1, a2 = _torch_resnet(img, temb, wts, G)
    # true per-band statistics of both GroupNorm inputs (x, and conv1's output)
    xs = _bands(img, n)
    st1 = np.stack([oracle.group_stats(xb, G) for xb in xs])
    hid_img = uo.conv3x3_band(a1.reshape(B, H * W, ci), W, wts["conv1_w"], wts["conv1_b"], None, None)
    hid_img = hid_img + oracle.linear(uo.silu(temb), wts["temb_w"], wts["temb_b"])[:, None, :]
    st2 = np.stack([oracle.group_stats(hb, G) for hb in _bands(hid_img.reshape(B, H, W, co), n)])
    edges1 = [uo.edge_rows(b_, W) for b_ in _bands(a1, n)]
    edges2 = [uo.edge_rows(b_, W) for b_ in _bands(a2, n)]
    for i in range(n):
        y, e1, e2 = uo.resnet_block(W, wts, xs[i], temb,
                                    edges1[i - 1] if i > 0 else None, edges1[i + 1] if i < n - 1 else None,
                                    edges2[i - 1] if i > 0 else None, edges2[i + 1] if i < n - 1 else None,
                                    groups=G, i=i, gn1_band_stats=st1, gn2_band_stats=st2)
        assert np.allclose(y.reshape(B, h, W, co), want[:, i * h:(i + 1) * h], rtol=1e-10, atol=1e-10), i
        assert np.allclose(e1[:, 0], a1[:, i * h]) and np.allclose(e1[:, 1], a1[:, (i + 1) * h - 1])
        assert np.allclose(e2[:, 0], a2[:, i * h]) and np.allclose(e2[:, 1], a2[:, (i + 1) * h - 1])


def test_u4_reverse_steps_against_closed_forms():
    rng = np.random.default_rng(5)
    x0 = rng.standard_normal((2, 24, 4))
    eps = rng.standard_normal((2, 24, 4))
    other = rng.standard_normal((2, 24, 4))
    abar = oracle.scaled_linear_alphabar()
    for t in (999, 500, 20, 1):
        a_t = abar[t] / abar[t - 1]
        x_t = math.sqrt(abar[t]) * x0 + math.sqrt(1 - abar[t]) * eps
        # Eq. 2 at s = 1 is the conditional prediction: here the true noise
        mu = uo.reverse_step_ddpm(x_t, other, eps, 1.0, a_t, abar[t], 0.0, None)
        beta = 1 - a_t
        post = (math.sqrt(abar[t - 1]) * beta / (1 - abar[t])) * x0 + \
               (math.sqrt(a_t) * (1 - abar[t - 1]) / (1 - abar[t])) * x_t
        assert np.allclose(mu, post, rtol=1e-9, atol=1e-9), t
        z = rng.standard_normal(x0.shape)
        assert np.allclose(uo.reverse_step_ddpm(x_t, other, eps, 1.0, a_t, abar[t], 0.3, z), post + 0.3 * z,
                           rtol=1e-9, atol=1e-9)
        # s = 0: the unconditional prediction decides
        assert np.allclose(uo.reverse_step_ddpm(x_t, eps, other, 0.0, a_t, abar[t], 0.0, None), post,
                           rtol=1e-9, atol=1e-9)
        for prev in (t - 1, max(t - 20, 0)):
            got = uo.reverse_step_ddim(x_t, other, eps, 1.0, abar[t], abar[prev])
            want = math.sqrt(abar[prev]) * x0 + math.sqrt(1 - abar[prev]) * eps
            assert np.allclose(got, want, rtol=1e-9, atol=1e-9), (t, prev)
        assert np.allclose(uo.reverse_step_ddim(x_t, eps, other, 0.0, abar[t], abar[t]), x_t, rtol=1e-12, atol=1e-12)
    # guidance at s = 5 (the scale the paper uses) is an affine combination
    e = uo.guided_noise(other, eps, 5.0)
    assert np.allclose(e, -4.0 * other + 5.0 * eps)


def test_u4_scaled_linear_schedule_endpoints():
    abar = oracle.scaled_linear_alphabar(1000, 0.00085, 0.012)
    betas = 1 - abar / np.concatenate([[1.0], abar[:-1]])
    assert abs(betas[0] - 0.00085) < 1e-15 and abs(betas[-1] - 0.012) < 1e-12
    d = np.diff(np.sqrt(betas))
    assert np.allclose(d, d[0], rtol=1e-9) and (np.diff(abar) < 0).all()


# ---------------------------------------------------------------------------
# U5 planted mistakes
# ---------------------------------------------------------------------------

def _battery():
    try:
        test_u1_band_conv_with_true_halos_is_the_whole_image_conv(1, 12, 7, 3, 5, 3)
        test_u2_whole_image_resnet_is_torchs(8, 12)
        test_u2_whole_image_resnet_is_torchs(8, 8)
        test_u3_bands_with_true_edges_and_statistics_rebuild_the_whole_block(3, 8, 12)
        test_u4_reverse_steps_against_closed_forms()
        test_u6_band_downsample_is_the_whole_image_stride2_conv(1, 12, 8, 3, 5, 3)
        test_u6_band_upsample_is_the_whole_image_nearest_then_conv(1, 6, 4, 3, 5, 3)
    except AssertionError:
        return False
    return True


def test_u5_unmodified_oracle_passes():
    assert _battery()


_ORIG = {k: getattr(uo, k) for k in ("conv3x3_band", "pad_band", "silu", "linear", "reverse_step_ddpm",
                                      "reverse_step_ddim", "edge_rows", "conv3x3_band_mode")}


def _down_grid_shifted(x, W, w, b, up, dn, mode):      # stride-2 grid one input row lower
    if mode != "down":
        return _ORIG["conv3x3_band_mode"](x, W, w, b, up, dn, mode)
    B, N, C = x.shape
    h = N // W
    xp = np.zeros((B, h + 2, W + 2, C))
    xp[:, 1:h + 1, 1:W + 1] = x.reshape(B, h, W, C)
    if up is not None:
        xp[:, 0, 1:W + 1] = up
    ho, wo = h // 2, W // 2
    out = np.zeros((B, ho, wo, w.shape[0]))
    for ky in range(3):
        for kx in range(3):
            out += xp[:, ky + 1:ky + 1 + 2 * ho:2, kx:kx + 2 * wo:2, :] @ w[:, ky, kx, :].T
    return (out + b).reshape(B, ho * wo, w.shape[0])


def _up_shifted_columns(x, W, w, b, up, dn, mode):     # upsampled grid shifted by one column
    if mode != "up":
        return _ORIG["conv3x3_band_mode"](x, W, w, b, up, dn, mode)
    B, N, C = x.shape
    h = N // W
    g = np.roll(np.repeat(np.repeat(x.reshape(B, h, W, C), 2, axis=1), 2, axis=2), 1, axis=2).reshape(B, 4 * N, C)
    up2 = lambda r: None if r is None else np.repeat(r, 2, axis=1)
    return uo.conv3x3_band(g, 2 * W, w, b, up2(up), up2(dn))


def _conv_taps_transposed(x, W, w, b, up, dn):
    return _ORIG["conv3x3_band"](x, W, np.ascontiguousarray(w.transpose(0, 2, 1, 3)), b, up, dn)


def _pad_sides_swapped(x, W, up, dn):
    return _ORIG["pad_band"](x, W, dn, up)


def _edges_reversed(a, W):
    return _ORIG["edge_rows"](a, W)[:, ::-1]


def _ddpm_beta_over_alphabar(x_t, eu, ec, s, a_t, abar_t, sig, z):
    e = uo.guided_noise(eu, ec, s)
    mu = (x_t - (1.0 - a_t) / (1.0 - abar_t) * e) / math.sqrt(a_t)   # sqrt dropped
    return mu if z is None else mu + sig * z


def _ddim_no_renoise(x_t, eu, ec, s, abar_t, abar_prev):
    e = uo.guided_noise(eu, ec, s)
    return math.sqrt(abar_prev) * (x_t - math.sqrt(1.0 - abar_t) * e) / math.sqrt(abar_t)


def _resnet_shortcut_of_normed(W, wts, x, temb, *a, **k):
    y, e1, e2 = _ORIG_RESNET(W, wts, x, temb, *a, **k)
    if "skip_w" in wts:
        return y, e1, e2
    xn = oracle.group_norm(x, k.get("groups", 32), wts["gn1_gamma"], wts["gn1_beta"], eps=1e-5)
    return y - x + xn, e1, e2


_ORIG_RESNET = uo.resnet_block


def _resnet_temb_without_silu(W, wts, x, temb, *a, **k):
    # silu(temb) replaced by temb: enter through the module's silu only for the temb call
    calls = {"n": 0}
    real = _ORIG["silu"]

    def silu_skip_second(v):
        calls["n"] += 1
        return v if calls["n"] == 2 else real(v)
    uo.silu = silu_skip_second
    try:
        return _ORIG_RESNET(W, wts, x, temb, *a, **k)
    finally:
        uo.silu = real


@pytest.mark.parametrize("name,mutant", [
    ("conv3x3_band", _conv_taps_transposed),
    ("pad_band", _pad_sides_swapped),
    ("edge_rows", _edges_reversed),
    ("reverse_step_ddpm", _ddpm_beta_over_alphabar),
    ("reverse_step_ddim", _ddim_no_renoise),
    ("resnet_block", _resnet_shortcut_of_normed),
    ("resnet_block", _resnet_temb_without_silu),
    ("conv3x3_band_mode", _down_grid_shifted),
    ("conv3x3_band_mode", _up_shifted_columns),
])
def test_u5_planted_mistakes_are_caught(monkeypatch, name, mutant):
    monkeypatch.setattr(uo, name, mutant)
    assert not _battery()


# ---------------------------------------------------------------------------
# U6: the downsampling and upsampling convolutions of the U-Net, per band
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("B,H,W,ci,co,n", [(1, 12, 8, 3, 5, 3), (2, 8, 6, 4, 4, 4), (1, 6, 10, 2, 3, 1),
                                           (1, 16, 4, 3, 2, 2)])
def test_u6_band_downsample_is_the_whole_image_stride2_conv(B, H, W, ci, co, n):
    rng = np.random.default_rng(11)
    img = rng.standard_normal((B, H, W, ci))
    w = rng.standard_normal((co, 3, 3, ci))
    b = rng.standard_normal(co)
    x = torch.from_numpy(img).permute(0, 3, 1, 2)
    k = torch.from_numpy(np.ascontiguousarray(w.transpose(0, 3, 1, 2)))
    want = F.conv2d(x, k, torch.from_numpy(b), stride=2, padding=1).permute(0, 2, 3, 1).numpy()
    h = H // n
    for i, xb in enumerate(_bands(img, n)):
        up = img[:, i * h - 1] if i > 0 else None
        got = uo.conv3x3_band_mode(xb, W, w, b, up, None, "down")
        assert np.allclose(got.reshape(B, h // 2, W // 2, co), want[:, i * h // 2:(i + 1) * h // 2],
                           rtol=1e-12, atol=1e-12), i
        # the row below never matters
        dn = rng.standard_normal((B, W, ci))
        assert np.array_equal(uo.conv3x3_band_mode(xb, W, w, b, up, dn, "down"), got)


@pytest.mark.parametrize("B,H,W,ci,co,n", [(1, 6, 4, 3, 5, 3), (2, 4, 3, 4, 4, 4), (1, 3, 5, 2, 3, 1)])
def test_u6_band_upsample_is_the_whole_image_nearest_then_conv(B, H, W, ci, co, n):
    rng = np.random.default_rng(12)
    img = rng.standard_normal((B, H, W, ci))
    w = rng.standard_normal((co, 3, 3, ci))
    b = rng.standard_normal(co)
    x = torch.from_numpy(img).permute(0, 3, 1, 2)
    k = torch.from_numpy(np.ascontiguousarray(w.transpose(0, 3, 1, 2)))
    want = F.conv2d(F.interpolate(x, scale_factor=2.0, mode="nearest"), k, torch.from_numpy(b), padding=1)
    want = want.permute(0, 2, 3, 1).numpy()
    h = H // n
    for i, xb in enumerate(_bands(img, n)):
        up = img[:, i * h - 1] if i > 0 else None
        dn = img[:, (i + 1) * h] if i < n - 1 else None
        got = uo.conv3x3_band_mode(xb, W, w, b, up, dn, "up")
        assert np.allclose(got.reshape(B, 2 * h, 2 * W, co), want[:, 2 * i * h:2 * (i + 1) * h],
                           rtol=1e-12, atol=1e-12), i


# ---------------------------------------------------------------------------
# U7: one band's U-Net step with n = 1 is the whole image's U-Net, composed
# from torch operators
# ---------------------------------------------------------------------------

def _torch_unet(layers, weights, latent, temb, text, H0, W0, groups, p):
    from tests.test_oracle_block_pins import _torch_module
    f = lambda a: None if a is None else oracle.from_bf16_bits(a)
    B = latent.shape[0]
    cur = f(latent).reshape(B, H0, W0, -1)
    t_emb, t_text = f(temb), f(text)
    skips = []
    for ly in layers:
        w = weights[ly["name"]]
        if ly["kind"] == "conv":
            x = torch.from_numpy(cur).permute(0, 3, 1, 2)
            k = torch.from_numpy(np.ascontiguousarray(f(w["w"]).transpose(0, 3, 1, 2)))
            if ly["mode"] == 2:
                x = F.interpolate(x, scale_factor=2.0, mode="nearest")
            y = F.conv2d(x, k, torch.from_numpy(f(w["b"])), stride=2 if ly["mode"] == 1 else 1, padding=1)
            out = y.permute(0, 2, 3, 1).numpy()
        elif ly["kind"] == "resnet":
            if ly.get("pop"):
                cur = np.concatenate([cur, skips.pop()], axis=-1)
            out, _, _ = _torch_resnet(cur, t_emb, {k: f(v) for k, v in w.items()}, groups)
        elif ly["kind"] == "module":
            Hh, Ww, C = cur.shape[1], cur.shape[2], cur.shape[3]
            zeros = [(np.zeros((B, Hh * Ww, C)), np.zeros((B, Hh * Ww, C))) for _ in w["blocks"]]
            y = _torch_module(Hh, Ww, 1, 0, p, w["heads"], {k: f(v) for k, v in w["module"].items()},
                              [{k: f(v) for k, v in b.items()} for b in w["blocks"]], cur.reshape(B, Hh * Ww, C),
                              t_text, zeros, groups)
            out = y.reshape(B, Hh, Ww, C)
        else:
            x = torch.from_numpy(cur).permute(0, 3, 1, 2)
            y = F.silu(F.group_norm(x, groups, torch.from_numpy(f(w["gamma"])), torch.from_numpy(f(w["beta"])), eps=1e-5))
            out = y.permute(0, 2, 3, 1).numpy()
        if ly.get("push"):
            skips.append(out)
        cur = out
    return cur.reshape(B, H0 * W0, -1)


def test_u7_one_band_step_is_the_whole_image_unet():
    import dataclasses
    from paper_2412_02962_amd import synth
    sp = dataclasses.replace(synth.UNET_TINY, n=1, i=0, H0=16, W0=8)
    layers = synth.unet_layers(sp)
    weights, stale, latent, temb, text = synth.unet_band_inputs(sp)
    f = lambda a: None if a is None else oracle.from_bf16_bits(a)
    fw = {}
    for ly in layers:
        w = weights[ly["name"]]
        if ly["kind"] == "module":
            fw[ly["name"]] = {"module": {k: f(v) for k, v in w["module"].items()},
                              "blocks": [{k: f(v) for k, v in b.items()} for b in w["blocks"]], "heads": w["heads"]}
        else:
            fw[ly["name"]] = {k: f(v) for k, v in w.items()}
    fs = {k: ([tuple(f(a) for a in s) for s in v] if isinstance(v, list) else {kk: f(vv) for kk, vv in v.items()})
          for k, v in stale.items()}
    got = uo.unet_band_step(layers, 1, 0, sp.p, sp.groups, fw, fs, f(latent), f(temb), f(text))
    want = _torch_unet(layers, weights, latent, temb, text, sp.H0, sp.W0, sp.groups, sp.p)
    assert got.shape == (1, sp.H0 * sp.W0, 64)
    assert np.allclose(got, want, rtol=1e-9, atol=1e-9)
    assert np.abs(got[..., 4:]).max() == 0.0          # conv_out's padding outputs stay zero


def test_u8_image_steps_reach_the_whole_image_unet():
    """Repeated PCPP image steps on constant inputs: each step hands every
    band its neighbours' exports of the step before, so once nothing changes
    the stale data equal the fresh data.  With n = 2, p = 1 (a band attends
    to the whole other band) and synchronized GroupNorm that fixed point is
    the whole-image U-Net, composed here from torch operators; the bands'
    outputs stop changing after finitely many steps (the exchange delays
    each layer's inputs by one step at most per hop)."""
    import dataclasses
    from paper_2412_02962_amd import synth
    sp = dataclasses.replace(synth.UNET_TINY, n=2, i=0, H0=16, W0=8, p=1.0)
    layers = synth.unet_layers(sp)
    weights, _, latent, temb, text = synth.unet_band_inputs(dataclasses.replace(sp, n=1))
    f = lambda a: None if a is None else oracle.from_bf16_bits(a)
    fw = {}
    for ly in layers:
        w = weights[ly["name"]]
        if ly["kind"] == "module":
            fw[ly["name"]] = {"module": {k: f(v) for k, v in w["module"].items()},
                              "blocks": [{k: f(v) for k, v in b.items()} for b in w["blocks"]], "heads": w["heads"]}
        else:
            fw[ly["name"]] = {k: f(v) for k, v in w.items()}
    lat = f(latent)
    h0 = sp.H0 // sp.n
    latents = [lat[:, i * h0 * sp.W0:(i + 1) * h0 * sp.W0] for i in range(sp.n)]
    prev, last, steps = None, None, 0
    while steps < 200:
        outs, prev = uo.image_step(layers, sp.n, sp.p, sp.groups, fw, prev, latents, f(temb), f(text), sync_gn=True)
        steps += 1
        cur = np.concatenate(outs, axis=1)
        if last is not None and np.array_equal(cur, last):
            break
        last = cur
    assert steps < 200, "no fixed point"
    want = _torch_unet(layers, weights, latent, temb, text, sp.H0, sp.W0, sp.groups, sp.p)
    assert np.allclose(cur, want, rtol=1e-9, atol=1e-9)
    first, _ = uo.image_step(layers, sp.n, sp.p, sp.groups, fw, None, latents, f(temb), f(text), sync_gn=True)
    assert not np.allclose(np.concatenate(first, axis=1), want, atol=1e-3)  # the stale data matter


def test_u9_first_image_step_computes_each_band_as_an_image_of_its_own():
    """Before the first exchange nothing has been received.  Without
    synchronous warm-up steps the bands are then computed separately (the
    setting of Fig. 1): the first image step of band i equals the whole
    U-Net, composed here from torch operators, run on that band alone as an
    image of h rows (no stale rows in any attention, zero padding around the
    band in every convolution, the band's own GroupNorm statistics)."""
    import dataclasses
    from paper_2412_02962_amd import synth
    sp = dataclasses.replace(synth.UNET_TINY, n=2, i=0, H0=16, W0=8, p=0.5)
    layers = synth.unet_layers(sp)
    weights, _, latent, temb, text = synth.unet_band_inputs(dataclasses.replace(sp, n=1))
    f = lambda a: None if a is None else oracle.from_bf16_bits(a)
    fw = {}
    for ly in layers:
        w = weights[ly["name"]]
        if ly["kind"] == "module":
            fw[ly["name"]] = {"module": {k: f(v) for k, v in w["module"].items()},
                              "blocks": [{k: f(v) for k, v in b.items()} for b in w["blocks"]], "heads": w["heads"]}
        else:
            fw[ly["name"]] = {k: f(v) for k, v in w.items()}
    lat = f(latent)
    h0 = sp.H0 // sp.n
    tok = h0 * sp.W0
    latents = [lat[:, i * tok:(i + 1) * tok] for i in range(sp.n)]
    band_layers = synth.unet_layers(dataclasses.replace(sp, H0=h0, n=1))
    for sync_gn in (False, True):
        outs, _ = uo.image_step(layers, sp.n, sp.p, sp.groups, fw, None, latents, f(temb), f(text), sync_gn=sync_gn)
        for i in range(sp.n):
            want = _torch_unet(band_layers, weights, latent[:, i * tok:(i + 1) * tok], temb, text, h0, sp.W0,
                               sp.groups, sp.p)
            assert np.allclose(outs[i], want, rtol=1e-9, atol=1e-9), (sync_gn, i)
