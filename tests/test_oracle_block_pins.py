"""Pins of the oracle's transformer-block pieces against torch.nn.functional
in float64 on the CPU (library routines), and of the whole block against a
torch composition that gathers the context by brute force from Eq. 1."""

import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from tests.oracle_pins_util import eq1_token_ids_brute

RNG = np.random.default_rng(7)


def _t(x):
    return torch.from_numpy(np.ascontiguousarray(x))


def test_group_norm_matches_torch():
    B, N, C, G = 2, 40, 24, 4
    x = RNG.standard_normal((B, N, C)) * 3 + 1.5
    gamma = 1 + 0.1 * RNG.standard_normal(C)
    beta = 0.1 * RNG.standard_normal(C)
    got = oracle.group_norm(x, G, gamma, beta, eps=1e-6)
    want = F.group_norm(_t(x).permute(0, 2, 1), G, _t(gamma), _t(beta), eps=1e-6).permute(0, 2, 1)
    np.testing.assert_allclose(got, want.numpy(), rtol=0, atol=1e-12)


def test_group_norm_groups_are_contiguous_channel_blocks():
    # shifting one group's channels must not move another group's output
    B, N, C, G = 1, 16, 12, 3
    x = RNG.standard_normal((B, N, C))
    one = np.ones(C)
    zero = np.zeros(C)
    a = oracle.group_norm(x, G, one, zero)
    x2 = x.copy()
    x2[:, :, 4:8] = x2[:, :, 4:8] * 5 + 7
    b = oracle.group_norm(x2, G, one, zero)
    np.testing.assert_allclose(a[:, :, :4], b[:, :, :4], atol=1e-13)
    np.testing.assert_allclose(a[:, :, 8:], b[:, :, 8:], atol=1e-13)
    np.testing.assert_allclose(a[:, :, 4:8], b[:, :, 4:8], atol=1e-5)  # affine-invariant up to eps


def test_layer_norm_matches_torch():
    x = RNG.standard_normal((2, 7, 33)) * 2 - 1
    gamma = 1 + 0.1 * RNG.standard_normal(33)
    beta = 0.1 * RNG.standard_normal(33)
    got = oracle.layer_norm(x, gamma, beta, eps=1e-5)
    want = F.layer_norm(_t(x), (33,), _t(gamma), _t(beta), eps=1e-5)
    np.testing.assert_allclose(got, want.numpy(), rtol=0, atol=1e-12)


def test_gelu_matches_torch_exact_gelu():
    x = np.linspace(-8, 8, 2001)
    np.testing.assert_allclose(oracle.gelu(x), F.gelu(_t(x), approximate="none").numpy(),
                               rtol=0, atol=1e-15)
    # closed forms: GELU(0) = 0, GELU(x) - GELU(-x) = x
    assert oracle.gelu(np.array([0.0]))[0] == 0.0
    np.testing.assert_allclose(oracle.gelu(x) - oracle.gelu(-x), x, atol=1e-14)


def test_linear_and_geglu_match_torch():
    x = RNG.standard_normal((1, 9, 16))
    w = RNG.standard_normal((2 * 12, 16))
    b = RNG.standard_normal(2 * 12)
    np.testing.assert_allclose(oracle.linear(x, w, b), F.linear(_t(x), _t(w), _t(b)).numpy(),
                               rtol=0, atol=1e-12)
    hcat = F.linear(_t(x), _t(w), _t(b))
    val, gate = hcat.chunk(2, dim=-1)
    want = val * F.gelu(gate)
    np.testing.assert_allclose(oracle.geglu(x, w, b), want.numpy(), rtol=0, atol=1e-12)


def _torch_block(H, W, n, i, p, heads, wts, x, text, stale_k_full, stale_v_full, groups):
    """The same block as a composition of torch.nn.functional calls, with the
    self-attention context gathered by brute force from Eq. 1."""
    T = {k: _t(v) for k, v in wts.items()}
    xt = _t(x)
    B, N, C = x.shape
    d = C // heads
    h = H // n

    def attn(q, k, v):
        def sp(z):
            return z.reshape(B, z.shape[1], heads, d).permute(0, 2, 1, 3)
        o = F.scaled_dot_product_attention(sp(q), sp(k), sp(v))
        return o.permute(0, 2, 1, 3).reshape(B, q.shape[1], C)

    t = F.group_norm(xt.permute(0, 2, 1), groups, T["gn_gamma"], T["gn_beta"], eps=1e-6).permute(0, 2, 1)
    hid = F.linear(t, T["proj_in_w"], T["proj_in_b"])
    n1 = F.layer_norm(hid, (C,), T["ln1_gamma"], T["ln1_beta"], eps=1e-5)
    q, k, v = F.linear(n1, T["attn1_qkv_w"]).chunk(3, dim=-1)
    kfull = _t(stale_k_full).clone()
    vfull = _t(stale_v_full).clone()
    kfull[:, i * h * W:(i + 1) * h * W] = k
    vfull[:, i * h * W:(i + 1) * h * W] = v
    ids = torch.from_numpy(eq1_token_ids_brute(H, W, n, i, p).astype(np.int64))
    hid = hid + F.linear(attn(q, kfull[:, ids], vfull[:, ids]), T["attn1_out_w"], T["attn1_out_b"])
    n2 = F.layer_norm(hid, (C,), T["ln2_gamma"], T["ln2_beta"], eps=1e-5)
    k2, v2 = F.linear(_t(text), T["attn2_kv_w"]).chunk(2, dim=-1)
    hid = hid + F.linear(attn(F.linear(n2, T["attn2_q_w"]), k2, v2), T["attn2_out_w"], T["attn2_out_b"])
    n3 = F.layer_norm(hid, (C,), T["ln3_gamma"], T["ln3_beta"], eps=1e-5)
    val, gate = F.linear(n3, T["ff1_w"], T["ff1_b"]).chunk(2, dim=-1)
    hid = hid + F.linear(val * F.gelu(gate), T["ff2_w"], T["ff2_b"])
    y = F.linear(hid, T["proj_out_w"], T["proj_out_b"]) + xt
    return y.numpy(), k.numpy(), v.numpy()


@pytest.mark.parametrize("i", [0, 1, 3])
def test_whole_block_matches_torch_composition(i):
    H, W, n, p, heads, d, groups = 16, 4, 4, 0.5, 2, 8, 4
    C, Tn, Td, Fi = heads * d, 5, 12, 24
    h = H // n
    shapes = {
        "gn_gamma": (C,), "gn_beta": (C,), "proj_in_w": (C, C), "proj_in_b": (C,),
        "ln1_gamma": (C,), "ln1_beta": (C,), "attn1_qkv_w": (3 * C, C),
        "attn1_out_w": (C, C), "attn1_out_b": (C,), "ln2_gamma": (C,), "ln2_beta": (C,),
        "attn2_q_w": (C, C), "attn2_kv_w": (2 * C, Td), "attn2_out_w": (C, C),
        "attn2_out_b": (C,), "ln3_gamma": (C,), "ln3_beta": (C,), "ff1_w": (2 * Fi, C),
        "ff1_b": (2 * Fi,), "ff2_w": (C, Fi), "ff2_b": (C,), "proj_out_w": (C, C),
        "proj_out_b": (C,),
    }
    wts = {}
    for name, shp in shapes.items():
        if name.endswith("_w"):
            wts[name] = RNG.standard_normal(shp) / math.sqrt(shp[1])
        elif name.endswith("gamma"):
            wts[name] = 1 + 0.1 * RNG.standard_normal(shp)
        else:
            wts[name] = 0.1 * RNG.standard_normal(shp)
    x = RNG.standard_normal((1, h * W, C))
    text = RNG.standard_normal((1, Tn, Td))
    stale_k = RNG.standard_normal((1, H * W, C))
    stale_v = RNG.standard_normal((1, H * W, C))

    def band(z, j):
        return z[:, j * h * W:(j + 1) * h * W] if 0 <= j < n else None

    y, k, v = oracle.transformer_block(H, W, n, i, p, heads, wts, x, text,
                                       band(stale_k, i - 1), band(stale_v, i - 1),
                                       band(stale_k, i + 1), band(stale_v, i + 1), gn_groups=groups)
    yt, kt, vt = _torch_block(H, W, n, i, p, heads, wts, x, text, stale_k, stale_v, groups)
    np.testing.assert_allclose(y, yt, rtol=0, atol=1e-11)
    np.testing.assert_allclose(k, kt, rtol=0, atol=1e-12)
    np.testing.assert_allclose(v, vt, rtol=0, atol=1e-12)


@pytest.mark.parametrize("n,i,B", [(4, 1, 1), (8, 7, 2), (2, 0, 1), (1, 0, 1)])
def test_synchronized_group_norm_is_whole_image_group_norm(n, i, B):
    # with every band's fresh statistics, the synchronized GroupNorm of band i
    # is torch's GroupNorm over the whole image restricted to band i's rows
    import torch
    import torch.nn.functional as F
    rng = np.random.default_rng(20 + n)
    h, W, C, G = 3, 5, 32, 8
    x = rng.standard_normal((B, n * h * W, C)) * 2.0 + 0.5
    gm, bt = 1 + 0.1 * rng.standard_normal(C), 0.1 * rng.standard_normal(C)
    bands = [x[:, j * h * W:(j + 1) * h * W] for j in range(n)]
    st = np.stack([oracle.group_stats(bj, G) for bj in bands])
    st_other = st.copy()
    st_other[i] = np.nan   # entry i is never read
    got = oracle.group_norm_synchronized(bands[i], G, gm, bt, st_other, i)
    full = F.group_norm(torch.from_numpy(x).permute(0, 2, 1), G, torch.from_numpy(gm), torch.from_numpy(bt),
                        eps=1e-6).permute(0, 2, 1).numpy()
    assert np.allclose(got, full[:, i * h * W:(i + 1) * h * W], rtol=0, atol=1e-12)


def test_group_stats_against_numpy():
    rng = np.random.default_rng(31)
    x = rng.standard_normal((2, 7, 12))
    st = oracle.group_stats(x, 3)
    for b in range(2):
        for g in range(3):
            blk = x[b, :, 4 * g:4 * g + 4].ravel()
            assert st[b, g, 0] == blk.size
            assert math.isclose(st[b, g, 1], float(np.mean(blk)), rel_tol=0, abs_tol=1e-14)
            assert math.isclose(st[b, g, 2], float(np.var(blk)) * blk.size, rel_tol=1e-12)


def _torch_module(H, W, n, i, p, heads, mw, bws, x, text, stale_full, groups):
    """A depth-d module as torch.nn.functional calls; block j's self-attention
    context gathered by brute force from Eq. 1 out of its own stale image."""
    T = {k: _t(v) for k, v in mw.items()}
    xt = _t(x)
    B, N, C = x.shape
    d = C // heads
    h = H // n
    ids = torch.from_numpy(eq1_token_ids_brute(H, W, n, i, p).astype(np.int64))

    def attn(q, k, v):
        def sp(z):
            return z.reshape(B, z.shape[1], heads, d).permute(0, 2, 1, 3)
        o = F.scaled_dot_product_attention(sp(q), sp(k), sp(v))
        return o.permute(0, 2, 1, 3).reshape(B, q.shape[1], C)

    t = F.group_norm(xt.permute(0, 2, 1), groups, T["gn_gamma"], T["gn_beta"], eps=1e-6).permute(0, 2, 1)
    hid = F.linear(t, T["proj_in_w"], T["proj_in_b"])
    for bw, (sk, sv) in zip(bws, stale_full):
        Tb = {k: _t(v) for k, v in bw.items()}
        n1 = F.layer_norm(hid, (C,), Tb["ln1_gamma"], Tb["ln1_beta"], eps=1e-5)
        q, k, v = F.linear(n1, Tb["attn1_qkv_w"]).chunk(3, dim=-1)
        kf, vf = _t(sk).clone(), _t(sv).clone()
        kf[:, i * h * W:(i + 1) * h * W] = k
        vf[:, i * h * W:(i + 1) * h * W] = v
        hid = hid + F.linear(attn(q, kf[:, ids], vf[:, ids]), Tb["attn1_out_w"], Tb["attn1_out_b"])
        n2 = F.layer_norm(hid, (C,), Tb["ln2_gamma"], Tb["ln2_beta"], eps=1e-5)
        k2, v2 = F.linear(_t(text), Tb["attn2_kv_w"]).chunk(2, dim=-1)
        hid = hid + F.linear(attn(F.linear(n2, Tb["attn2_q_w"]), k2, v2), Tb["attn2_out_w"], Tb["attn2_out_b"])
        n3 = F.layer_norm(hid, (C,), Tb["ln3_gamma"], Tb["ln3_beta"], eps=1e-5)
        val, gate = F.linear(n3, Tb["ff1_w"], Tb["ff1_b"]).chunk(2, dim=-1)
        hid = hid + F.linear(val * F.gelu(gate), Tb["ff2_w"], Tb["ff2_b"])
    return (F.linear(hid, T["proj_out_w"], T["proj_out_b"]) + xt).numpy()


@pytest.mark.parametrize("depth,i", [(1, 1), (2, 0), (3, 2)])
def test_transformer_module_matches_torch_composition(depth, i):
    H, W, n, p, heads, d, groups = 12, 4, 3, 0.5, 2, 8, 4
    C, Tn, Td, Fi = heads * d, 5, 12, 24
    h = H // n
    rng = np.random.default_rng(31 + depth)

    def draw(shp, name):
        if name.endswith("_w"):
            return rng.standard_normal(shp) / math.sqrt(shp[1])
        return (1 + 0.1 * rng.standard_normal(shp)) if name.endswith("gamma") else 0.1 * rng.standard_normal(shp)
    mw = {k: draw(s, k) for k, s in {"gn_gamma": (C,), "gn_beta": (C,), "proj_in_w": (C, C), "proj_in_b": (C,),
                                     "proj_out_w": (C, C), "proj_out_b": (C,)}.items()}
    bshapes = {"ln1_gamma": (C,), "ln1_beta": (C,), "attn1_qkv_w": (3 * C, C), "attn1_out_w": (C, C),
               "attn1_out_b": (C,), "ln2_gamma": (C,), "ln2_beta": (C,), "attn2_q_w": (C, C),
               "attn2_kv_w": (2 * C, Td), "attn2_out_w": (C, C), "attn2_out_b": (C,), "ln3_gamma": (C,),
               "ln3_beta": (C,), "ff1_w": (2 * Fi, C), "ff1_b": (2 * Fi,), "ff2_w": (C, Fi), "ff2_b": (C,)}
    assert tuple(bshapes) == oracle.MODULE_BLOCK_KEYS
    bws = [{k: draw(s, k) for k, s in bshapes.items()} for _ in range(depth)]
    x = rng.standard_normal((1, h * W, C))
    text = rng.standard_normal((1, Tn, Td))
    stale_full = [(rng.standard_normal((1, H * W, C)), rng.standard_normal((1, H * W, C))) for _ in range(depth)]

    def band(z, j):
        return z[:, j * h * W:(j + 1) * h * W] if 0 <= j < n else None
    stale = [(band(k, i - 1), band(v, i - 1), band(k, i + 1), band(v, i + 1)) for k, v in stale_full]
    y, ks, vs = oracle.transformer_module(H, W, n, i, p, heads, mw, bws, x, text, stale, gn_groups=groups)
    yt = _torch_module(H, W, n, i, p, heads, mw, bws, x, text, stale_full, groups)
    np.testing.assert_allclose(y, yt, rtol=0, atol=1e-10)
    assert len(ks) == depth and len(vs) == depth
    if depth == 1:   # the depth-1 module is the block
        wb = dict(mw)
        wb.update(bws[0])
        yb, kb, vb = oracle.transformer_block(H, W, n, i, p, heads, wb, x, text, *stale[0], gn_groups=groups)
        np.testing.assert_array_equal(y, yb)
        np.testing.assert_array_equal(ks[0], kb)
    else:            # each block reads its own stale K/V: swapping two blocks' changes the result
        y2, _, _ = oracle.transformer_module(H, W, n, i, p, heads, mw, bws, x, text, stale[::-1], gn_groups=groups)
        assert not np.allclose(y2, y) or i == 0 and n == 1
