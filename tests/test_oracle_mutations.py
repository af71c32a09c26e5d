"""Planted mistakes in the oracle (on the CPU, via monkeypatch) must be caught
by the pins: each mutant below fails at least one check of the battery, and
the unmodified oracle passes all of them."""

import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import oracle.pcpp_oracle as po
from paper_2412_02962_amd import synth
from tests.oracle_pins_util import eq1_token_ids_brute, full_grid


def _sdpa(q, k, v, heads):
    B, nq, C = q.shape
    d = C // heads
    sp = lambda x: torch.from_numpy(x).reshape(B, x.shape[1], heads, d).permute(0, 2, 1, 3)
    return F.scaled_dot_product_attention(sp(q), sp(k), sp(v)).permute(0, 2, 1, 3).reshape(B, nq, C).numpy()


def _battery():
    """True when every pin holds for the oracle as currently bound."""
    # P1: index sets on a grid of geometries, fractional p*h included
    for H, n in ((16, 4), (30, 3), (32, 2)):
        for i in range(n):
            for p in (0.0, 0.3, 0.5, 0.8, 1.0):
                if not np.array_equal(po.context_token_ids(H, 2, n, i, p),
                                      eq1_token_ids_brute(H, 2, n, i, p)):
                    return False
    # P2: attention over the brute-force context, two geometries
    for geo in (dict(H=16, W=4, n=4, i=1, p=0.5), dict(H=16, W=4, n=4, i=3, p=0.25)):
        cfg = synth.AttnConfig(name="m", heads=2, d=8, dtype="f32", seed_id=21, **geo)
        g = {"q": synth.patch_tensor(cfg, cfg.i, "q", False, "sharp"),
             "kf": synth.patch_tensor(cfg, cfg.i, "k", False, "sharp"),
             "vf": synth.patch_tensor(cfg, cfg.i, "v", False, "sharp")}
        nb = {}
        for tag, j in (("up", cfg.i - 1), ("dn", cfg.i + 1)):
            ok = 0 <= j < cfg.n
            nb["k" + tag] = synth.patch_tensor(cfg, j, "k", True, "sharp") if ok else None
            nb["v" + tag] = synth.patch_tensor(cfg, j, "v", True, "sharp") if ok else None
        got = oracle.partial_attention(cfg.H, cfg.W, cfg.n, cfg.i, cfg.p, cfg.heads, g["q"], g["kf"],
                                       g["vf"], nb["kup"], nb["vup"], nb["kdn"], nb["vdn"])
        ids = eq1_token_ids_brute(cfg.H, cfg.W, cfg.n, cfg.i, cfg.p)
        kfull = full_grid(cfg, "k", cfg.i, "sharp", synth)
        vfull = full_grid(cfg, "v", cfg.i, "sharp", synth)
        if not np.allclose(got, _sdpa(g["q"], kfull[:, ids], vfull[:, ids], cfg.heads), rtol=0, atol=1e-10):
            return False
    # block pieces against torch.nn.functional
    rng = np.random.default_rng(3)
    x = rng.standard_normal((1, 10, 16))
    gm, bt = 1 + 0.1 * rng.standard_normal(16), 0.1 * rng.standard_normal(16)
    t = torch.from_numpy
    if not np.allclose(oracle.layer_norm(x, gm, bt), F.layer_norm(t(x), (16,), t(gm), t(bt)).numpy(), atol=1e-10):
        return False
    if not np.allclose(oracle.group_norm(x, 4, gm, bt),
                       F.group_norm(t(x).permute(0, 2, 1), 4, t(gm), t(bt), eps=1e-6).permute(0, 2, 1).numpy(),
                       atol=1e-10):
        return False
    w, b = rng.standard_normal((12, 16)), rng.standard_normal(12)
    val, gate = F.linear(t(x), t(w), t(b)).chunk(2, dim=-1)
    if not np.allclose(oracle.geglu(x, w, b), (val * F.gelu(gate)).numpy(), atol=1e-10):
        return False
    return True


def test_unmodified_oracle_passes_battery():
    assert _battery()


def _rows_round(H, n, i, p):
    h = H // n
    r = min(h, int(round(p * h)))
    return h, (r if i > 0 else 0), (r if i < n - 1 else 0), (r if i > 0 else 0) + h + (r if i < n - 1 else 0)


def _assemble_wrong_band(H, W, n, i, p, fresh, up, dn):
    h, nu, nd, _ = po.context_rows(H, n, i, p)
    parts = []
    if nu:
        parts.append(up[:, 0:nu * W])          # upper rows of the patch above (wrong)
    parts.append(fresh)
    if nd:
        parts.append(dn[:, 0:nd * W])
    return np.concatenate(parts, axis=1)


def _mha_scale_1_over_d(q, k, v, heads, return_probs=False):
    B, nq, C = q.shape
    d = C // heads
    out = np.empty_like(q)
    for bb in range(B):
        for a in range(heads):
            s = q[bb, :, a * d:(a + 1) * d] @ k[bb, :, a * d:(a + 1) * d].T / d
            w = np.exp(s - s.max(axis=1, keepdims=True))
            out[bb, :, a * d:(a + 1) * d] = (w / w.sum(axis=1, keepdims=True)) @ v[bb, :, a * d:(a + 1) * d]
    return out


def _mha_v_is_k(q, k, v, heads, return_probs=False):
    return po.__dict__["_orig_mha"](q, k, k, heads)


def _mha_heads_interleaved(q, k, v, heads, return_probs=False):
    # head a taken as channels a, a+heads, ... instead of a contiguous block
    B, nq, C = q.shape
    perm = np.arange(C).reshape(C // heads, heads).T.reshape(-1)
    o = po.__dict__["_orig_mha"](q[:, :, perm], k[:, :, perm], v[:, :, perm], heads)
    out = np.empty_like(o)
    out[:, :, perm] = o
    return out


def _layer_norm_unbiased(x, gamma, beta, eps=1e-5):
    return (x - x.mean(-1, keepdims=True)) / np.sqrt(x.var(-1, ddof=1, keepdims=True) + eps) * gamma + beta


def _geglu_swapped(x, w, b):
    hc = po.linear(x, w, b)
    f = hc.shape[-1] // 2
    return hc[..., f:] * po.gelu(hc[..., :f])


def _group_norm_per_token(x, groups, gamma, beta, eps=1e-6):
    B, N, C = x.shape
    xr = x.reshape(B, N, groups, C // groups)
    m = xr.mean(-1, keepdims=True)
    v = ((xr - m) ** 2).mean(-1, keepdims=True)
    return ((xr - m) / np.sqrt(v + eps)).reshape(B, N, C) * gamma + beta


MUTANTS = {
    "rows_rounded": ("context_rows", _rows_round),
    "wrong_neighbour_band": ("assemble_context", _assemble_wrong_band),
    "scale_1_over_d": ("mha", _mha_scale_1_over_d),
    "v_replaced_by_k": ("mha", _mha_v_is_k),
    "heads_interleaved": ("mha", _mha_heads_interleaved),
    "layer_norm_unbiased": ("layer_norm", _layer_norm_unbiased),
    "geglu_swapped": ("geglu", _geglu_swapped),
    "group_norm_per_token": ("group_norm", _group_norm_per_token),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setitem(po.__dict__, "_orig_mha", po.mha)
    monkeypatch.setattr(po, attr, fn)
    monkeypatch.setattr(oracle, attr, fn)
    assert not _battery(), name
