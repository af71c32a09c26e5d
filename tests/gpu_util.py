"""Helpers of the GPU parity tests: move synthetic inputs to the device, call
the library through its C ABI binding, bring results back as float64."""

import numpy as np
import torch

from paper_2412_02962_amd import synth

DEV = "cuda:0"

# Tolerances against the float64 oracle (per output element).
TOL_F32_MAX = 1e-5
TOL_BF16_MAX = 2e-2
TOL_BF16_MEAN = 2e-3


def to_dev(x, dtype):
    """Stored array (float32 or uint16 bf16 bits) -> device tensor."""
    if x is None:
        return None
    if dtype == synth.DTYPE_BF16:
        t = torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(DEV)


def to_f64(t):
    return t.detach().to("cpu", torch.float64).numpy()


def lib_dtype(cfg):
    from paper_2412_02962_amd import pcpp
    return pcpp.PCPP_DTYPE_BF16 if cfg.dtype == synth.DTYPE_BF16 else pcpp.PCPP_DTYPE_F32


def geom(cfg, **over):
    from paper_2412_02962_amd import pcpp
    kw = dict(H=cfg.H, W=cfg.W, n_patches=cfg.n, patch_idx=cfg.i, partial=cfg.p, heads=cfg.heads,
              head_dim=cfg.d, batch=cfg.batch, step=cfg.step, dtype=lib_dtype(cfg))
    kw.update(over)
    return pcpp.make_geom(**kw)


def run_attention(cfg, inputs, g=None, stream=None):
    """Run pcpp_partial_attention on stored-dtype inputs; returns the device output."""
    from paper_2412_02962_amd import pcpp
    g = geom(cfg) if g is None else g
    d = {k: to_dev(v, cfg.dtype) for k, v in inputs.items()}
    out = torch.empty_like(d["q"])
    ws_bytes = pcpp.pcpp_partial_attention_workspace_size(g)
    ws = torch.zeros(max(ws_bytes, 1), dtype=torch.uint8, device=DEV)
    if stream is not None:  # another stream: the inputs and the cleared workspace must be in place
        torch.cuda.synchronize()
    pcpp.pcpp_partial_attention(g, d["q"], d["k_fresh"], d["v_fresh"], d["k_up"], d["v_up"], d["k_dn"],
                                d["v_dn"], out, ws, ws_bytes, stream)
    torch.cuda.synchronize()
    return out


def oracle_attention(cfg, inputs):
    import oracle
    f = {k: oracle.as_f64(v, cfg.dtype) for k, v in inputs.items()}
    return oracle.partial_attention(cfg.H, cfg.W, cfg.n, cfg.i, cfg.p, cfg.heads, f["q"], f["k_fresh"],
                                    f["v_fresh"], f["k_up"], f["v_up"], f["k_dn"], f["v_dn"])


def assert_close(cfg, got, want, tag=""):
    err = np.abs(got - want)
    mx, mean = float(err.max()), float(err.mean())
    if cfg.dtype == synth.DTYPE_F32:
        assert mx <= TOL_F32_MAX, f"{tag} f32 max-abs {mx:.3e} > {TOL_F32_MAX}"
    else:
        assert mx <= TOL_BF16_MAX, f"{tag} bf16 max-abs {mx:.3e} > {TOL_BF16_MAX}"
        assert mean <= TOL_BF16_MEAN, f"{tag} bf16 mean-abs {mean:.3e} > {TOL_BF16_MEAN}"
    return mx, mean


def multihop_inputs(cfg):
    """Stored-dtype inputs of a multi-hop call: q, fresh K/V of band i and
    the compact stale rows above and below it, cut from the stale copies of
    the other bands."""
    import oracle
    _, up, dn, _ = oracle.context_rows_multihop(cfg.H, cfg.n, cfg.i, cfg.p)
    W, h, i = cfg.W, cfg.h, cfg.i
    out = {"q": synth.store(synth.patch_tensor(cfg, i, "q", False), cfg.dtype)}
    for kind in ("k", "v"):
        grid = np.concatenate([synth.patch_tensor(cfg, j, kind, stale=(j != i)) for j in range(cfg.n)], axis=1)
        out[kind + "_fresh"] = synth.store(grid[:, i * h * W:(i + 1) * h * W], cfg.dtype)
        out[kind + "_above"] = synth.store(grid[:, (i * h - up) * W:i * h * W], cfg.dtype) if up else None
        out[kind + "_below"] = synth.store(grid[:, (i + 1) * h * W:((i + 1) * h + dn) * W], cfg.dtype) if dn else None
    return out


# ---------------------------------------------------------------------------
# Element-wise bound for compositions of bf16-rounded stages
# ---------------------------------------------------------------------------
#
# A composition (a transformer block, a module of d blocks, a U-Net) stores
# S of its intermediates in bf16 before they feed a GEMM or the next layer,
# and rounds its output once.  Each stored rounding is a relative error
# uniform in +-2^-9, standard deviation 2^-9 / sqrt(3) of that tensor; a
# GEMM turns it into a near-Gaussian error of the same relative size of the
# product, and the residual sums carry it to the output.  Errors of
# different stages are independent, so they add in quadrature: the output's
# error has a standard deviation of about 2^-9 / sqrt(3) * sqrt(S) * rms(y).
#   per element:  |dy| <= 2^-8 |y| + 2.45 sqrt(S) 2^-8 rms(y)
#   mean-abs:     <= 2^-8 rms(y) sqrt(S / 6)
# The first term is the output's own rounding.  The second is about 6.8
# standard deviations (the largest of a million Gaussian draws is about 5);
# at S = 6 (one transformer block) both are the block test's derived bound,
# 2^-8 |y| + 6 * 2^-8 rms(y) per element and 2^-8 rms(y) on average.  The
# mean bound is about 2.5 standard deviations (the mean absolute value of a
# Gaussian is 0.8 of one).

def composition_bound(want, stages):
    rms = float(np.sqrt(np.mean(want ** 2)))
    per = 2.0 ** -8 * np.abs(want) + 2.45 * np.sqrt(stages) * 2.0 ** -8 * rms
    mean = 2.0 ** -8 * rms * np.sqrt(stages / 6.0)
    return per, mean, rms


def check_composition(got, want, stages, tag=""):
    """Asserts the element-wise and mean bounds above; returns (worst
    err/bound, mean-abs / mean bound)."""
    per, mean_bound, rms = composition_bound(want, stages)
    err = np.abs(got - want)
    worst = float((err / per).max())
    mean = float(err.mean())
    print(f"{tag}: stages {stages}, max-abs {err.max():.3e}, worst err/bound {worst:.3f}, "
          f"mean-abs {mean:.3e} ({mean / mean_bound:.3f} of its bound), rms {rms:.3f}", flush=True)
    assert np.isfinite(got).all(), f"{tag}: non-finite output"
    assert worst <= 1.0, f"{tag}: max error exceeds the bound by {worst:.2f}x"
    assert mean <= mean_bound, f"{tag}: mean-abs {mean:.3e} > {mean_bound:.3e}"
    return worst, mean / mean_bound


def block_rows(n_q, block, rng, extra=1):
    """Query rows that cover every block of `block` queries: its first and
    last row and `extra` random rows in between (all rows of short blocks)."""
    rows = []
    for b0 in range(0, n_q, block):
        b1 = min(b0 + block, n_q)
        rows += [b0, b1 - 1]
        if b1 - b0 > 2:
            rows += list(rng.choice(np.arange(b0 + 1, b1 - 1), min(extra, b1 - b0 - 2), replace=False))
    return np.unique(np.asarray(rows))


def attention_block_queries(cfg):
    """Queries per workgroup block of the bf16 attention launch on this device."""
    from paper_2412_02962_amd import pcpp
    return pcpp.pcpp_partial_attention_plan(geom(cfg))[0]
