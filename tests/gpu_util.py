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
