"""Benchmark of the PCPP per-patch hot path on one MI355X.

A step is one pcpp_partial_attention call on the 2048 px SDXL level-1
workload (128 x 128 token grid, 640 channels = 10 heads x 64, 8 row bands,
band 3, partial value 0.25: 2048 queries x 3072 keys), inputs resident in HBM.
The K timed steps are captured in one HIP graph and replayed (the paper runs
with CUDA graphs to cut launch overhead), bracketed by HIP events on the
stream the kernels run on.  Prints one JSON line.

The CPU baseline is the float64 oracle timed on the host on a bounded sample
of whole steps of the same workload.
"""

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E

METRIC = "partial-attention TFLOP/s + % bf16 MFMA peak; ms/patch-step at 2048px, 1/8 patch"
WORKLOAD = "sdxl2048_l1_p25"


def attn_flops(cfg, n_kv):
    # QK^T and PV: 2 * 2 * heads * nq * n_kv * d (exp not counted)
    return 4.0 * cfg.batch * cfg.heads * cfg.n_q * n_kv * cfg.d


def attn_bytes(cfg, n_kv):
    # algorithmic bytes: Q read, K and V context read once, O written (bf16)
    return 2.0 * cfg.batch * cfg.C * (2 * cfg.n_q + 2 * n_kv)


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "attn_bf16_sdxl2048_l1_p25_traffic.txt")
CALIB_BYTES = 256 << 20      # plain device-to-device copy used to scale the memory counters
MEM_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "memory_kernels_sdxl2048_traffic.txt")


def kernel_source_hash():
    p = os.path.join(ROOT, "paper_2412_02962_amd", "csrc", "attention_bf16.hip")
    return hashlib.sha256(open(p, "rb").read()).hexdigest()[:16]


def load_traffic():
    """HBM traffic per launch from the committed rocprofv3 counter summary,
    only if it was taken on the current kernel source."""
    p = TRAFFIC_FILE
    if not os.path.exists(p):
        return None
    kv = {}
    for line in open(p):
        if ":" in line:
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("kernel_source_sha256_16") != kernel_source_hash():
        return None
    try:
        return float(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(cfg, inputs, budget_s=8.0):
    """The float64 oracle on the host: whole steps of the workload with every
    BLAS thread, then with one (threadpoolctl), each timed for about
    budget_s after one warm-up step."""
    import oracle
    from threadpoolctl import threadpool_info, threadpool_limits
    f = {k: oracle.as_f64(v, cfg.dtype) for k, v in inputs.items()}

    def step():
        return oracle.partial_attention(cfg.H, cfg.W, cfg.n, cfg.i, cfg.p, cfg.heads, f["q"], f["k_fresh"],
                                        f["v_fresh"], f["k_up"], f["v_up"], f["k_dn"], f["v_dn"])

    def timed(max_steps):
        step()  # warm
        n, t0 = 0, time.perf_counter()
        while True:
            step()
            n += 1
            el = time.perf_counter() - t0
            if el >= budget_s or n >= max_steps:
                return n, el

    threads = max([t.get("num_threads", 1) for t in threadpool_info() if t.get("user_api") == "blas"] or [1])
    n_all, el_all = timed(50)
    with threadpool_limits(limits=1, user_api="blas"):
        n_one, el_one = timed(5)
    _, _, _, rows = oracle.context_rows(cfg.H, cfg.n, cfg.i, cfg.p)
    fl = attn_flops(cfg, rows * cfg.W)
    return {"value": round(fl * n_all / el_all / 1e12, 6), "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
            "value_1thread": round(fl * n_one / el_one / 1e12, 6), "ms_per_step": round(el_all / n_all * 1e3, 2),
            "ms_per_step_1thread": round(el_one / n_one * 1e3, 2), "nproc": os.cpu_count(), "cpu_model": cpu_model(),
            "sample": f"whole steps of {WORKLOAD} (float64 numpy oracle): {n_all} steps with {threads} BLAS threads "
                      f"in {el_all:.1f} s, {n_one} steps with 1 thread in {el_one:.1f} s"}


def block_flops(bc, n_kv):
    """Algorithmic FLOPs of one transformer-block call (GEMMs + attention cores)."""
    cfg = bc.attn
    N, C, F, T, Td = cfg.n_q * cfg.batch, cfg.C, bc.ff_inner, bc.n_text * cfg.batch, bc.text_dim
    gemm = 2.0 * N * C * (C + 3 * C + C + C + C + 2 * F + C) + 2.0 * N * F * C + 2.0 * T * Td * 2 * C
    attn = 4.0 * N * n_kv * C + 4.0 * N * bc.n_text * C
    return gemm + attn


def resnet_flops(rc):
    """Algorithmic FLOPs of one ResNet-block call: the two 3x3 convolutions,
    the 1x1 shortcut when the width changes, the time-embedding projection."""
    M = rc.batch * rc.h * rc.W
    f = 2.0 * M * 9 * rc.c_in * rc.c_out + 2.0 * M * 9 * rc.c_out * rc.c_out
    if rc.c_in != rc.c_out:
        f += 2.0 * M * rc.c_in * rc.c_out
    return f + 2.0 * rc.batch * rc.temb_dim * rc.c_out


def resnet_call(torch, pcpp, synth, rc, dev):
    """(fn, tensors): one pcpp_resnet_block call on band rc.i with its inputs on dev."""
    import numpy as np
    to_dev = lambda x: None if x is None else torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(
        torch.bfloat16).to(dev)
    d = {k: to_dev(v) for k, v in synth.resnet_inputs(rc).items()}
    g = pcpp.make_resnet_geom(rc.H, rc.W, rc.n, rc.i, rc.c_in, rc.c_out, rc.temb_dim, rc.groups, rc.batch, 1e-5)
    w = pcpp.make_resnet_weights(d)
    y = torch.empty((rc.batch, rc.h * rc.W, rc.c_out), dtype=torch.bfloat16, device=dev)
    e1 = torch.empty((rc.batch, 2, rc.W, rc.c_in), dtype=torch.bfloat16, device=dev)
    e2 = torch.empty((rc.batch, 2, rc.W, rc.c_out), dtype=torch.bfloat16, device=dev)
    wsb = pcpp.pcpp_resnet_block_workspace_size(g)
    ws = torch.empty(wsb, dtype=torch.uint8, device=dev)

    def fn():
        pcpp.pcpp_resnet_block(g, w, d["x"], d["temb"], d["edges1_up"], d["edges1_dn"], d["edges2_up"],
                               d["edges2_dn"], None, None, None, None, y, e1, e2, ws, wsb)
    return fn, (d, y, e1, e2, ws)


def unet_flops(pcpp, synth, sp):
    """Algorithmic FLOPs of band sp.i's U-Net forward (the accounting of
    unet_device_inputs, without drawing anything)."""
    B, n, i, flops = sp.batch, sp.n, sp.i, 0.0
    for ly in synth.unet_layers(sp):
        H, W, ci, co = ly["H"], ly["W"], ly["c_in"], ly["c_out"]
        h = H // n
        if ly["kind"] == "conv":
            tok = {0: h * W, 1: (h // 2) * (W // 2), 2: 4 * h * W}[ly["mode"]]
            flops += 2.0 * B * tok * 9 * ci * co
        elif ly["kind"] == "resnet":
            flops += resnet_flops(synth.ResnetConfig(ly["name"], H, W, n, i, ci, co, temb_dim=sp.temb_dim,
                                                     groups=sp.groups, batch=B))
        elif ly["kind"] == "module":
            heads = co // 64
            bc = synth.BlockConfig(ly["name"], synth.AttnConfig(name=ly["name"], H=H, W=W, n=n, i=i, p=sp.p,
                                                                heads=heads, d=64, dtype="bf16", seed_id=0,
                                                                batch=B),
                                   n_text=sp.n_text, text_dim=sp.text_dim, ff_inner=4 * co, gn_groups=sp.groups)
            g = pcpp.make_geom(H, W, n, i, sp.p, heads, 64, B, 0, pcpp.PCPP_DTYPE_BF16)
            _, _, _, nkv = pcpp.pcpp_context_rows(g)
            proj = 2.0 * B * h * W * co * co * 2
            flops += ly["depth"] * (block_flops(bc, nkv) - proj) + proj
    return flops


def unet_device_inputs(torch, pcpp, synth, sp, dev, seed=7, sync_gn=True):
    """Seeded random weights and stale neighbour data of an SDXL-sized band
    U-Net drawn on the device (the same shapes and scales as
    synth.unet_band_inputs; a host draw of 2.6 G parameters would take
    minutes).  Returns (layers, weights, stale, latent, temb, text, flops)."""
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed)
    bf = torch.bfloat16
    rnd = lambda *shape: torch.randn(*shape, generator=gen, device=dev, dtype=torch.float32)
    lin = lambda shape, fan: (rnd(*shape) / fan ** 0.5).to(bf)
    B, n, i = sp.batch, sp.n, sp.i
    layers = synth.unet_layers(sp)
    weights, stale, flops = {}, {}, 0.0

    def band_stats(G, count):   # every band's (count, mean, M2), as synth._band_stats draws them
        st = torch.empty(n, B, G, 3, device=dev, dtype=torch.float32)
        st[..., 0] = count
        st[..., 1] = 0.1 * rnd(n, B, G)
        st[..., 2] = count * (0.8 + 0.4 * torch.rand(n, B, G, generator=gen, device=dev))
        return st
    for ly in layers:
        H, W, ci, co = ly["H"], ly["W"], ly["c_in"], ly["c_out"]
        h = H // n
        up, dn = i > 0, i < n - 1
        if ly["kind"] == "conv":
            weights[ly["name"]] = {"w": lin((co, 3, 3, ci), 9 * ci), "b": (0.02 * rnd(co)).to(bf)}
            stale[ly["name"]] = {"row_up": rnd(B, W, ci).to(bf) if up else None,
                                 "row_dn": rnd(B, W, ci).to(bf) if dn and ly["mode"] != 1 else None}
            tok = {0: h * W, 1: (h // 2) * (W // 2), 2: 4 * h * W}[ly["mode"]]
            flops += 2.0 * B * tok * 9 * ci * co
        elif ly["kind"] == "resnet":
            rc = synth.ResnetConfig(ly["name"], H, W, n, i, ci, co, temb_dim=sp.temb_dim, groups=sp.groups, batch=B)
            wd = {}
            for k, shp in synth.resnet_weight_shapes(rc).items():
                if k.endswith("_w"):
                    wd[k] = lin(shp, math.prod(shp[1:]))
                elif k.endswith("gamma"):
                    wd[k] = (1.0 + 0.1 * rnd(*shp)).to(bf)
                else:
                    wd[k] = ((0.02 if k.endswith("_b") else 0.1) * rnd(*shp)).to(bf)
            weights[ly["name"]] = wd
            stale[ly["name"]] = {"edges1_up": rnd(B, 2, W, ci).clamp_min(-0.28).to(bf) if up else None,
                                 "edges1_dn": rnd(B, 2, W, ci).clamp_min(-0.28).to(bf) if dn else None,
                                 "edges2_up": rnd(B, 2, W, co).clamp_min(-0.28).to(bf) if up else None,
                                 "edges2_dn": rnd(B, 2, W, co).clamp_min(-0.28).to(bf) if dn else None}
            if sync_gn:
                stale[ly["name"]]["gn1_bands"] = band_stats(sp.groups, h * W * ci / sp.groups)
                stale[ly["name"]]["gn2_bands"] = band_stats(sp.groups, h * W * co / sp.groups)
            flops += resnet_flops(rc)
        elif ly["kind"] == "module":
            heads, F = co // 64, 4 * co
            bc = synth.BlockConfig(ly["name"], synth.AttnConfig(name=ly["name"], H=H, W=W, n=n, i=i, p=sp.p,
                                                                heads=heads, d=64, dtype="bf16", seed_id=0,
                                                                batch=B),
                                   n_text=sp.n_text, text_dim=sp.text_dim, ff_inner=F, gn_groups=sp.groups)
            shapes = synth.block_weight_shapes(bc)

            def draw(k, shp):
                if k.endswith("_w"):
                    return lin(shp, shp[1])
                if k.endswith("gamma"):
                    return (1.0 + 0.1 * rnd(*shp)).to(bf)
                return ((0.02 if k.endswith("_b") else 0.1) * rnd(*shp)).to(bf)
            module = {k: draw(k, shapes[k]) for k in synth.MODULE_WEIGHT_NAMES}
            blocks = [{k: draw(k, shp) for k, shp in shapes.items() if k not in synth.MODULE_WEIGHT_NAMES}
                      for _ in range(ly["depth"])]
            weights[ly["name"]] = {"module": module, "blocks": blocks, "ff_inner": F, "heads": heads}
            nb = h * W
            stale[ly["name"]] = [tuple(rnd(B, nb, co).to(bf) if side else None for side in (up, up, dn, dn))
                                 for _ in range(ly["depth"])]
            g = pcpp.make_geom(H, W, n, i, sp.p, heads, 64, B, 0, pcpp.PCPP_DTYPE_BF16)
            _, _, _, nkv = pcpp.pcpp_context_rows(g)
            proj = 2.0 * B * nb * co * co * 2
            flops += ly["depth"] * (block_flops(bc, nkv) - proj) + proj
            if sync_gn:
                stale[ly["name"] + ":gn_bands"] = band_stats(sp.groups, nb * ci / sp.groups)
        else:  # the output GroupNorm
            weights[ly["name"]] = {"gamma": (1.0 + 0.1 * rnd(co)).to(bf), "beta": (0.1 * rnd(co)).to(bf)}
            stale[ly["name"]] = {"gn_bands": band_stats(sp.groups, h * W * co / sp.groups) if sync_gn else None}
    h0 = sp.H0 // n
    latent = torch.zeros(B, h0 * sp.W0, synth.LATENT_PAD, device=dev, dtype=bf)
    latent[:, :, :4] = rnd(B, h0 * sp.W0, 4).to(bf)
    temb = rnd(B, sp.temb_dim).to(bf)
    text = rnd(B, sp.n_text, sp.text_dim).to(bf)
    return layers, weights, stale, latent, temb, text, flops


def graph_time_us(torch, fn, K, use_graph=True, replays=5):
    """Microseconds per call of fn: K calls captured in one HIP graph, the
    graph replayed `replays` times after one untimed replay, the median replay
    divided by K (or K eager calls)."""
    for _ in range(3):
        fn()
    torch.cuda.synchronize()
    if not use_graph:
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(K):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / K * 1e3
    gr = torch.cuda.CUDAGraph()
    with torch.cuda.graph(gr):
        for _ in range(K):
            fn()
    gr.replay()
    torch.cuda.synchronize()
    times = []
    for _ in range(replays):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        gr.replay()
        e1.record()
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1))
    return sorted(times)[len(times) // 2] / K * 1e3


def extras(torch, pcpp, synth, dev, out_l1_us, use_graph=True, reps=200):
    """Context lines: materialised gather (GB/s vs HBM peak), the p = 0.5
    variant of the 2048 px level-1 workload, the level-2 shapes, and the full
    block."""
    import numpy as np

    def to_dev(x):
        return None if x is None else torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(
            torch.bfloat16).to(dev)

    out = {}
    cfg = synth.ATTN_CONFIGS[WORKLOAD]
    d = {k: to_dev(v) for k, v in synth.attention_inputs(cfg).items()}
    g = pcpp.make_geom(cfg.H, cfg.W, cfg.n, cfg.i, cfg.p, cfg.heads, cfg.d, 1, 0, pcpp.PCPP_DTYPE_BF16)
    _, _, _, n_kv = pcpp.pcpp_context_rows(g)
    idx = torch.empty(n_kv, dtype=torch.int32, device=dev)
    kc = torch.empty((1, n_kv, cfg.C), dtype=torch.bfloat16, device=dev)
    vc = torch.empty_like(kc)
    us = graph_time_us(torch, lambda: pcpp.pcpp_gather_context(g, d["k_fresh"], d["v_fresh"], d["k_up"], d["v_up"],
                                                               d["k_dn"], d["v_dn"], idx, kc, vc), reps, use_graph)
    gbytes = 2 * 2 * n_kv * cfg.C * 2 + 4 * n_kv
    out["gather_us"] = round(us, 3)
    out["gather_GBps"] = round(gbytes / us / 1e3, 1)
    out["gather_frac_hbm"] = round(gbytes / us / 1e3 / PEAK_HBM_GBS, 4)

    # The same copy with the caches flushed before each call (a 512 MiB
    # write between calls).
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)

    def flushed_us(fn, n=20):
        # graph of n x (flush, call) minus a graph of n x flush
        t_both = graph_time_us(torch, lambda: (flush.fill_(1), fn()), n, use_graph)
        t_flush = graph_time_us(torch, lambda: flush.fill_(1), n, use_graph)
        return max(t_both - t_flush, 1e-3)

    us = flushed_us(lambda: pcpp.pcpp_gather_context(g, d["k_fresh"], d["v_fresh"], d["k_up"], d["v_up"],
                                                     d["k_dn"], d["v_dn"], idx, kc, vc))
    out["gather_flushed_us"] = round(us, 3)
    out["gather_flushed_GBps"] = round(gbytes / us / 1e3, 1)

    # p-aware boundary messages of the same band: both messages packed from
    # the fresh K/V (sender side) and both placed into the stale buffers
    # (receiver side); bytes = read + write of every message.
    nb = pcpp.pcpp_boundary_bytes(g)
    s_up = torch.empty(nb // 2, dtype=torch.bfloat16, device=dev)
    s_dn = torch.empty(nb // 2, dtype=torch.bfloat16, device=dev)
    ku, vu, kd, vd = (torch.empty_like(d["k_fresh"]) for _ in range(4))
    us = graph_time_us(torch, lambda: pcpp.pcpp_pack_boundary(g, d["k_fresh"], d["v_fresh"], s_up, s_dn), reps,
                       use_graph)
    out["pack_us"] = round(us, 3)
    out["pack_GBps"] = round(2 * 2 * nb / us / 1e3, 1)
    out["pack_frac_hbm"] = round(2 * 2 * nb / us / 1e3 / PEAK_HBM_GBS, 4)
    out["message_bytes"] = nb
    us = graph_time_us(torch, lambda: pcpp.pcpp_unpack_boundary(g, s_dn, s_up, ku, vu, kd, vd), reps, use_graph)
    out["unpack_us"] = round(us, 3)
    out["unpack_GBps"] = round(2 * 2 * nb / us / 1e3, 1)
    us = flushed_us(lambda: pcpp.pcpp_pack_boundary(g, d["k_fresh"], d["v_fresh"], s_up, s_dn))
    out["pack_flushed_us"] = round(us, 3)
    out["pack_flushed_GBps"] = round(2 * 2 * nb / us / 1e3, 1)
    del flush

    # GroupNorm of the block's input alone (pcpp_group_norm: the statistics
    # kernel reads x, the apply kernel reads x and writes y; 2048 tokens x 640
    # channels, 32 groups): algorithmic bytes 3 x 2.6 MB.
    gx = torch.randn(1, cfg.n_q, cfg.C, device=dev).to(torch.bfloat16)
    gy = torch.empty_like(gx)
    gam = torch.ones(cfg.C, dtype=torch.bfloat16, device=dev)
    bet = torch.zeros(cfg.C, dtype=torch.bfloat16, device=dev)
    gws = pcpp.pcpp_group_norm_workspace_size(1, cfg.n_q, cfg.C, 32)
    gwsb = torch.empty(gws, dtype=torch.uint8, device=dev)
    us = graph_time_us(torch, lambda: pcpp.pcpp_group_norm(1, cfg.n_q, cfg.C, 32, 1e-6, 0, gx, gam, bet, gy, gwsb,
                                                           gws), reps, use_graph)
    gbytes = 3 * cfg.n_q * cfg.C * 2
    out["group_norm_us"] = round(us, 3)
    out["group_norm_GBps"] = round(gbytes / us / 1e3, 1)
    out["group_norm_frac_hbm"] = round(gbytes / us / 1e3 / PEAK_HBM_GBS, 4)

    # LayerNorm of a block's float32 stream alone (pcpp_layer_norm, 2048 x 640:
    # fp32 rows read, bf16 rows written): algorithmic bytes 6 x 2048 x 640.
    lx = torch.randn(cfg.n_q, cfg.C, device=dev)
    ly = torch.empty(cfg.n_q, cfg.C, dtype=torch.bfloat16, device=dev)
    us = graph_time_us(torch, lambda: pcpp.pcpp_layer_norm(cfg.n_q, cfg.C, 1e-5, lx, gam, bet, ly), reps, use_graph)
    lbytes = cfg.n_q * cfg.C * (4 + 2)
    out["layer_norm_us"] = round(us, 3)
    out["layer_norm_GBps"] = round(lbytes / us / 1e3, 1)
    out["layer_norm_frac_hbm"] = round(lbytes / us / 1e3 / PEAK_HBM_GBS, 4)

    c50 = synth.ATTN_CONFIGS["sdxl2048_l1_p50"]
    d50 = {k: to_dev(v) for k, v in synth.attention_inputs(c50).items()}
    g50 = pcpp.make_geom(c50.H, c50.W, c50.n, c50.i, c50.p, c50.heads, c50.d, 1, 0, pcpp.PCPP_DTYPE_BF16)
    _, _, _, nkv50 = pcpp.pcpp_context_rows(g50)
    o50 = torch.empty_like(d50["q"])
    w50 = pcpp.pcpp_partial_attention_workspace_size(g50)
    ws50 = torch.zeros(max(w50, 1), dtype=torch.uint8, device=dev)
    us = graph_time_us(torch, lambda: pcpp.pcpp_partial_attention(g50, d50["q"], d50["k_fresh"], d50["v_fresh"],
                                                                  d50["k_up"], d50["v_up"], d50["k_dn"],
                                                                  d50["v_dn"], o50, ws50, w50), reps, use_graph)
    out["p50_us"] = round(us, 3)
    out["p50_TFLOPs"] = round(attn_flops(c50, nkv50) / us / 1e6, 1)

    # SDXL's other self-attention shape at 2048 px: the 64 x 64 level-2 grid,
    # 1280 channels (20 heads), same 8 bands and p; the edge band (one
    # neighbour) and an interior band.  Derived, labelled as such: the
    # self-attention share of one whole U-Net step for one band, 10 level-1
    # layers + 60 level-2 layers (SDXL's transformer depths).
    l2 = {}
    for name, band in (("edge", None), ("interior", 3)):
        c2 = synth.ATTN_CONFIGS["sdxl2048_l2_edge"]
        if band is not None:
            import dataclasses
            c2 = dataclasses.replace(c2, i=band)
        d2 = {k: to_dev(v) for k, v in synth.attention_inputs(c2).items()}
        g2 = pcpp.make_geom(c2.H, c2.W, c2.n, c2.i, c2.p, c2.heads, c2.d, 1, 0, pcpp.PCPP_DTYPE_BF16)
        _, _, _, nkv2 = pcpp.pcpp_context_rows(g2)
        o2 = torch.empty_like(d2["q"])
        w2 = pcpp.pcpp_partial_attention_workspace_size(g2)
        ws2 = torch.zeros(max(w2, 1), dtype=torch.uint8, device=dev)
        us = graph_time_us(torch, lambda: pcpp.pcpp_partial_attention(g2, d2["q"], d2["k_fresh"], d2["v_fresh"],
                                                                      d2["k_up"], d2["v_up"], d2["k_dn"],
                                                                      d2["v_dn"], o2, ws2, w2), reps, use_graph)
        l2[name] = us
        out[f"l2_{name}_us"] = round(us, 3)
        out[f"l2_{name}_keys"] = nkv2
        out[f"l2_{name}_TFLOPs"] = round(attn_flops(c2, nkv2) / us / 1e6, 1)
    out["derived_unet_selfattn_ms_per_band_step"] = round((10 * out_l1_us + 60 * l2["interior"]) / 1e3, 4)

    # The same shapes with both guidance branches of a step in one launch
    # (batch 2: the conditional and unconditional images, as the U-Net step
    # with classifier-free guidance runs them); per-image time is half the
    # launch.
    cfg2 = {}
    for name, base, band in (("l1", WORKLOAD, None), ("l2_edge", "sdxl2048_l2_edge", None),
                             ("l2_interior", "sdxl2048_l2_edge", 3)):
        import dataclasses
        cb = dataclasses.replace(synth.ATTN_CONFIGS[base], batch=2)
        if band is not None:
            cb = dataclasses.replace(cb, i=band)
        db = {k: to_dev(v) for k, v in synth.attention_inputs(cb).items()}
        gb = pcpp.make_geom(cb.H, cb.W, cb.n, cb.i, cb.p, cb.heads, cb.d, 2, 0, pcpp.PCPP_DTYPE_BF16)
        _, _, _, nkvb = pcpp.pcpp_context_rows(gb)
        ob = torch.empty_like(db["q"])
        wb = pcpp.pcpp_partial_attention_workspace_size(gb)
        wsb_ = torch.zeros(max(wb, 1), dtype=torch.uint8, device=dev)
        us = graph_time_us(torch, lambda: pcpp.pcpp_partial_attention(gb, db["q"], db["k_fresh"], db["v_fresh"],
                                                                      db["k_up"], db["v_up"], db["k_dn"],
                                                                      db["v_dn"], ob, wsb_, wb), reps, use_graph)
        cfg2[name] = us / 2
        out[f"{name}_cfg_batch2_us"] = round(us, 3)
        out[f"{name}_cfg_batch2_us_per_image"] = round(us / 2, 3)
        out[f"{name}_cfg_batch2_TFLOPs"] = round(attn_flops(cb, nkvb) / us / 1e6, 1)
        del db, ob, wsb_
    out["derived_unet_selfattn_ms_per_band_step_cfg_batch2_per_image"] = round(
        (10 * cfg2["l1"] + 60 * cfg2["l2_interior"]) / 1e3, 4)

    # Multi-hop context (p > 1): 8 bands at 2048 px level 1, p = 1.5 (24 rows
    # on each side, from two bands), the stale rows given compactly.
    import dataclasses
    cm = dataclasses.replace(synth.ATTN_CONFIGS[WORKLOAD], p=1.5)
    h_, upm, dnm = cm.h, 24, 24
    qm = to_dev(synth.store(synth.patch_tensor(cm, cm.i, "q", False), "bf16"))
    mh = {}
    for kind in ("k", "v"):
        grid = np.concatenate([synth.patch_tensor(cm, j, kind, stale=(j != cm.i)) for j in range(cm.n)], axis=1)
        W_ = cm.W
        mh[kind + "_fresh"] = to_dev(synth.store(grid[:, cm.i * h_ * W_:(cm.i + 1) * h_ * W_], "bf16"))
        mh[kind + "_above"] = to_dev(synth.store(grid[:, (cm.i * h_ - upm) * W_:cm.i * h_ * W_], "bf16"))
        mh[kind + "_below"] = to_dev(synth.store(grid[:, (cm.i + 1) * h_ * W_:((cm.i + 1) * h_ + dnm) * W_], "bf16"))
        del grid
    gm = pcpp.make_geom(cm.H, cm.W, cm.n, cm.i, cm.p, cm.heads, cm.d, 1, 0, pcpp.PCPP_DTYPE_BF16)
    om = torch.empty_like(qm)
    wm = pcpp.pcpp_partial_attention_multihop_workspace_size(gm)
    wsm = torch.zeros(max(wm, 1), dtype=torch.uint8, device=dev)
    us = graph_time_us(torch, lambda: pcpp.pcpp_partial_attention_multihop(
        gm, qm, mh["k_fresh"], mh["v_fresh"], mh["k_above"], mh["v_above"], mh["k_below"], mh["v_below"], om, wsm,
        wm), reps, use_graph)
    nkm = (upm + h_ + dnm) * cm.W
    out["multihop_p1.5_us"] = round(us, 3)
    out["multihop_p1.5_keys"] = nkm
    out["multihop_p1.5_TFLOPs"] = round(attn_flops(cm, nkm) / us / 1e6, 1)

    # The paper's own band splits (two bands at p = 0.3, four at p = 0.8) on
    # both SDXL self-attention grids at 1024, 2048 and 3840 px; repetitions
    # scaled to about 20 ms of GPU time per shape.  Derived per split and
    # resolution: 10 level-1 + 60 level-2 layers of one band.
    geo = {}
    for name, c in synth.PAPER_GEOMETRIES.items():
        dg = {k: to_dev(v) for k, v in synth.attention_inputs(c).items()}
        gg = pcpp.make_geom(c.H, c.W, c.n, c.i, c.p, c.heads, c.d, 1, 0, pcpp.PCPP_DTYPE_BF16)
        _, _, _, nkvg = pcpp.pcpp_context_rows(gg)
        og = torch.empty_like(dg["q"])
        wg = pcpp.pcpp_partial_attention_workspace_size(gg)
        wsg = torch.zeros(max(wg, 1), dtype=torch.uint8, device=dev)
        fl = attn_flops(c, nkvg)
        k_reps = int(max(5, min(reps, 2e10 / fl)))
        us = graph_time_us(torch, lambda: pcpp.pcpp_partial_attention(gg, dg["q"], dg["k_fresh"], dg["v_fresh"],
                                                                      dg["k_up"], dg["v_up"], dg["k_dn"],
                                                                      dg["v_dn"], og, wsg, wg), k_reps, use_graph)
        geo[name] = {"us": round(us, 3), "keys": nkvg, "queries": c.n_q, "TFLOPs": round(fl / us / 1e6, 1)}
        del dg, og, wsg
    out["paper_geometries"] = geo
    der = {}
    for res in (1024, 2048, 3840):
        for n, pp in ((2, 0.3), (4, 0.8)):
            l1, l2 = geo[f"paper_{res}_l1_n{n}_p{pp}"]["us"], geo[f"paper_{res}_l2_n{n}_p{pp}"]["us"]
            der[f"{res}px_n{n}_p{pp}"] = round((10 * l1 + 60 * l2) / 1e3, 4)
    out["derived_unet_selfattn_ms_per_band_step_paper"] = der

    bc = synth.BLOCK_CONFIG
    bcfg = bc.attn
    bi = {k: to_dev(v) for k, v in synth.block_inputs(bc).items()}
    gb = pcpp.make_geom(bcfg.H, bcfg.W, bcfg.n, bcfg.i, bcfg.p, bcfg.heads, bcfg.d, 1, 0, pcpp.PCPP_DTYPE_BF16)
    _, _, _, nkvb = pcpp.pcpp_context_rows(gb)
    wts = pcpp.make_block_weights(bi, bc.ff_inner, bc.gn_groups)
    y = torch.empty_like(bi["x"])
    ko = torch.empty_like(bi["x"])
    vo = torch.empty_like(bi["x"])
    wsb = pcpp.pcpp_transformer_block_workspace_size(gb, wts, bc.n_text, bc.text_dim)
    wsb_t = torch.zeros(wsb, dtype=torch.uint8, device=dev)
    us = graph_time_us(torch, lambda: pcpp.pcpp_transformer_block(gb, wts, bi["x"], bi["text"], bc.n_text,
                                                                  bc.text_dim, bi["k_up"], bi["v_up"], bi["k_dn"],
                                                                  bi["v_dn"], y, ko, vo, wsb_t, wsb), max(reps // 4, 1),
                        use_graph)
    out["block_us"] = round(us, 3)
    out["block_TFLOPs"] = round(block_flops(bc, nkvb) / us / 1e6, 1)
    out["block_gflop"] = round(block_flops(bc, nkvb) / 1e9, 2)

    # the block at the second transformer level (1280 channels, 20 heads)
    bc2 = synth.BLOCK_CONFIG_L2
    c2 = bc2.attn
    b2 = {k: to_dev(v) for k, v in synth.block_inputs(bc2).items()}
    g2 = pcpp.make_geom(c2.H, c2.W, c2.n, c2.i, c2.p, c2.heads, c2.d, 1, 0, pcpp.PCPP_DTYPE_BF16)
    _, _, _, nkv2 = pcpp.pcpp_context_rows(g2)
    w2 = pcpp.make_block_weights(b2, bc2.ff_inner, bc2.gn_groups)
    y2, k2o, v2o = (torch.empty_like(b2["x"]) for _ in range(3))
    ws2b = pcpp.pcpp_transformer_block_workspace_size(g2, w2, bc2.n_text, bc2.text_dim)
    ws2 = torch.zeros(ws2b, dtype=torch.uint8, device=dev)
    us = graph_time_us(torch, lambda: pcpp.pcpp_transformer_block(g2, w2, b2["x"], b2["text"], bc2.n_text,
                                                                  bc2.text_dim, b2["k_up"], b2["v_up"], b2["k_dn"],
                                                                  b2["v_dn"], y2, k2o, v2o, ws2, ws2b),
                       max(reps // 4, 1), use_graph)
    out["block_l2_us"] = round(us, 3)
    out["block_l2_TFLOPs"] = round(block_flops(bc2, nkv2) / us / 1e6, 1)
    out["block_l2_gflop"] = round(block_flops(bc2, nkv2) / 1e9, 2)

    # SDXL's transformer modules: depth 2 at level 1, depth 10 at level 2
    for tag, bcm, depth in (("l1_depth2", synth.BLOCK_CONFIG, 2), ("l2_depth10", synth.BLOCK_CONFIG_L2, 10)):
        cm = bcm.attn
        x, text, module, blocks, stale = synth.module_inputs(bcm, depth)
        md = {k: to_dev(v) for k, v in module.items()}
        bd = [{k: to_dev(v) for k, v in blk.items()} for blk in blocks]
        wm, keep = pcpp.make_module_weights(md, bd, bcm.ff_inner, bcm.gn_groups)
        gm = pcpp.make_geom(cm.H, cm.W, cm.n, cm.i, cm.p, cm.heads, cm.d, 1, 0, pcpp.PCPP_DTYPE_BF16)
        _, _, _, nkvm = pcpp.pcpp_context_rows(gm)
        xd, td = to_dev(x), to_dev(text)
        cols = [[to_dev(a) for a in c] for c in zip(*stale)]
        ym = torch.empty_like(xd)
        kom = [torch.empty_like(xd) for _ in range(depth)]
        vom = [torch.empty_like(xd) for _ in range(depth)]
        wsm = pcpp.pcpp_transformer_module_workspace_size(gm, wm, bcm.n_text, bcm.text_dim)
        wsmt = torch.zeros(wsm, dtype=torch.uint8, device=dev)
        us = graph_time_us(torch, lambda: pcpp.pcpp_transformer_module(gm, wm, xd, td, bcm.n_text, bcm.text_dim,
                                                                       *cols, None, None, ym, kom, vom, wsmt, wsm),
                           max(reps // 20, 1), use_graph)
        cmf = block_flops(bcm, nkvm)
        proj = 2.0 * cm.n_q * cm.C * cm.C * 2          # proj_in and proj_out, once per module
        flops = depth * (cmf - proj) + proj
        out[f"module_{tag}_us"] = round(us, 3)
        out[f"module_{tag}_TFLOPs"] = round(flops / us / 1e6, 1)
        del keep, cols, bd, md

    # ResNet blocks of the three levels (bf16, batch 1: one guidance branch per device)
    for name, rc in synth.RESNET_CONFIGS.items():
        fn, keep = resnet_call(torch, pcpp, synth, rc, dev)
        us = graph_time_us(torch, fn, max(reps // 4, 1), use_graph)
        out[f"resnet_{name}_us"] = round(us, 3)
        out[f"resnet_{name}_TFLOPs"] = round(resnet_flops(rc) / us / 1e6, 1)
        del keep

    # the U-Net's resolution-changing convolutions (2048 px, 8 bands, band 3)
    for name, (H, W, n, i, ci, co, mode) in synth.CONV_CONFIGS.items():
        d = {k: to_dev(v) for k, v in synth.conv_inputs(H, W, n, i, ci, co, 1, 60).items()}
        g = pcpp.make_conv_geom(H, W, n, i, ci, co, 1, mode)
        h = H // n
        tokens = {0: h * W, 1: (h // 2) * (W // 2), 2: 4 * h * W}[mode]
        y = torch.empty((1, tokens, co), dtype=torch.bfloat16, device=dev)
        wsb = pcpp.pcpp_conv3x3_workspace_size(g)
        ws = torch.empty(wsb, dtype=torch.uint8, device=dev)
        us = graph_time_us(torch, lambda: pcpp.pcpp_conv3x3(g, d["x"], d["row_up"], d["row_dn"], d["w"], d["b"], y,
                                                            ws, wsb), max(reps // 4, 1), use_graph)
        out[f"conv_{name}_us"] = round(us, 3)
        out[f"conv_{name}_TFLOPs"] = round(2.0 * tokens * 9 * ci * co / us / 1e6, 1)

    # one band's whole U-Net forward at 2048 px (8 bands, band 3, one guidance branch,
    # synchronized GroupNorm)
    from paper_2412_02962_amd.unet import BandUNet
    sp = synth.UNET_SDXL_2048
    layers, uw, ust, ulat, utemb, utext, uflops = unet_device_inputs(torch, pcpp, synth, sp, dev)
    net = BandUNet(sp, layers, uw, ust, dev, sync_gn=True)
    us = graph_time_us(torch, lambda: net.forward(ulat, utemb, utext), 3, use_graph)
    out["unet_sdxl2048_band_step_ms"] = round(us / 1e3, 3)
    out["unet_sdxl2048_band_step_TFLOPs"] = round(uflops / us / 1e6, 1)
    out["unet_sdxl2048_band_step_gflop"] = round(uflops / 1e9, 1)
    del net, uw, ust, ulat, utemb, utext
    # the same band step with both guidance branches (unconditional and
    # conditional, Eq. 2) stacked as a batch of 2 in one pass
    sp2 = dataclasses.replace(sp, batch=2)
    layers, uw, ust, ulat, utemb, utext, uflops2 = unet_device_inputs(torch, pcpp, synth, sp2, dev)
    net = BandUNet(sp2, layers, uw, ust, dev, sync_gn=True)
    us = graph_time_us(torch, lambda: net.forward(ulat, utemb, utext), 3, use_graph)
    out["unet_sdxl2048_band_step_cfg_batch2_ms"] = round(us / 1e3, 3)
    out["unet_sdxl2048_band_step_cfg_batch2_TFLOPs"] = round(uflops2 / us / 1e6, 1)
    del net, uw, ust, ulat, utemb, utext
    # one whole-image PCPP step at 2048 px on this one device: the 8 bands'
    # U-Net forwards in turn, each with its neighbours' exports of the step
    # before (the exchange as zero-copy buffers), synchronized GroupNorm
    from paper_2412_02962_amd.image_step import ImageStep
    layers, uw, _, ulat, utemb, utext, _ = unet_device_inputs(torch, pcpp, synth, sp, dev)
    net = ImageStep(sp, layers, uw, dev, sync_gn=True)
    bands = [ulat.clone() for _ in range(sp.n)]
    flops_img = sum(unet_flops(pcpp, synth, dataclasses.replace(sp, i=i)) for i in range(sp.n))
    us = graph_time_us(torch, lambda: net.step(bands, utemb, utext), 2, use_graph)
    out["image_step_sdxl2048_8bands_one_gpu_ms"] = round(us / 1e3, 3)
    out["image_step_sdxl2048_8bands_one_gpu_TFLOPs"] = round(flops_img / us / 1e6, 1)
    del net, uw, ulat, utemb, utext, bands

    # the latent update of one band of the 2048 px image (latent 256 x 256 x 4, 8 bands)
    n = 256 // 8 * 256 * 4
    lat = [torch.randn(n, dtype=torch.float32, device=dev) for _ in range(4)]
    abar = 0.5
    sp = pcpp.make_step_params(pcpp.PCPP_STEP_DDIM, 5.0, alphabar_t=abar, alphabar_prev=0.55)
    us = graph_time_us(torch, lambda: pcpp.pcpp_guided_step(sp, n, lat[0], lat[1], lat[2], None, lat[3]), reps,
                       use_graph)
    out["guided_step_2048px_band_us"] = round(us, 3)
    return out


def pmc_run(args):
    """Workload for one rocprofv3 --pmc pass: a plain copy of CALIB_BYTES
    (calibrates the counters), then the timed workload's attention call
    repeated, nothing else."""
    import numpy as np
    import torch

    from paper_2412_02962_amd import pcpp, synth

    dev = "cuda:0"
    src = torch.ones(CALIB_BYTES // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    cfg = synth.ATTN_CONFIGS[args.workload]
    d = {k: (None if v is None else torch.from_numpy(np.ascontiguousarray(v).view(np.int16)).view(torch.bfloat16).to(dev))
         for k, v in synth.attention_inputs(cfg).items()}
    g = pcpp.make_geom(cfg.H, cfg.W, cfg.n, cfg.i, cfg.p, cfg.heads, cfg.d, cfg.batch, 0, pcpp.PCPP_DTYPE_BF16)
    out = torch.empty_like(d["q"])
    wsb = pcpp.pcpp_partial_attention_workspace_size(g)
    ws = torch.zeros(max(wsb, 1), dtype=torch.uint8, device=dev)
    for _ in range(args.steps):
        pcpp.pcpp_partial_attention(g, d["q"], d["k_fresh"], d["v_fresh"], d["k_up"], d["v_up"], d["k_dn"],
                                    d["v_dn"], out, ws, wsb, None)
    torch.cuda.synchronize()
    # the memory-bound kernels: the materialised gather of the same band, a
    # GroupNorm of the block's input shape, and whole blocks (their GroupNorm
    # and LayerNorm kernels)
    _, _, _, n_kv = pcpp.pcpp_context_rows(g)
    idx = torch.empty(n_kv, dtype=torch.int32, device=dev)
    kc = torch.empty((1, n_kv, cfg.C), dtype=torch.bfloat16, device=dev)
    vc = torch.empty_like(kc)
    gx = torch.randn(1, cfg.n_q, cfg.C, device=dev).to(torch.bfloat16)
    gy = torch.empty_like(gx)
    gam = torch.ones(cfg.C, dtype=torch.bfloat16, device=dev)
    bet = torch.zeros(cfg.C, dtype=torch.bfloat16, device=dev)
    gws = pcpp.pcpp_group_norm_workspace_size(1, cfg.n_q, cfg.C, 32)
    gwsb = torch.empty(gws, dtype=torch.uint8, device=dev)
    for _ in range(args.steps):
        pcpp.pcpp_gather_context(g, d["k_fresh"], d["v_fresh"], d["k_up"], d["v_up"], d["k_dn"], d["v_dn"], idx, kc,
                                 vc)
        pcpp.pcpp_group_norm(1, cfg.n_q, cfg.C, 32, 1e-6, 0, gx, gam, bet, gy, gwsb, gws)
    torch.cuda.synchronize()
    block_run(argparse.Namespace(level=1, steps=max(2, args.steps // 4)))
    print("pmc run done", flush=True)


def headline_attention(rows):
    """Dispatch ids of the attention calls of the timed workload in a
    --pmc-run counter file: the attention dispatches before the first gather
    (the block calls later in the run launch the same kernel on their own
    inputs, and a cross-attention shape)."""
    ids = sorted(int(r["Dispatch_Id"]) for r in rows if "attn_bf16_kernel" in r["Kernel_Name"])
    later = [int(r["Dispatch_Id"]) for r in rows if "gather_copy" in r["Kernel_Name"]]
    first_other = min(later) if later else None
    return {str(i) for i in ids if first_other is None or i < first_other}


def pmc_summarize(fetch_dir, write_dir):
    """Writes the traffic summary from two rocprofv3 --pmc outputs
    (FETCH_SIZE, then WRITE_SIZE; KiB per dispatch), each scaled by what the
    same counter reads for the calibration copy."""
    import csv
    import glob

    def per_kernel(d, counter):
        f = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)[0]
        rows = list(csv.DictReader(open(f)))
        head = headline_attention(rows)
        vals = {}
        for r in rows:
            if r["Counter_Name"] != counter:
                continue
            if "attn_bf16_kernel" in r["Kernel_Name"] and r["Dispatch_Id"] not in head:
                continue
            vals.setdefault(r["Kernel_Name"], {}).setdefault(r["Dispatch_Id"], 0.0)
            vals[r["Kernel_Name"]][r["Dispatch_Id"]] += float(r["Counter_Value"])
        return vals

    out = {}
    for d, counter in ((fetch_dir, "FETCH_SIZE"), (write_dir, "WRITE_SIZE")):
        v = per_kernel(d, counter)
        copy = [x for k, x in v.items() if "copy" in k.lower() or "elementwise" in k.lower()]
        attn = [x for k, x in v.items() if "attn_bf16_kernel" in k]
        copy_kib = max(max(x.values()) for x in copy)     # the 256 MiB copy dispatches
        attn_kib = sorted(attn[0].values())
        med = attn_kib[len(attn_kib) // 2]
        scale = copy_kib / (CALIB_BYTES / 1024.0)
        out[counter] = (med, copy_kib, scale)
    fetch, write = out["FETCH_SIZE"], out["WRITE_SIZE"]
    hbm = fetch[0] / fetch[2] * 1024.0 + write[0] / write[2] * 1024.0
    text = (
        "# Memory traffic of attn_bf16_kernel, 2048 px level-1 workload (one launch)\n"
        "# FETCH_SIZE and WRITE_SIZE are KiB per dispatch (L2 misses to the memory fabric), each divided by\n"
        "# its reading for a plain 256 MiB device-to-device copy over the copy's true size.\n"
        f"fetch_kib_per_launch: {fetch[0]:.1f}\n"
        f"write_kib_per_launch: {write[0]:.1f}\n"
        f"copy_fetch_kib: {fetch[1]:.1f}\n"
        f"copy_write_kib: {write[1]:.1f}\n"
        f"fetch_scale: {fetch[2]:.4f}\n"
        f"write_scale: {write[2]:.4f}\n"
        f"hbm_bytes_per_launch: {hbm:.0f}\n"
        f"kernel_source_sha256_16: {kernel_source_hash()}\n")
    open(TRAFFIC_FILE, "w").write(text)
    print(text)

    # Memory-bound kernels of the same run: median scaled HBM bytes per
    # dispatch against their algorithmic bytes at these shapes.
    cfg_c, tokens = 640, 2048
    algo = {
        "gather_copy": 4 * 3072 * cfg_c * 2 + 4 * 3072,      # read + write K and V context, indices
        "gn_stats": tokens * cfg_c * 2,                        # read x
        "gn_apply": 2 * tokens * cfg_c * 2,                    # read x, write y
        "ln_kernel": tokens * cfg_c * 4 + tokens * cfg_c * 2,  # read the fp32 stream, write bf16
    }
    fv = per_kernel(fetch_dir, "FETCH_SIZE")
    wv = per_kernel(write_dir, "WRITE_SIZE")
    rows = ["# HBM traffic of the memory-bound kernels (one dispatch; median over the run's dispatches of each),",
            "# FETCH_SIZE and WRITE_SIZE scaled as above; shapes of the 2048 px level-1 band (gather: 3072 keys x 640",
            "# channels, K and V; GroupNorm and LayerNorm: 2048 tokens x 640 channels, the block's and pcpp_group_norm's).",
            f"fetch_scale: {fetch[2]:.4f}",
            f"write_scale: {write[2]:.4f}",
            "kernel | fetched MB | written MB | HBM MB | algorithmic MB | HBM / algorithmic"]
    for key, ab in algo.items():
        fk = [sorted(x.values()) for k, x in fv.items() if key in k]
        wk = [sorted(x.values()) for k, x in wv.items() if key in k]
        if not fk or not wk:
            continue
        fmed = sorted(v for lst in fk for v in lst)
        wmed = sorted(v for lst in wk for v in lst)
        fb = fmed[len(fmed) // 2] / fetch[2] * 1024.0
        wb = wmed[len(wmed) // 2] / write[2] * 1024.0
        rows.append(f"{key} | {fb / 1e6:.2f} | {wb / 1e6:.2f} | {(fb + wb) / 1e6:.2f} | {ab / 1e6:.2f} | "
                    f"{(fb + wb) / ab:.2f}")
    mem = "\n".join(rows) + "\n"
    open(MEM_TRAFFIC_FILE, "w").write(mem)
    print(mem)


def block_run(args):
    """Workload for a kernel-trace profile of the transformer block: --steps
    calls of pcpp_transformer_block on the 2048 px level-1 band (--level 2:
    the level-2 band), nothing else."""
    import numpy as np
    import torch

    from paper_2412_02962_amd import pcpp, synth
    dev = "cuda:0"
    to_dev = lambda x: None if x is None else torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(
        torch.bfloat16).to(dev)
    bc = synth.BLOCK_CONFIG_L2 if args.level == 2 else synth.BLOCK_CONFIG
    c = bc.attn
    bi = {k: to_dev(v) for k, v in synth.block_inputs(bc).items()}
    g = pcpp.make_geom(c.H, c.W, c.n, c.i, c.p, c.heads, c.d, 1, 0, pcpp.PCPP_DTYPE_BF16)
    w = pcpp.make_block_weights(bi, bc.ff_inner, bc.gn_groups)
    y, ko, vo = (torch.empty_like(bi["x"]) for _ in range(3))
    wsb = pcpp.pcpp_transformer_block_workspace_size(g, w, bc.n_text, bc.text_dim)
    ws = torch.zeros(wsb, dtype=torch.uint8, device=dev)
    for _ in range(args.steps):
        pcpp.pcpp_transformer_block(g, w, bi["x"], bi["text"], bc.n_text, bc.text_dim, bi["k_up"], bi["v_up"],
                                    bi["k_dn"], bi["v_dn"], y, ko, vo, ws, wsb)
    torch.cuda.synchronize()
    print(f"block run: {args.steps} calls", flush=True)


def resnet_run(args):
    """Workload for a kernel-trace profile of the ResNet blocks: --steps calls
    of each 2048 px level-1 ResNet block, nothing else."""
    import torch

    from paper_2412_02962_amd import pcpp, synth
    for name, rc in synth.RESNET_CONFIGS.items():
        fn, keep = resnet_call(torch, pcpp, synth, rc, "cuda:0")
        for _ in range(args.steps):
            fn()
        torch.cuda.synchronize()
        print(f"resnet run {name}: {args.steps} calls", flush=True)
        del keep


def unet_run(args):
    """Workload for a kernel-trace profile of one band's U-Net forward at
    2048 px (8 bands, band 3): --steps forwards, nothing else."""
    import torch

    from paper_2412_02962_amd import pcpp, synth
    from paper_2412_02962_amd.unet import BandUNet
    sp = synth.UNET_SDXL_2048
    layers, w, st, lat, temb, text, _ = unet_device_inputs(torch, pcpp, synth, sp, "cuda:0")
    net = BandUNet(sp, layers, w, st, "cuda:0", sync_gn=True)
    torch.cuda.synchronize()
    for _ in range(args.steps):
        net.forward(lat, temb, text)
    torch.cuda.synchronize()
    print(f"unet run: {args.steps} band steps", flush=True)


def gemm_calibration():
    """hipBLASLt (through torch.matmul, bf16, HIP graph of 20 calls) on the
    GEMM shapes of the 2048 px level-1 block and ResNets: a yardstick for the
    library's own GEMM kernels at these small-M shapes."""
    import torch
    dev = "cuda:0"
    shapes = [("3x3 convolution 640 -> 640 as a plain GEMM", 2048, 640, 5760),
              ("3x3 convolution 320 -> 640 as a plain GEMM", 2048, 640, 2880),
              ("640 x 640 projection", 2048, 640, 640), ("Q/K/V", 2048, 1920, 640),
              ("GEGLU product (no GELU)", 2048, 5120, 640), ("FF-out", 2048, 640, 2560),
              ("large square", 8192, 8192, 8192)]
    for name, M, N, K in shapes:
        a = torch.randn(M, K, device=dev, dtype=torch.bfloat16)
        w = torch.randn(N, K, device=dev, dtype=torch.bfloat16)
        out = torch.empty(M, N, device=dev, dtype=torch.bfloat16)
        us = graph_time_us(torch, lambda: torch.matmul(a, w.t(), out=out), 20 if M < 8192 else 5)
        print(f"{name:45s} M={M:5d} N={N:5d} K={K:5d}: {us:8.2f} us {2.0 * M * N * K / us / 1e6:7.1f} TFLOP/s",
              flush=True)


def pmc_report(dirs):
    """Per-dispatch averages of every counter rocprofv3 --pmc recorded for the
    attention kernel in the given output folders (one folder per pass), with
    the dispatch durations, for the counter summary under profiles/."""
    import csv
    import glob
    lines = ["# Hardware counters of attn_bf16_kernel, 2048 px level-1 workload, per dispatch "
             "(rocprofv3 --pmc; averages over the dispatches of each pass)"]
    for d in dirs:
        f = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)[0]
        rows = list(csv.DictReader(open(f)))
        head = headline_attention(rows)
        vals, durs = {}, {}
        for r in rows:
            if r["Dispatch_Id"] not in head:
                continue
            vals.setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
            durs[r["Dispatch_Id"]] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        dd = sorted(durs.values())
        lines.append(f"## pass {os.path.basename(os.path.normpath(d))}: {len(dd)} dispatches, "
                     f"median duration {dd[len(dd) // 2]:.2f} us")
        for k in sorted(vals):
            v = vals[k]
            lines.append(f"{k}: {sum(v) / len(v):.1f}")
    lines.append(f"kernel_source_sha256_16: {kernel_source_hash()}")
    print("\n".join(lines))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=WORKLOAD)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-graph", action="store_true", help="time eager launches instead of a graph")
    ap.add_argument("--no-extras", action="store_true", help="skip the gather / p=0.5 / block context lines")
    ap.add_argument("--pmc-run", action="store_true",
                    help="counter-collection workload: a calibration copy, --steps attention calls, then the "
                         "gather, GroupNorm and block calls whose memory-bound kernels the summary covers")
    ap.add_argument("--pmc-summarize", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="write the traffic summary from two rocprofv3 --pmc output folders")
    ap.add_argument("--block-run", action="store_true",
                    help="profiling workload: --steps transformer-block calls, nothing else")
    ap.add_argument("--level", type=int, default=1, choices=(1, 2), help="transformer level of --block-run")
    ap.add_argument("--resnet-run", action="store_true",
                    help="profiling workload: --steps calls of each ResNet block, nothing else")
    ap.add_argument("--unet-run", action="store_true",
                    help="profiling workload: --steps band U-Net forwards at 2048 px, nothing else")
    ap.add_argument("--gemm-calibration", action="store_true",
                    help="time hipBLASLt (torch.matmul) on the block's and ResNets' GEMM shapes")
    ap.add_argument("--pmc-report", nargs="+", metavar="DIR",
                    help="print per-dispatch counter averages of the attention kernel from rocprofv3 --pmc folders")
    args = ap.parse_args()
    if args.pmc_summarize:
        pmc_summarize(*args.pmc_summarize)
        return
    if args.pmc_report:
        pmc_report(args.pmc_report)
        return
    if args.block_run:
        block_run(args)
        return
    if args.resnet_run:
        resnet_run(args)
        return
    if args.gemm_calibration:
        gemm_calibration()
        return
    if args.unet_run:
        unet_run(args)
        return
    if args.pmc_run:
        pmc_run(args)
        return

    if args.gpus != 1:
        print(f"bench.py measures one GPU only (the per-band hot path); --gpus {args.gpus} is not supported. "
              "Multi-GPU sharding is a design note, not part of this build.", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2412_02962_amd import pcpp, synth

    dev = "cuda:0"
    torch.cuda.set_device(0)
    cfg = synth.ATTN_CONFIGS[args.workload]
    inputs = synth.attention_inputs(cfg)

    def to_dev(x):
        if x is None:
            return None
        import numpy as np
        return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).to(dev)

    d = {k: to_dev(v) for k, v in inputs.items()}
    g = pcpp.make_geom(cfg.H, cfg.W, cfg.n, cfg.i, cfg.p, cfg.heads, cfg.d, cfg.batch, 0, pcpp.PCPP_DTYPE_BF16)
    h, up, dn, n_kv = pcpp.pcpp_context_rows(g)
    out = torch.empty_like(d["q"])
    wsb = pcpp.pcpp_partial_attention_workspace_size(g)
    ws = torch.zeros(max(wsb, 1), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()

    def step():
        # stream=None: the launch goes to torch's current stream, which is the
        # capture stream inside torch.cuda.graph()
        pcpp.pcpp_partial_attention(g, d["q"], d["k_fresh"], d["v_fresh"], d["k_up"], d["v_up"], d["k_dn"],
                                    d["v_dn"], out, ws, wsb, None)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    K = args.steps
    graph = None
    if not args.no_graph:
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for _ in range(K):
                step()
        graph.replay()  # untimed: first replay uploads the graph
        torch.cuda.synchronize()

    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(stream)
    if graph is not None:
        graph.replay()
    else:
        for _ in range(K):
            step()
    ev1.record(stream)
    torch.cuda.synchronize()
    ms_total = ev0.elapsed_time(ev1)
    ms_step = ms_total / K

    # per-launch durations: an event pair around each of 200 eager launches
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(200)]
    for e0, e1 in evs:
        e0.record(stream)
        step()
        e1.record(stream)
    torch.cuda.synchronize()
    per = sorted(e0.elapsed_time(e1) * 1e3 for e0, e1 in evs)
    pct = {q: round(per[min(len(per) - 1, int(q / 100 * len(per)))], 3) for q in (10, 50, 90)}

    # eager rate as context (includes host launch overhead of the ctypes call)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(50):
        step()
    torch.cuda.synchronize()
    eager_ms = (time.perf_counter() - t0) / 50 * 1e3

    flops = attn_flops(cfg, n_kv)
    abytes = attn_bytes(cfg, n_kv)
    tflops = flops / (ms_step * 1e-3) / 1e12
    traffic = load_traffic()
    res = {
        "metric": METRIC,
        "value": round(tflops, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": args.workload, "grid": f"{cfg.H}x{cfg.W}", "bands": cfg.n, "band": cfg.i,
                   "partial": cfg.p, "heads": cfg.heads, "head_dim": cfg.d, "queries": cfg.n_q,
                   "keys": n_kv, "batch": cfg.batch, "timing": "hip-graph" if graph is not None else "eager"},
        "roofline": {"bound": "mfma", "achieved": round(tflops, 3), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(tflops / PEAK_BF16_TFLOPS, 4), "traffic": traffic,
                     "algorithmic_bytes": abytes, "kernel_avg_us": round(ms_step * 1e3, 3)},
        "extra": {"pct_bf16_peak": round(100 * tflops / PEAK_BF16_TFLOPS, 2), "eager_ms_per_call": round(eager_ms, 4),
                  "workspace_bytes": wsb, "gflop_per_step": round(flops / 1e9, 3),
                  "launch_us_p10": pct[10], "launch_us_p50": pct[50], "launch_us_p90": pct[90]},
    }
    if not args.no_extras:
        res["extra"].update(extras(torch, pcpp, synth, dev, ms_step * 1e3, graph is not None, min(K, 200)))
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(cfg, inputs)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
