"""GPU parity of pcpp_partial_attention and pcpp_gather_context against the
float64 oracle, through the C ABI, on seeded synthetic inputs."""

import dataclasses

import numpy as np
import pytest

import oracle
from paper_2412_02962_amd import synth
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu


def _cfg(name, **over):
    return dataclasses.replace(synth.ATTN_CONFIGS[name], **over)


def _say(*a):
    print("[case]", *a, flush=True)


@pytest.mark.parametrize("name", list(synth.ATTN_CONFIGS))
@pytest.mark.parametrize("variant", ["unit", "prescaled", "sharp"])
def test_attention_matches_oracle_on_workloads(name, variant):
    cfg = synth.ATTN_CONFIGS[name]
    _say("attention", name, variant)
    inp = synth.attention_inputs(cfg, variant)
    got = gu.to_f64(gu.run_attention(cfg, inp))
    want = gu.oracle_attention(cfg, inp)
    mx, mean = gu.assert_close(cfg, got, want, f"{name}/{variant}")
    rel = np.linalg.norm(got - want) / np.linalg.norm(want)
    print(f"{name}/{variant}: max {mx:.2e} mean {mean:.2e} rel {rel:.2e}")
    assert rel < (1e-5 if cfg.dtype == "f32" else 1e-2)


@pytest.mark.parametrize("geo", [
    dict(H=12, W=20, n=3, i=1, p=0.5),      # ragged: 80 queries, 120 keys
    dict(H=12, W=20, n=3, i=0, p=1.0),      # top band, whole neighbour
    dict(H=12, W=20, n=3, i=2, p=0.34),     # bottom band, fractional p*h
    dict(H=1, W=1, n=1, i=0, p=0.0),        # one query, one key
    dict(H=6, W=7, n=1, i=0, p=0.5),        # n = 1: full-image attention
    dict(H=32, W=48, n=2, i=1, p=0.3),      # the paper's 2-band split, p*h fractional
    dict(H=64, W=64, n=4, i=2, p=0.0),      # p = 0: band-local attention
    dict(H=40, W=72, n=4, i=1, p=0.8),      # the paper's p for 8 devices
])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_attention_edge_geometries(geo, dtype):
    cfg = synth.AttnConfig(name="edge", heads=3, d=64, dtype=dtype, seed_id=40, **geo)
    _say("edge", geo, dtype)
    inp = synth.attention_inputs(cfg, "sharp")
    got = gu.to_f64(gu.run_attention(cfg, inp))
    gu.assert_close(cfg, got, gu.oracle_attention(cfg, inp), str(geo))


@pytest.mark.parametrize("batch", [2, 3])
def test_attention_batched(batch):
    cfg = _cfg("sdxl1024_l1", batch=batch, H=32, W=32)
    _say("batched", batch)
    inp = synth.attention_inputs(cfg)
    got = gu.to_f64(gu.run_attention(cfg, inp))
    gu.assert_close(cfg, got, gu.oracle_attention(cfg, inp), "batched")


@pytest.mark.parametrize("band", [0, 3])
def test_attention_level2_guidance_pair(band):
    """Both guidance branches of a step in one launch (batch 2) at the full
    2048 px level-2 shape (64 x 64 grid, 20 heads), an edge and an interior
    band: every output element against the oracle."""
    cfg = _cfg("sdxl2048_l2_edge", batch=2, i=band)
    _say("level-2 guidance pair, band", band)
    inp = synth.attention_inputs(cfg)
    got = gu.to_f64(gu.run_attention(cfg, inp))
    gu.assert_close(cfg, got, gu.oracle_attention(cfg, inp), f"l2 batch 2 band {band}")


def test_attention_f32_at_workload_shape():
    cfg = _cfg("sdxl1024_l1", dtype="f32")
    _say("f32 at 1024px level-1 shape")
    inp = synth.attention_inputs(cfg)
    got = gu.to_f64(gu.run_attention(cfg, inp))
    gu.assert_close(cfg, got, gu.oracle_attention(cfg, inp), "f32 big")


def _monotone_score_inputs(cfg, slope, rng):
    """Inputs whose scores rise (slope > 0) or fall (slope < 0) along the
    image rows of the key context: every query of head h points along one
    unit direction u_h, and the keys of image row R are slope * R * u_h plus
    noise, so each later row's scores exceed the earlier ones' by a fixed
    margin.  float64 draws, returned in the stored dtype."""
    from paper_2412_02962_amd import synth as sy
    h_rows, W, C, d = cfg.h, cfg.W, cfg.C, cfg.d
    u = rng.standard_normal((cfg.heads, d))
    u /= np.linalg.norm(u, axis=1, keepdims=True)
    u_full = u.reshape(C)

    def band(j, kind):
        x = 0.3 * rng.standard_normal((cfg.batch, h_rows * W, C))
        if kind == "q":
            x += 3.0 * u_full
        elif kind == "k":
            rows = j * h_rows + np.arange(h_rows * W) // W      # image row of each token
            base = abs(slope) * (rows if slope > 0 else (cfg.H - 1 - rows))
            x += base[None, :, None] * u_full[None, None, :]
        return sy.store(x, cfg.dtype)

    i = cfg.i
    out = {"q": band(i, "q"), "k_fresh": band(i, "k"), "v_fresh": band(i, "v")}
    for tag, j in (("up", i - 1), ("dn", i + 1)):
        ok = 0 <= j < cfg.n
        out["k_" + tag] = band(j, "k") if ok else None
        out["v_" + tag] = band(j, "v") if ok else None
    return out


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("slope", [10.0, -10.0])
def test_running_max_rises_across_the_keys(dtype, slope):
    """The online softmax's late rescale: with slope 10 the scores of each key
    row exceed the row before by about 5.4 in log2 units, so within a key piece
    the running maximum taken from its first half-tile is passed by 20 and more
    several times (each time the maximum is raised and O and l are rescaled),
    and the key pieces of a block end with maxima tens of log2 units apart
    before they are merged.  With slope -10 the first keys dominate and the
    later probabilities underflow.  Both against the float64 oracle."""
    cfg = synth.AttnConfig(name="rise", H=32, W=64, n=4, i=1, p=0.5, heads=2, d=64, dtype=dtype, seed_id=77)
    _say("monotone scores", dtype, slope)
    rng = np.random.default_rng(4100 + int(slope) + (0 if dtype == "bf16" else 1))
    inp = _monotone_score_inputs(cfg, slope, rng)
    got = gu.to_f64(gu.run_attention(cfg, inp))
    want = gu.oracle_attention(cfg, inp)
    assert np.isfinite(got).all()
    mx, mean = gu.assert_close(cfg, got, want, f"monotone {slope} {dtype}")
    print(f"monotone scores slope {slope} {dtype}: max {mx:.2e} mean {mean:.2e}")


def test_step_does_not_change_the_result():
    import torch
    cfg = synth.ATTN_CONFIGS["sdxl1024_l1"]
    _say("step independence")
    inp = synth.attention_inputs(cfg)
    a = gu.run_attention(cfg, inp, g=gu.geom(cfg, step=0))
    b = gu.run_attention(cfg, inp, g=gu.geom(cfg, step=37))
    assert torch.equal(a, b)


def test_stale_rows_outside_window_never_read():
    cfg = synth.ATTN_CONFIGS["sdxl2048_l1_p25"]
    _say("NaN outside window")
    inp = synth.attention_inputs(cfg)
    ref = gu.run_attention(cfg, inp)
    h, W, C = cfg.h, cfg.W, cfg.C
    r = 4
    bad = dict(inp)
    nan = np.uint16(0x7FC0)
    for key in ("k_up", "v_up"):
        x = inp[key].copy()
        x[:, :(h - r) * W] = nan
        bad[key] = x
    for key in ("k_dn", "v_dn"):
        x = inp[key].copy()
        x[:, r * W:] = nan
        bad[key] = x
    got = gu.run_attention(cfg, bad)
    assert bool((got == ref).all())


def test_workspace_reuse_across_geometries():
    # one zero-filled workspace serves calls of different geometries in a row:
    # the per-block work counters must come back to zero after every call
    import torch
    from paper_2412_02962_amd import pcpp
    names = ["sdxl2048_l1_p50", "sdxl1024_l1", "sdxl2048_l2_edge", "sdxl2048_l1_p50", "sdxl1024_l1"]
    cfgs = [synth.ATTN_CONFIGS[n] for n in names]
    need = max(pcpp.pcpp_partial_attention_workspace_size(gu.geom(c)) for c in cfgs)
    ws = torch.zeros(need, dtype=torch.uint8, device=gu.DEV)
    for n, cfg in zip(names, cfgs):
        _say("reuse", n)
        inp = synth.attention_inputs(cfg)
        d = {k: gu.to_dev(v, cfg.dtype) for k, v in inp.items()}
        out = torch.empty_like(d["q"])
        pcpp.pcpp_partial_attention(gu.geom(cfg), d["q"], d["k_fresh"], d["v_fresh"], d["k_up"], d["v_up"],
                                    d["k_dn"], d["v_dn"], out, ws, need)
        torch.cuda.synchronize()
        gu.assert_close(cfg, gu.to_f64(out), gu.oracle_attention(cfg, inp), f"reuse {n}")


def test_graph_replays_match_eager():
    import torch
    from paper_2412_02962_amd import pcpp
    cfg = synth.ATTN_CONFIGS["sdxl2048_l1_p25"]
    _say("graph replays")
    inp = synth.attention_inputs(cfg)
    d = {k: gu.to_dev(v, cfg.dtype) for k, v in inp.items()}
    g = gu.geom(cfg)
    wsb = pcpp.pcpp_partial_attention_workspace_size(g)
    ws = torch.zeros(wsb, dtype=torch.uint8, device=gu.DEV)
    out = torch.empty_like(d["q"])

    def call():
        pcpp.pcpp_partial_attention(g, d["q"], d["k_fresh"], d["v_fresh"], d["k_up"], d["v_up"], d["k_dn"],
                                    d["v_dn"], out, ws, wsb)

    call()
    torch.cuda.synchronize()
    eager = out.clone()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        call()
    for rep in range(3):
        out.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager), f"replay {rep} differs"
        call()  # eager work between replays on the same workspace
        torch.cuda.synchronize()
        assert torch.equal(out, eager)


def test_virtual_patches_each_match_oracle():
    # every band of one image, run one after another on the same GPU
    base = synth.AttnConfig(name="virt", H=32, W=24, n=4, i=0, p=0.5, heads=2, d=64, dtype="bf16", seed_id=41)
    for i in range(base.n):
        cfg = dataclasses.replace(base, i=i)
        _say("virtual band", i)
        inp = synth.attention_inputs(cfg)
        gu.assert_close(cfg, gu.to_f64(gu.run_attention(cfg, inp)), gu.oracle_attention(cfg, inp), f"band {i}")


def test_largest_workload_sampled_rows():
    # 3840 px level-1 grid (240 x 240, 640 channels) on 2 bands, p = 0.3:
    # 28800 queries x 37440 keys; the oracle checks a sample of query rows
    cfg = synth.AttnConfig(name="3840", H=240, W=240, n=2, i=0, p=0.3, heads=10, d=64, dtype="bf16",
                           seed_id=42)
    _say("3840px level-1, sampled")
    inp = synth.attention_inputs(cfg)
    out = gu.run_attention(cfg, inp)
    assert bool(out.isfinite().all())
    got = gu.to_f64(out)
    # every workgroup block of queries: its first and last row and one more
    rows = gu.block_rows(cfg.n_q, gu.attention_block_queries(cfg), np.random.default_rng(5))
    f = {k: oracle.as_f64(v, cfg.dtype) for k, v in inp.items()}
    want = oracle.partial_attention(cfg.H, cfg.W, cfg.n, cfg.i, cfg.p, cfg.heads, f["q"][:, rows],
                                    f["k_fresh"], f["v_fresh"], f["k_up"], f["v_up"], f["k_dn"], f["v_dn"])
    gu.assert_close(cfg, got[:, rows], want, "3840 sampled")


@pytest.mark.parametrize("name", list(synth.ATTN_CONFIGS))
def test_gather_is_bit_exact(name):
    import torch
    from paper_2412_02962_amd import pcpp
    cfg = synth.ATTN_CONFIGS[name]
    _say("gather", name)
    inp = synth.attention_inputs(cfg)
    g = gu.geom(cfg)
    h, up, dn, nkv = pcpp.pcpp_context_rows(g)
    d = {k: gu.to_dev(v, cfg.dtype) for k, v in inp.items()}
    idx = torch.full((nkv,), -1, dtype=torch.int32, device=gu.DEV)
    kc = torch.empty((cfg.batch, nkv, cfg.C), dtype=d["k_fresh"].dtype, device=gu.DEV)
    vc = torch.empty_like(kc)
    pcpp.pcpp_gather_context(g, d["k_fresh"], d["v_fresh"], d["k_up"], d["v_up"], d["k_dn"], d["v_dn"],
                             idx, kc, vc)
    torch.cuda.synchronize()
    want_idx = oracle.context_token_ids(cfg.H, cfg.W, cfg.n, cfg.i, cfg.p)
    assert np.array_equal(idx.cpu().numpy(), want_idx)
    for got, key in ((kc, "k"), (vc, "v")):
        want = oracle.assemble_context(cfg.H, cfg.W, cfg.n, cfg.i, cfg.p, inp[key + "_fresh"],
                                       inp[key + "_up"], inp[key + "_dn"])
        raw = got.cpu()
        raw = raw.view(torch.int16).numpy().view(np.uint16) if cfg.dtype == "bf16" else raw.numpy()
        assert np.array_equal(raw, want), key


def test_gather_index_only_and_unaligned_width():
    import torch
    from paper_2412_02962_amd import pcpp
    cfg = synth.AttnConfig(name="g", H=15, W=3, n=5, i=2, p=0.67, heads=1, d=4, dtype="bf16", seed_id=43)
    _say("gather odd sizes")
    inp = synth.attention_inputs(cfg)
    g = gu.geom(cfg)
    _, _, _, nkv = pcpp.pcpp_context_rows(g)
    d = {k: gu.to_dev(v, cfg.dtype) for k, v in inp.items()}
    idx = torch.full((nkv,), -1, dtype=torch.int32, device=gu.DEV)
    pcpp.pcpp_gather_context(g, None, None, None, None, None, None, idx, None, None)
    kc = torch.empty((1, nkv, cfg.C), dtype=torch.bfloat16, device=gu.DEV)
    vc = torch.empty_like(kc)
    pcpp.pcpp_gather_context(g, d["k_fresh"], d["v_fresh"], d["k_up"], d["v_up"], d["k_dn"], d["v_dn"],
                             None, kc, vc)
    torch.cuda.synchronize()
    assert np.array_equal(idx.cpu().numpy(), oracle.context_token_ids(cfg.H, cfg.W, cfg.n, cfg.i, cfg.p))
    want = oracle.assemble_context(cfg.H, cfg.W, cfg.n, cfg.i, cfg.p, inp["v_fresh"], inp["v_up"], inp["v_dn"])
    assert np.array_equal(vc.cpu().view(torch.int16).numpy().view(np.uint16), want)


@pytest.mark.parametrize("name", list(synth.PAPER_GEOMETRIES))
def test_paper_geometries(name):
    # the paper's band splits (n = 2 at p = 0.3, n = 4 at p = 0.8) on both SDXL
    # self-attention grids at 1024, 2048 and 3840 px; fractional p*h throughout.
    # Large shapes are checked on a sample of query rows.
    cfg = synth.PAPER_GEOMETRIES[name]
    _say("paper geometry", name)
    inp = synth.attention_inputs(cfg)
    out = gu.run_attention(cfg, inp)
    assert bool(out.isfinite().all())
    got = gu.to_f64(out)
    f = {k: oracle.as_f64(v, cfg.dtype) for k, v in inp.items()}
    if cfg.n_q <= 1024:
        rows = np.arange(cfg.n_q)
    else:  # every workgroup block of queries: first, last and two more rows
        rows = gu.block_rows(cfg.n_q, gu.attention_block_queries(cfg), np.random.default_rng(6), extra=2)
    want = oracle.partial_attention(cfg.H, cfg.W, cfg.n, cfg.i, cfg.p, cfg.heads, f["q"][:, rows],
                                    f["k_fresh"], f["v_fresh"], f["k_up"], f["v_up"], f["k_dn"], f["v_dn"])
    gu.assert_close(cfg, got[:, rows], want, name)


def test_workspace_reuse_with_multi_wave_launches():
    # shapes whose pieces run in several waves of workgroups share one
    # workspace with one-wave shapes; the counters must come back to zero
    import torch
    from paper_2412_02962_amd import pcpp
    names = ["paper_2048_l1_n2_p0.3", "sdxl2048_l1_p25", "paper_2048_l1_n4_p0.8", "sdxl1024_l1",
             "paper_2048_l2_n2_p0.3", "sdxl2048_l1_p25"]
    allc = dict(synth.ATTN_CONFIGS)
    allc.update(synth.PAPER_GEOMETRIES)
    cfgs = [allc[n] for n in names]
    need = max(pcpp.pcpp_partial_attention_workspace_size(gu.geom(c)) for c in cfgs)
    ws = torch.zeros(need, dtype=torch.uint8, device=gu.DEV)
    rows_rng = np.random.default_rng(8)
    for n, cfg in zip(names, cfgs):
        _say("reuse (waves)", n)
        inp = synth.attention_inputs(cfg)
        d = {k: gu.to_dev(v, cfg.dtype) for k, v in inp.items()}
        out = torch.empty_like(d["q"])
        pcpp.pcpp_partial_attention(gu.geom(cfg), d["q"], d["k_fresh"], d["v_fresh"], d["k_up"], d["v_up"],
                                    d["k_dn"], d["v_dn"], out, ws, need)
        torch.cuda.synchronize()
        assert bool(out.isfinite().all())
        rows = gu.block_rows(cfg.n_q, gu.attention_block_queries(cfg), rows_rng)
        f = {k: oracle.as_f64(v, cfg.dtype) for k, v in inp.items()}
        want = oracle.partial_attention(cfg.H, cfg.W, cfg.n, cfg.i, cfg.p, cfg.heads, f["q"][:, rows],
                                        f["k_fresh"], f["v_fresh"], f["k_up"], f["v_up"], f["k_dn"], f["v_dn"])
        gu.assert_close(cfg, gu.to_f64(out)[:, rows], want, f"reuse {n}")
    assert int(ws[:65536 * 4].view(torch.int32).abs().sum().item()) == 0   # counters left zero


@pytest.mark.parametrize("geo", [
    dict(H=64, W=64, n=8, i=3, p=1.5, heads=10),     # 24 rows each side: bands i-1 and i-2
    dict(H=64, W=64, n=8, i=1, p=2.5, heads=10),     # clipped above (8 rows), 20 rows below
    dict(H=32, W=24, n=4, i=2, p=3.0, heads=3),      # p = n - 1: the whole image
    dict(H=40, W=20, n=5, i=0, p=1.3, heads=2),      # top band, fractional p*h
])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_multihop_attention_matches_oracle(geo, dtype):
    import torch
    from paper_2412_02962_amd import pcpp
    cfg = synth.AttnConfig(name="mh", d=64, dtype=dtype, seed_id=45, **geo)
    _say("multi-hop", geo, dtype)
    inp = gu.multihop_inputs(cfg)
    d = {k: gu.to_dev(v, cfg.dtype) for k, v in inp.items()}
    g = gu.geom(cfg)
    wsb = pcpp.pcpp_partial_attention_multihop_workspace_size(g)
    ws = torch.zeros(max(wsb, 1), dtype=torch.uint8, device=gu.DEV)
    out = torch.empty_like(d["q"])
    pcpp.pcpp_partial_attention_multihop(g, d["q"], d["k_fresh"], d["v_fresh"], d["k_above"], d["v_above"],
                                         d["k_below"], d["v_below"], out, ws, wsb)
    torch.cuda.synchronize()
    f = {k: (None if v is None else oracle.as_f64(v, cfg.dtype)) for k, v in inp.items()}
    want = oracle.partial_attention_multihop(cfg.H, cfg.W, cfg.n, cfg.i, cfg.p, cfg.heads, f["q"], f["k_fresh"],
                                             f["v_fresh"], f["k_above"], f["v_above"], f["k_below"], f["v_below"])
    gu.assert_close(cfg, gu.to_f64(out), want, f"multi-hop {geo}")


def test_multihop_equals_neighbour_form_for_p_up_to_one():
    # same kernel, same rows: bit-identical to pcpp_partial_attention
    import torch
    from paper_2412_02962_amd import pcpp
    cfg = synth.ATTN_CONFIGS["sdxl2048_l1_p25"]
    _say("multi-hop p <= 1")
    inp = synth.attention_inputs(cfg)
    ref = gu.run_attention(cfg, inp)
    h, up, dn, _ = oracle.context_rows(cfg.H, cfg.n, cfg.i, cfg.p)
    d = {k: gu.to_dev(v, cfg.dtype) for k, v in inp.items()}
    W = cfg.W
    g = gu.geom(cfg)
    wsb = pcpp.pcpp_partial_attention_multihop_workspace_size(g)
    ws = torch.zeros(wsb, dtype=torch.uint8, device=gu.DEV)
    out = torch.empty_like(d["q"])
    pcpp.pcpp_partial_attention_multihop(g, d["q"], d["k_fresh"], d["v_fresh"],
                                         d["k_up"][:, (h - up) * W:].contiguous(), d["v_up"][:, (h - up) * W:].contiguous(),
                                         d["k_dn"][:, :dn * W].contiguous(), d["v_dn"][:, :dn * W].contiguous(), out, ws, wsb)
    torch.cuda.synchronize()
    assert torch.equal(out, ref)


def test_plan_splits_on_the_default_stream():
    """The CU-mask query works on this device: an unmasked stream gets the
    split plan the bench workload needs (pieces merged per XCD)."""
    from paper_2412_02962_amd import pcpp
    cfg = synth.ATTN_CONFIGS["sdxl2048_l1_p25"]
    _say("plan on the default stream")
    bq, k, wg = pcpp.pcpp_partial_attention_plan(gu.geom(cfg))
    cus = torch_cus()
    assert (bq, k, wg) == pcpp.pcpp_partial_attention_plan(gu.geom(cfg), cus, cus)
    assert k > 1


def torch_cus():
    import torch
    return torch.cuda.get_device_properties(0).multi_processor_count


def _masked_stream(n_enabled):
    """A HIP stream restricted to the first n_enabled compute units."""
    import ctypes

    import torch
    hip = ctypes.CDLL("libamdhip64.so")
    words = (torch_cus() + 31) // 32
    mask = (ctypes.c_uint32 * words)()
    for c in range(n_enabled):
        mask[c // 32] |= 1 << (c % 32)
    s = ctypes.c_void_p()
    assert hip.hipExtStreamCreateWithCUMask(ctypes.byref(s), ctypes.c_uint32(words), mask) == 0
    return hip, s


@pytest.mark.parametrize("name", ["sdxl2048_l1_p25", "sdxl2048_l2_edge"])
def test_attention_on_a_cu_masked_stream_runs_unsplit(name):
    """On a stream with a CU mask the dispatch of workgroups to XCDs is not
    known: the launch computes whole blocks (no merge through an L2) and
    still matches the oracle."""
    import torch
    from paper_2412_02962_amd import pcpp
    cfg = synth.ATTN_CONFIGS[name]
    _say("CU-masked stream", name)
    hip, s = _masked_stream(torch_cus() // 2)
    try:
        assert pcpp.pcpp_partial_attention_plan(gu.geom(cfg), stream=s.value)[1] == 1
        inp = synth.attention_inputs(cfg)
        out = gu.run_attention(cfg, inp, stream=s.value)
        assert hip.hipStreamSynchronize(s) == 0
        gu.assert_close(cfg, gu.to_f64(out), gu.oracle_attention(cfg, inp), f"masked {name}")
        torch.cuda.synchronize()
    finally:
        hip.hipStreamDestroy(s)
