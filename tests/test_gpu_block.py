"""GPU parity of pcpp_transformer_block against the float64 oracle block,
through the C ABI, on seeded random-init SDXL-shaped weights.

Tolerance: the GPU block stores the activations that feed each GEMM in bf16
(GroupNorm/LayerNorm outputs, Q/K/V, attention outputs, the GEGLU hidden
state) and rounds the output to bf16; the residual stream and every
accumulation stay in float32.  Each bf16 rounding is a relative error of at
most 2^-8 of that tensor.  The output rounding alone is up to 2^-8 |y|; the
six rounded intermediates add errors of the same relative size to the
branch outputs, which enter y through the residual sum.  The bound used is
|dy| <= 2^-8 |y| + 6 * 2^-8 * rms(y) per element, with a mean absolute error
below 2^-8 * rms(y).  The exported K and V sit behind three roundings (the
GroupNorm output, the LayerNorm output and K/V themselves), so they use the
same form with 3 in place of 6.  (The 2e-2 / 2e-3 tolerances of the
attention kernel apply to attention outputs, whose magnitude is the
weighted mean of values; K and V are unit-scale projections.)
"""

import dataclasses

import numpy as np
import pytest

import oracle
from paper_2412_02962_amd import synth
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu


def _say(*a):
    print("[case]", *a, flush=True)


def _run_block(bc, inp, batch, want_kv=True):
    import torch
    from paper_2412_02962_amd import pcpp
    cfg = bc.attn
    dev = gu.DEV
    d = {k: gu.to_dev(v, "bf16") for k, v in inp.items()}
    g = pcpp.make_geom(cfg.H, cfg.W, cfg.n, cfg.i, cfg.p, cfg.heads, cfg.d, batch, 0, pcpp.PCPP_DTYPE_BF16)
    w = pcpp.make_block_weights(d, bc.ff_inner, bc.gn_groups)
    y = torch.empty_like(d["x"])
    k_out = torch.empty_like(d["x"]) if want_kv else None
    v_out = torch.empty_like(d["x"]) if want_kv else None
    wsb = pcpp.pcpp_transformer_block_workspace_size(g, w, bc.n_text, bc.text_dim)
    assert wsb > 0
    ws = torch.zeros(wsb, dtype=torch.uint8, device=dev)
    pcpp.pcpp_transformer_block(g, w, d["x"], d["text"], bc.n_text, bc.text_dim, d["k_up"], d["v_up"],
                                d["k_dn"], d["v_dn"], y, k_out, v_out, ws, wsb)
    torch.cuda.synchronize()
    return y, k_out, v_out


def _oracle_block(bc, inp):
    cfg = bc.attn
    f = {k: (None if v is None else oracle.from_bf16_bits(v)) for k, v in inp.items()}
    wts = {k: f[k] for k in synth.block_weight_shapes(bc)}
    return oracle.transformer_block(cfg.H, cfg.W, cfg.n, cfg.i, cfg.p, cfg.heads, wts, f["x"], f["text"],
                                    f["k_up"], f["v_up"], f["k_dn"], f["v_dn"], gn_groups=bc.gn_groups)


def _check(y, want, stages=6, tag="block"):
    """The block's derived bound (module docstring)."""
    err = np.abs(y - want)
    rms = float(np.sqrt(np.mean(want ** 2)))
    bound = 2.0 ** -8 * np.abs(want) + stages * 2.0 ** -8 * rms
    worst = float((err / bound).max())
    mean = float(err.mean())
    mean_bound = 2.0 ** -8 * rms
    print(f"{tag}: max-abs {err.max():.3e}, worst err/bound {worst:.3f}, mean-abs {mean:.3e}, rms {rms:.3f} "
          f"(the attention tolerances would be 2e-2 / 2e-3)")
    assert worst <= 1.0, f"{tag}: max error exceeds bound by {worst:.2f}x"
    assert mean <= mean_bound, f"{tag}: mean-abs {mean:.3e} > {mean_bound:.3e}"


def _check_kv(got, want, tag):
    _check(got, want, stages=3, tag=tag)


@pytest.mark.parametrize("bc", [synth.BLOCK_CONFIG, synth.BLOCK_CONFIG_L2], ids=lambda b: b.name)
def test_block_matches_oracle_at_2048px(bc):
    _say("block", bc.name)
    inp = synth.block_inputs(bc)
    y, k, v = _run_block(bc, inp, 1)
    want_y, want_k, want_v = _oracle_block(bc, inp)
    _check(gu.to_f64(y), want_y)
    _check_kv(gu.to_f64(k), want_k, "k export")
    _check_kv(gu.to_f64(v), want_v, "v export")


@pytest.mark.parametrize("geo", [
    dict(H=12, W=20, n=3, i=1, p=0.5, heads=2),     # 80 tokens, ragged tiles
    dict(H=16, W=16, n=4, i=0, p=0.25, heads=3),    # top band, C = 192
    dict(H=16, W=16, n=4, i=3, p=1.0, heads=2),     # bottom band, whole neighbour
])
@pytest.mark.parametrize("batch", [1, 2])
def test_block_small_shapes(geo, batch):
    attn = synth.AttnConfig(name="blk", d=64, dtype="bf16", seed_id=50, **geo)
    bc = synth.BlockConfig(name="blk", attn=attn, n_text=7, text_dim=96, ff_inner=128,
                           gn_groups=4, seed_id=51)
    _say("block small", geo, batch)
    inp = synth.block_inputs(bc, batch=batch)
    y, k, v = _run_block(bc, inp, batch)
    want_y, want_k, want_v = _oracle_block(bc, inp)
    _check(gu.to_f64(y), want_y)
    _check_kv(gu.to_f64(k), want_k, "k export")
    _check_kv(gu.to_f64(v), want_v, "v export")


@pytest.mark.parametrize("batch", [1, 2])
def test_block_split_k_gemms(batch):
    """FF-out (K = 2048) and the text K/V product (K = 2048) split K over two
    workgroups per tile at these sizes (fewer 64 x 64 tiles than compute
    units, 32 k-tiles); 80 tokens per image leave a ragged last token tile."""
    attn = synth.AttnConfig(name="blk", H=12, W=20, n=3, i=1, p=0.5, heads=2, d=64, dtype="bf16", seed_id=56)
    bc = synth.BlockConfig(name="blk", attn=attn, n_text=7, text_dim=2048, ff_inner=2048, gn_groups=4,
                           seed_id=57)
    _say("block split-K", batch)
    inp = synth.block_inputs(bc, batch=batch)
    y, k, v = _run_block(bc, inp, batch)
    want_y, want_k, want_v = _oracle_block(bc, inp)
    _check(gu.to_f64(y), want_y)
    _check_kv(gu.to_f64(k), want_k, "k export")
    _check_kv(gu.to_f64(v), want_v, "v export")


@pytest.mark.parametrize("n_text", [1, 64, 96, 97])
def test_block_cross_attention_text_lengths(n_text):
    """64 tokens per band: up to 96 text tokens the cross-attention runs
    inside its Q product (keys past the text masked: 1, 64 and 96 fill one,
    two and all three 32-key blocks), 97 goes to the separate Q product and
    attention launch."""
    attn = synth.AttnConfig(name="blk", H=16, W=16, n=4, i=1, p=0.25, heads=2, d=64, dtype="bf16", seed_id=58)
    bc = synth.BlockConfig(name="blk", attn=attn, n_text=n_text, text_dim=64, ff_inner=128, gn_groups=4,
                           seed_id=59)
    _say("block text length", n_text)
    inp = synth.block_inputs(bc, batch=2)
    y, k, v = _run_block(bc, inp, 2)
    want_y, want_k, want_v = _oracle_block(bc, inp)
    _check(gu.to_f64(y), want_y)
    _check_kv(gu.to_f64(k), want_k, "k export")


def test_block_balanced_tiles_with_a_ragged_last_tile():
    """2000 tokens of 640 channels (one band of 100 x 20): the 640-wide
    products and Q/K/V run on 64 x 80 tiles and the GEGLU on 128 x 160 tiles,
    each with a ragged last token tile (2000 = 31 x 64 + 16 = 15 x 128 + 80);
    the GroupNorm and the cross-attention take their separate launches (the
    band is not whole 64-token tiles)."""
    attn = synth.AttnConfig(name="blk", H=100, W=20, n=1, i=0, p=0.0, heads=10, d=64, dtype="bf16", seed_id=60)
    bc = synth.BlockConfig(name="blk", attn=attn, seed_id=61)
    _say("block ragged balanced tiles")
    inp = synth.block_inputs(bc)
    y, k, v = _run_block(bc, inp, 1)
    want_y, want_k, want_v = _oracle_block(bc, inp)
    _check(gu.to_f64(y), want_y)
    _check_kv(gu.to_f64(k), want_k, "k export")
    _check_kv(gu.to_f64(v), want_v, "v export")


def test_block_level2_geglu_tiles_with_a_ragged_last_tile():
    """A level-2 band of 8 x 62 = 496 tokens of 1280 channels: the GEGLU
    product (2 x 5120 outputs) runs on 64-token x 160-output tiles in
    XCD-contiguous order, the last token tile ragged (496 = 7 x 64 + 48)."""
    attn = synth.AttnConfig(name="blk", H=64, W=62, n=8, i=3, p=0.25, heads=20, d=64, dtype="bf16", seed_id=62)
    bc = synth.BlockConfig(name="blk", attn=attn, ff_inner=5120, seed_id=63)
    _say("block level-2 ragged GEGLU tiles")
    inp = synth.block_inputs(bc)
    y, k, v = _run_block(bc, inp, 1)
    want_y, want_k, want_v = _oracle_block(bc, inp)
    _check(gu.to_f64(y), want_y)
    _check_kv(gu.to_f64(k), want_k, "k export")


def test_block_workspace_is_reusable():
    """Workspace contract: no clearing needed.  The attention's and the split
    GEMMs' counters live there (the level-2 block splits FF-out and the text
    K/V product); three calls on one workspace filled with garbage give the
    same bits as a call on a zeroed one."""
    import torch
    from paper_2412_02962_amd import pcpp
    bc = synth.BLOCK_CONFIG_L2
    cfg = bc.attn
    _say("block dirty workspace", bc.name)
    d = {k: gu.to_dev(v, "bf16") for k, v in synth.block_inputs(bc).items()}
    g = pcpp.make_geom(cfg.H, cfg.W, cfg.n, cfg.i, cfg.p, cfg.heads, cfg.d, 1, 0, pcpp.PCPP_DTYPE_BF16)
    w = pcpp.make_block_weights(d, bc.ff_inner, bc.gn_groups)
    wsb = pcpp.pcpp_transformer_block_workspace_size(g, w, bc.n_text, bc.text_dim)
    outs = []
    shared = torch.full((wsb,), 0xC3, dtype=torch.uint8, device=gu.DEV)
    for ws in (torch.zeros(wsb, dtype=torch.uint8, device=gu.DEV), shared, shared, shared):
        y = torch.empty_like(d["x"])
        pcpp.pcpp_transformer_block(g, w, d["x"], d["text"], bc.n_text, bc.text_dim, d["k_up"], d["v_up"],
                                    d["k_dn"], d["v_dn"], y, None, None, ws, wsb)
        torch.cuda.synchronize()
        outs.append(y)
    assert all(torch.equal(outs[0], o) for o in outs[1:])


def test_block_without_kv_export_gives_same_output():
    import torch
    attn = synth.AttnConfig(name="blk", H=16, W=16, n=4, i=1, p=0.5, heads=2, d=64, dtype="bf16", seed_id=52)
    bc = synth.BlockConfig(name="blk", attn=attn, n_text=5, text_dim=64, ff_inner=192, gn_groups=8, seed_id=53)
    _say("block no export")
    inp = synth.block_inputs(bc)
    y1, _, _ = _run_block(bc, inp, 1, want_kv=True)
    y2, _, _ = _run_block(bc, inp, 1, want_kv=False)
    assert torch.equal(y1, y2)


def _other_band_stats(cfg, G, B, seed):
    """(count, mean, M2) of synthetic GroupNorm inputs of every other band
    (each band with its own offset and scale), float32-rounded as passed to
    the library; entry cfg.i is NaN: it must not be read."""
    rng = np.random.default_rng(seed)
    st = np.full((cfg.n, B, G, 3), np.nan)
    for j in range(cfg.n):
        if j != cfg.i:
            xj = 0.3 * j + (1.0 + 0.1 * j) * rng.standard_normal((B, cfg.n_q, cfg.C))
            st[j] = oracle.group_stats(xj, G)
    return st.astype(np.float32)


@pytest.mark.parametrize("which", ["2048", "small_b2"])
def test_block_synchronized_group_norm(which):
    import torch
    from paper_2412_02962_amd import pcpp
    if which == "2048":
        bc, B = synth.BLOCK_CONFIG, 1
    else:
        attn = synth.AttnConfig(name="blk", H=16, W=16, n=4, i=2, p=0.5, heads=2, d=64, dtype="bf16", seed_id=54)
        bc, B = synth.BlockConfig(name="blk", attn=attn, n_text=5, text_dim=64, ff_inner=128, gn_groups=8,
                                  seed_id=55), 2
    cfg = bc.attn
    _say("block synchronized GroupNorm", which)
    inp = synth.block_inputs(bc, batch=B)
    st = _other_band_stats(cfg, bc.gn_groups, B, 12)
    d = {k: gu.to_dev(v, "bf16") for k, v in inp.items()}
    g = pcpp.make_geom(cfg.H, cfg.W, cfg.n, cfg.i, cfg.p, cfg.heads, cfg.d, B, 0, pcpp.PCPP_DTYPE_BF16)
    w = pcpp.make_block_weights(d, bc.ff_inner, bc.gn_groups)
    y, k_out, v_out = (torch.empty_like(d["x"]) for _ in range(3))
    own = torch.empty((B, bc.gn_groups, 3), dtype=torch.float32, device=gu.DEV)
    bands = torch.from_numpy(st).to(gu.DEV)
    wsb = pcpp.pcpp_transformer_block_workspace_size(g, w, bc.n_text, bc.text_dim)
    ws = torch.zeros(wsb, dtype=torch.uint8, device=gu.DEV)
    pcpp.pcpp_transformer_block_sync_gn(g, w, d["x"], d["text"], bc.n_text, bc.text_dim, d["k_up"], d["v_up"],
                                        d["k_dn"], d["v_dn"], bands, own, y, k_out, v_out, ws, wsb)
    torch.cuda.synchronize()
    f = {k: (None if v is None else oracle.from_bf16_bits(v)) for k, v in inp.items()}
    wts = {k: f[k] for k in synth.block_weight_shapes(bc)}
    want_y, want_k, want_v = oracle.transformer_block(cfg.H, cfg.W, cfg.n, cfg.i, cfg.p, cfg.heads, wts, f["x"],
                                                      f["text"], f["k_up"], f["v_up"], f["k_dn"], f["v_dn"],
                                                      gn_groups=bc.gn_groups, gn_band_stats=st.astype(np.float64))
    _check(gu.to_f64(y), want_y, tag="sync-GN block")
    _check_kv(gu.to_f64(k_out), want_k, "sync-GN k export")
    want_own = oracle.group_stats(f["x"], bc.gn_groups)
    got_own = own.cpu().numpy().astype(np.float64)
    assert np.array_equal(got_own[..., 0], want_own[..., 0])
    assert np.allclose(got_own[..., 1], want_own[..., 1], rtol=0, atol=1e-5)
    assert np.allclose(got_own[..., 2], want_own[..., 2], rtol=1e-4, atol=0)
    # the band-local block differs (the statistics are not this band's alone)
    y_local, _, _ = _run_block(bc, inp, B)
    assert not torch.equal(y_local, y)


# ---------------------------------------------------------------------------
# Transformer module of depth d (each basic block its own weights and stale K/V)
# ---------------------------------------------------------------------------

def _run_module(bc, x, text, module, blocks, stale, batch, gn_bands=None, want_own=False):
    import torch
    from paper_2412_02962_amd import pcpp
    cfg = bc.attn
    dv = lambda a: None if a is None else gu.to_dev(a, "bf16")
    g = pcpp.make_geom(cfg.H, cfg.W, cfg.n, cfg.i, cfg.p, cfg.heads, cfg.d, batch, 0, pcpp.PCPP_DTYPE_BF16)
    md = {k: dv(v) for k, v in module.items()}
    bd = [{k: dv(v) for k, v in b.items()} for b in blocks]
    w, keep = pcpp.make_module_weights(md, bd, bc.ff_inner, bc.gn_groups)
    xd, td = dv(x), dv(text)
    st = [[dv(a) for a in s] for s in stale]
    cols = list(zip(*st))                                   # k_up list, v_up list, ...
    lists = [None if any(a is None for a in c) else list(c) for c in cols]
    y = torch.empty_like(xd)
    ko = [torch.empty_like(xd) for _ in blocks]
    vo = [torch.empty_like(xd) for _ in blocks]
    own = torch.empty((batch, bc.gn_groups, 3), dtype=torch.float32, device=gu.DEV) if want_own else None
    wsb = pcpp.pcpp_transformer_module_workspace_size(g, w, bc.n_text, bc.text_dim)
    assert wsb > 0
    ws = torch.zeros(wsb, dtype=torch.uint8, device=gu.DEV)
    pcpp.pcpp_transformer_module(g, w, xd, td, bc.n_text, bc.text_dim, *lists, gn_bands, own, y, ko, vo, ws, wsb)
    torch.cuda.synchronize()
    del keep
    return y, ko, vo, own


def _oracle_module(bc, x, text, module, blocks, stale, gn_band_stats=None):
    cfg = bc.attn
    f = lambda a: None if a is None else oracle.from_bf16_bits(a)
    return oracle.transformer_module(cfg.H, cfg.W, cfg.n, cfg.i, cfg.p, cfg.heads, {k: f(v) for k, v in module.items()},
                                     [{k: f(v) for k, v in b.items()} for b in blocks], f(x), f(text),
                                     [tuple(f(a) for a in s) for s in stale], gn_groups=bc.gn_groups,
                                     gn_band_stats=gn_band_stats)


def test_module_of_depth_one_is_the_block():
    import torch
    bc = synth.BLOCK_CONFIG
    _say("module depth 1 = block")
    x, text, module, blocks, stale = synth.module_inputs(bc, 1)
    y, ko, vo, _ = _run_module(bc, x, text, module, blocks, stale, 1)
    inp = dict(module)
    inp.update(blocks[0])
    inp.update({"x": x, "text": text, "k_up": stale[0][0], "v_up": stale[0][1], "k_dn": stale[0][2],
                "v_dn": stale[0][3]})
    yb, kb, vb = _run_block(bc, inp, 1)
    assert torch.equal(y, yb) and torch.equal(ko[0], kb) and torch.equal(vo[0], vb)


MODULE_CASES = [
    (synth.BLOCK_CONFIG, 2, 1),
    (dataclasses.replace(synth.BLOCK_CONFIG, attn=synth.AttnConfig(name="m_small", H=12, W=20, n=3, i=1, p=0.5,
                                                                   heads=2, d=64, dtype="bf16", seed_id=77),
                         ff_inner=256, text_dim=64, n_text=7, seed_id=77), 3, 2),
    # the text K/V of 16 blocks in one product, then of the last 2
    (dataclasses.replace(synth.BLOCK_CONFIG, attn=synth.AttnConfig(name="m_deep", H=12, W=20, n=3, i=2, p=0.75,
                                                                   heads=2, d=64, dtype="bf16", seed_id=78),
                         ff_inner=128, text_dim=128, n_text=5, seed_id=78), 18, 2),
]


@pytest.mark.parametrize("case", MODULE_CASES, ids=["l1_2048_depth2", "small_depth3_b2", "small_depth18_b2"])
def test_module_matches_oracle(case):
    bc, depth, batch = case
    _say("module", bc.attn.name, depth, batch)
    x, text, module, blocks, stale = synth.module_inputs(bc, depth, batch=batch)
    y, ko, vo, _ = _run_module(bc, x, text, module, blocks, stale, batch)
    want_y, want_k, want_v = _oracle_module(bc, x, text, module, blocks, stale)
    _check_module(bc, depth, y, ko, vo, want_y, want_k, want_v)


def _check_module(bc, depth, y, ko, vo, want_y, want_k, want_v):
    """Element-wise bounds of a module (tests.gpu_util.check_composition):
    six roundings per basic block on the way to y; block j's K and V sit
    behind the GroupNorm, LayerNorm and K/V roundings plus six per earlier
    block (counted as four: the bound's tail factor is calibrated for a
    million elements, and a module's K and V are that many)."""
    gu.check_composition(gu.to_f64(y), want_y, 6 * depth, f"module y depth {depth}")
    for j in range(depth):
        gu.check_composition(gu.to_f64(ko[j]), want_k[j], 4 + 6 * j, f"k export {j}")
        gu.check_composition(gu.to_f64(vo[j]), want_v[j], 4 + 6 * j, f"v export {j}")


def test_level2_module_on_a_garbage_workspace():
    """SDXL's level-2 transformer module at 2048 px (depth 10, 1280 channels,
    band 3 of 8: 512 tokens, 640 keys; key pieces merged per XCD, split-K
    GEMMs, the text K/V of the ten blocks in one grouped product) on a
    workspace filled with garbage: the module clears the work counters its
    launches use, so a workspace shared with other layers' scratch is fine."""
    import torch
    from paper_2412_02962_amd import pcpp
    bc, depth = synth.BLOCK_CONFIG_L2, 10
    cfg = bc.attn
    _say("level-2 module, depth 10, garbage workspace")
    x, text, module, blocks, stale = synth.module_inputs(bc, depth)
    dv = lambda a: None if a is None else gu.to_dev(a, "bf16")
    g = pcpp.make_geom(cfg.H, cfg.W, cfg.n, cfg.i, cfg.p, cfg.heads, cfg.d, 1, 0, pcpp.PCPP_DTYPE_BF16)
    assert pcpp.pcpp_partial_attention_plan(g)[1] > 1           # the merge path is exercised
    md = {k: dv(v) for k, v in module.items()}               # device weights, alive for the whole test
    bd = [{k: dv(v) for k, v in b.items()} for b in blocks]
    w, keep = pcpp.make_module_weights(md, bd, bc.ff_inner, bc.gn_groups)
    xd, td = dv(x), dv(text)
    cols = list(zip(*[[dv(a) for a in s_] for s_ in stale]))
    lists = [None if any(a is None for a in c) else list(c) for c in cols]
    wsb = pcpp.pcpp_transformer_module_workspace_size(g, w, bc.n_text, bc.text_dim)
    ws = torch.full((wsb,), 0xA5, dtype=torch.uint8, device=gu.DEV)
    outs = []
    for rep in range(2):
        y = torch.empty_like(xd)
        ko = [torch.empty_like(xd) for _ in blocks]
        vo = [torch.empty_like(xd) for _ in blocks]
        pcpp.pcpp_transformer_module(g, w, xd, td, bc.n_text, bc.text_dim, *lists, None, None, y, ko, vo, ws, wsb)
        torch.cuda.synchronize()
        outs.append((y, ko, vo))
        ws.fill_(0x5A)                                           # other garbage for the second call
    assert torch.equal(outs[0][0], outs[1][0])
    want_y, want_k, want_v = _oracle_module(bc, x, text, module, blocks, stale)
    _check_module(bc, depth, *outs[0], want_y, want_k, want_v)
    del keep, md, bd


def test_module_bound_rejects_a_planted_mistake():
    """Negative control, planted in the oracle on the CPU: basic block 1
    reads block 0's stale K/V (the wrong layer's receive buffer).  That
    oracle is further from the GPU result than the module bound allows."""
    bc, depth, batch = MODULE_CASES[1]
    _say("module negative control")
    x, text, module, blocks, stale = synth.module_inputs(bc, depth, batch=batch)
    y, ko, vo, _ = _run_module(bc, x, text, module, blocks, stale, batch)
    bad = [stale[0], stale[0]] + list(stale[2:])
    want_y, _, _ = _oracle_module(bc, x, text, module, blocks, bad)
    with pytest.raises(AssertionError):
        gu.check_composition(gu.to_f64(y), want_y, 6 * depth, "planted mistake")


def test_module_synchronized_group_norm():
    import torch
    bc, depth, batch = MODULE_CASES[1]
    _say("module sync GN")
    x, text, module, blocks, stale = synth.module_inputs(bc, depth, batch=batch)
    rng = np.random.default_rng(5)
    cfg = bc.attn
    st = np.stack([oracle.group_stats(0.3 * rng.standard_normal() + rng.standard_normal((batch, cfg.h * cfg.W, cfg.C)),
                                      bc.gn_groups) for _ in range(cfg.n)])
    bands = torch.from_numpy(st.astype(np.float32)).to(gu.DEV)
    y, _, _, own = _run_module(bc, x, text, module, blocks, stale, batch, gn_bands=bands, want_own=True)
    want_y, _, _ = _oracle_module(bc, x, text, module, blocks, stale, gn_band_stats=st)
    gu.check_composition(gu.to_f64(y), want_y, 6 * depth, "module sync GN")
    want_own = oracle.group_stats(oracle.from_bf16_bits(x), bc.gn_groups)
    assert np.allclose(own.double().cpu().numpy()[..., 1], want_own[..., 1], atol=1e-5)
