"""GPU parity of the p-aware boundary messages (pcpp_pack_boundary,
pcpp_unpack_boundary) against the float64 oracle, through the C ABI: both are
pure data movement, so the bar is bit-exact."""

import dataclasses

import numpy as np
import pytest

import oracle
from paper_2412_02962_amd import synth
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

GEOS = [
    dict(H=128, W=128, n=8, i=3, p=0.25, heads=10, batch=1),   # the 2048 px level-1 band
    dict(H=64, W=64, n=8, i=0, p=0.25, heads=20, batch=1),     # top band: one message
    dict(H=64, W=64, n=8, i=7, p=0.25, heads=20, batch=2),     # bottom band, two images
    dict(H=32, W=48, n=2, i=1, p=0.3, heads=3, batch=1),       # fractional p*h
    dict(H=40, W=72, n=4, i=1, p=0.8, heads=3, batch=3),
    dict(H=12, W=5, n=3, i=1, p=1.0, heads=1, batch=2),        # whole neighbour, odd width
]


def _say(*a):
    print("[case]", *a, flush=True)


def _cfg(geo, dtype, seed_id=50):
    return synth.AttnConfig(name="bnd", H=geo["H"], W=geo["W"], n=geo["n"], i=geo["i"], p=geo["p"],
                            heads=geo["heads"], d=64, dtype=dtype, seed_id=seed_id, batch=geo["batch"])


def _raw(t, dtype):
    import torch
    t = t.cpu()
    return t.view(torch.int16).numpy().view(np.uint16) if dtype == synth.DTYPE_BF16 else t.numpy()


def _stored(cfg, band, kind, stale):
    x = synth.patch_tensor(cfg, band, kind, stale)
    return synth.store(x, cfg.dtype)


@pytest.mark.parametrize("geo", GEOS)
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_pack_is_bit_exact(geo, dtype):
    import torch
    from paper_2412_02962_amd import pcpp
    cfg = _cfg(geo, dtype)
    _say("pack", geo, dtype)
    k, v = _stored(cfg, cfg.i, "k", False), _stored(cfg, cfg.i, "v", False)
    g = gu.geom(cfg)
    nbytes = pcpp.pcpp_boundary_bytes(g)
    want_up, want_dn = oracle.boundary_messages(cfg.H, cfg.W, cfg.n, cfg.i, cfg.p, k, v)
    tdt = torch.bfloat16 if dtype == synth.DTYPE_BF16 else torch.float32
    esize = 2 if dtype == synth.DTYPE_BF16 else 4
    send = [torch.full((max(nbytes, esize) // esize,), 7, dtype=tdt, device=gu.DEV) for _ in range(2)]
    pcpp.pcpp_pack_boundary(g, gu.to_dev(k, dtype), gu.to_dev(v, dtype), send[0], send[1])
    torch.cuda.synchronize()
    for got, want in zip(send, (want_up, want_dn)):
        raw = _raw(got, dtype)
        if want is None:
            assert (raw == _raw(torch.full((1,), 7, dtype=tdt), dtype)[0]).all()  # untouched
        else:
            assert want.size * esize == nbytes
            assert np.array_equal(raw, want.reshape(-1))


@pytest.mark.parametrize("geo", GEOS)
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_unpack_is_bit_exact_and_leaves_other_rows(geo, dtype):
    import torch
    from paper_2412_02962_amd import pcpp
    cfg = _cfg(geo, dtype)
    _say("unpack", geo, dtype)
    g = gu.geom(cfg)
    i, n = cfg.i, cfg.n
    # messages as the neighbours would build them from their previous-step tensors
    up_msg = (oracle.boundary_messages(cfg.H, cfg.W, n, i - 1, cfg.p, _stored(cfg, i - 1, "k", True),
                                       _stored(cfg, i - 1, "v", True))[1] if i > 0 else None)
    dn_msg = (oracle.boundary_messages(cfg.H, cfg.W, n, i + 1, cfg.p, _stored(cfg, i + 1, "k", True),
                                       _stored(cfg, i + 1, "v", True))[0] if i < n - 1 else None)
    # stale buffers start as some other tensor's values
    base = [_stored(cfg, (i + 2) % n, kind, False) for kind in ("k", "v", "k", "v")]
    dev = [gu.to_dev(b, dtype) for b in base]
    pcpp.pcpp_unpack_boundary(g, gu.to_dev(up_msg, dtype), gu.to_dev(dn_msg, dtype), *dev)
    torch.cuda.synchronize()
    want = oracle.place_boundary_messages(cfg.H, cfg.W, n, i, cfg.p, up_msg, dn_msg, *base)
    for got, w in zip(dev, want):
        assert np.array_equal(_raw(got, dtype), w)


@pytest.mark.parametrize("geo", [GEOS[0], GEOS[2], GEOS[4]])
def test_attention_over_exchanged_rows_only(geo):
    """Every band packs its previous-step K/V on the GPU; band i unpacks its
    two messages into stale buffers that are NaN elsewhere; the attention
    output equals the one over the whole stale neighbour bands, bit for bit."""
    import torch
    from paper_2412_02962_amd import pcpp
    cfg = _cfg(geo, "bf16")
    _say("exchange + attention", geo)
    i, n = cfg.i, cfg.n
    inp = synth.attention_inputs(cfg)
    ref = gu.run_attention(cfg, inp)
    d = {k: gu.to_dev(v, cfg.dtype) for k, v in inp.items()}
    msgs = {}
    for j, tag in ((i - 1, "up"), (i + 1, "dn")):
        if not 0 <= j < n:
            continue
        gj = gu.geom(dataclasses.replace(cfg, i=j))
        nb = pcpp.pcpp_boundary_bytes(gj)
        s_up = torch.empty(nb // 2, dtype=torch.bfloat16, device=gu.DEV)
        s_dn = torch.empty(nb // 2, dtype=torch.bfloat16, device=gu.DEV)
        # band j's previous-step K/V are exactly the stale buffer band i holds for it
        pcpp.pcpp_pack_boundary(gj, d["k_" + tag], d["v_" + tag], s_up if j > 0 else None,
                                s_dn if j < n - 1 else None)
        msgs[tag] = s_dn if tag == "up" else s_up   # band i-1 sends down, band i+1 sends up
    stale = {}
    for key in ("k_up", "v_up", "k_dn", "v_dn"):
        stale[key] = None if d[key] is None else torch.full_like(d[key], float("nan"))
    g = gu.geom(cfg)
    pcpp.pcpp_unpack_boundary(g, msgs.get("up"), msgs.get("dn"), stale["k_up"], stale["v_up"], stale["k_dn"],
                              stale["v_dn"])
    out = torch.empty_like(d["q"])
    ws_bytes = pcpp.pcpp_partial_attention_workspace_size(g)
    ws = torch.zeros(max(ws_bytes, 1), dtype=torch.uint8, device=gu.DEV)
    pcpp.pcpp_partial_attention(g, d["q"], d["k_fresh"], d["v_fresh"], stale["k_up"], stale["v_up"],
                                stale["k_dn"], stale["v_dn"], out, ws, ws_bytes)
    torch.cuda.synchronize()
    assert not torch.isnan(out).any()
    assert torch.equal(out, ref)


# ---------------------------------------------------------------------------
# Multi-hop messages (p > 1): band i sends each band within reach its rows
# ---------------------------------------------------------------------------

MH_GEOS = [
    dict(H=64, W=64, n=8, i=3, p=1.5, heads=10, batch=1),    # two bands each way, 4 of 8 rows from the far ones
    dict(H=64, W=64, n=8, i=1, p=2.5, heads=4, batch=2),     # clipped above, three bands below
    dict(H=32, W=24, n=4, i=2, p=3.0, heads=3, batch=1),     # p = n - 1: every band whole
    dict(H=40, W=20, n=5, i=0, p=1.3, heads=2, batch=3),     # top band, fractional p*h
    dict(H=48, W=16, n=6, i=4, p=0.5, heads=2, batch=1),     # p <= 1: the neighbour messages
]


def _mh_cfg(geo, dtype, seed_id=46):
    return synth.AttnConfig(name="mhx", d=64, dtype=dtype, seed_id=seed_id, **geo)


@pytest.mark.parametrize("geo", MH_GEOS)
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_pack_multihop_is_bit_exact(geo, dtype):
    import torch
    from paper_2412_02962_amd import pcpp
    cfg = _mh_cfg(geo, dtype)
    _say("pack multi-hop", geo, dtype)
    k, v = _stored(cfg, cfg.i, "k", False), _stored(cfg, cfg.i, "v", False)
    g = gu.geom(cfg)
    kd, vd = gu.to_dev(k, dtype), gu.to_dev(v, dtype)
    tdt = torch.bfloat16 if dtype == synth.DTYPE_BF16 else torch.float32
    esize = 2 if dtype == synth.DTYPE_BF16 else 4
    for j in range(cfg.n):
        want = oracle.multihop_message(cfg.H, cfg.W, cfg.n, cfg.i, cfg.p, j, k, v)
        nbytes = pcpp.pcpp_multihop_message_bytes(g, j)
        if want is None:
            assert nbytes == 0
            pcpp.pcpp_pack_multihop(g, j, None, None, None)       # nothing to send: no pointers needed
            continue
        assert want.size * esize == nbytes
        send = torch.full((nbytes // esize,), 7, dtype=tdt, device=gu.DEV)
        pcpp.pcpp_pack_multihop(g, j, kd, vd, send)
        torch.cuda.synchronize()
        assert np.array_equal(_raw(send, dtype), want.reshape(-1)), (geo, j)
        if cfg.p <= 1.0 and abs(j - cfg.i) == 1:                   # same bytes as the neighbour form
            both = [torch.zeros_like(send) for _ in range(2)]
            pcpp.pcpp_pack_boundary(g, kd, vd, both[0], both[1])
            torch.cuda.synchronize()
            assert np.array_equal(_raw(send, dtype), _raw(both[0] if j < cfg.i else both[1], dtype))


@pytest.mark.parametrize("geo", MH_GEOS[:4])
def test_multihop_exchange_then_attention(geo):
    """Every other band packs its previous-step K/V for band i on the GPU;
    band i unpacks all of them into NaN-filled compact blocks, which then
    equal the blocks cut from the whole stale image, and the multi-hop
    attention over them equals the one over the cut blocks, bit for bit."""
    import torch
    from paper_2412_02962_amd import pcpp
    cfg = _mh_cfg(geo, "bf16")
    _say("multi-hop exchange + attention", geo)
    i, n = cfg.i, cfg.n
    inp = gu.multihop_inputs(cfg)
    d = {k: gu.to_dev(v, cfg.dtype) for k, v in inp.items()}
    blocks = {key: None if d[key] is None else torch.full_like(d[key], float("nan"))
              for key in ("k_above", "v_above", "k_below", "v_below")}
    g = gu.geom(cfg)
    sent = 0
    for j in range(n):
        if j == i:
            continue
        gj = gu.geom(dataclasses.replace(cfg, i=j))
        nb = pcpp.pcpp_multihop_message_bytes(gj, i)
        assert nb == pcpp.pcpp_multihop_message_bytes(g, j)
        if nb == 0:
            continue
        kj = gu.to_dev(_stored(cfg, j, "k", True), cfg.dtype)
        vj = gu.to_dev(_stored(cfg, j, "v", True), cfg.dtype)
        msg = torch.empty(nb // 2, dtype=torch.bfloat16, device=gu.DEV)
        pcpp.pcpp_pack_multihop(gj, i, kj, vj, msg)
        pcpp.pcpp_unpack_multihop(g, j, msg, blocks["k_above"], blocks["v_above"], blocks["k_below"],
                                  blocks["v_below"])
        sent += 1
    torch.cuda.synchronize()
    assert sent > 0
    for key, blk in blocks.items():
        if blk is None:
            assert d[key] is None
            continue
        assert torch.equal(blk.view(torch.int16), d[key].view(torch.int16)), key
    wsb = pcpp.pcpp_partial_attention_multihop_workspace_size(g)
    ws = torch.zeros(wsb, dtype=torch.uint8, device=gu.DEV)
    outs = []
    for src in (blocks, d):
        out = torch.empty_like(d["q"])
        pcpp.pcpp_partial_attention_multihop(g, d["q"], d["k_fresh"], d["v_fresh"], src["k_above"], src["v_above"],
                                             src["k_below"], src["v_below"], out, ws, wsb)
        outs.append(out)
    torch.cuda.synchronize()
    assert not torch.isnan(outs[0]).any()
    assert torch.equal(outs[0], outs[1])
