"""Pins of the oracle's boundary messages (Sec. 3.2 with Eq. 1), CPU only.

  B1  the rows a message carries are exactly the patch's tokens that the
      receiving neighbour's context holds, by the brute-force Eq. 1 mask
      (exact rationals, 1-based patches), keys and values alike
  B2  placing the messages a patch receives into otherwise-NaN stale
      buffers reproduces the context assembled from the whole neighbour
      patches, for every band
  B3  placing leaves every other row of the stale buffers as it was
"""

import numpy as np
import pytest

import oracle
from tests.oracle_pins_util import eq1_token_ids_brute

PS = [0.0, 0.1, 0.25, 0.3, 0.5, 0.8, 1.0]


def _id_tensors(H, W, n, i, B=2, C=3):
    """k[b, t, c] = global token id of token t of band i (+ 1000 b), v = -k."""
    h = H // n
    ids = i * h * W + np.arange(h * W, dtype=np.float64)
    k = np.broadcast_to(ids[None, :, None], (B, h * W, C)) + 1000.0 * np.arange(B)[:, None, None]
    return np.ascontiguousarray(k), -np.ascontiguousarray(k)


@pytest.mark.parametrize("n", [1, 2, 3, 4, 6])
@pytest.mark.parametrize("h", [1, 3, 4, 7])
@pytest.mark.parametrize("W", [1, 3])
def test_messages_carry_the_rows_the_neighbours_read(n, h, W):
    H = n * h
    for p in PS:
        for i in range(n):
            k, v = _id_tensors(H, W, n, i)
            band = set(range(i * h * W, (i + 1) * h * W))
            to_up, to_dn = oracle.boundary_messages(H, W, n, i, p, k, v)
            for msg, j in ((to_up, i - 1), (to_dn, i + 1)):
                want = ([] if not 0 <= j < n else
                        sorted(set(eq1_token_ids_brute(H, W, n, j, p).tolist()) & band))
                if not want:
                    assert msg is None, (n, h, W, p, i, j)
                    continue
                assert msg.shape == (2, 2, len(want), 3)
                for b in range(2):
                    got = msg[b, 0, :, 0] - 1000.0 * b
                    assert got.tolist() == [float(x) for x in want], (n, h, W, p, i, j)
                    assert np.array_equal(msg[b, 1], -msg[b, 0])
                    assert np.array_equal(msg[b, 0, :, 1], msg[b, 0, :, 0])


@pytest.mark.parametrize("geo", [
    dict(H=12, W=5, n=3, p=0.5),
    dict(H=16, W=4, n=4, p=0.25),
    dict(H=20, W=3, n=2, p=0.3),
    dict(H=40, W=2, n=4, p=0.8),
    dict(H=8, W=6, n=4, p=1.0),
])
def test_placed_messages_reproduce_the_whole_band_context(geo):
    H, W, n, p = geo["H"], geo["W"], geo["n"], geo["p"]
    h, B, C = H // n, 2, 4
    rng = np.random.default_rng(3)
    prev = [(rng.standard_normal((B, h * W, C)), rng.standard_normal((B, h * W, C))) for _ in range(n)]
    fresh = [(rng.standard_normal((B, h * W, C)), rng.standard_normal((B, h * W, C))) for _ in range(n)]
    msgs = [oracle.boundary_messages(H, W, n, j, p, *prev[j]) for j in range(n)]
    nan = np.full((B, h * W, C), np.nan)
    for i in range(n):
        from_up = msgs[i - 1][1] if i > 0 else None
        from_dn = msgs[i + 1][0] if i < n - 1 else None
        ku, vu, kd, vd = oracle.place_boundary_messages(H, W, n, i, p, from_up, from_dn, nan, nan, nan, nan)
        for t, (fk, up_whole, dn_whole, up_placed, dn_placed) in enumerate((
                (fresh[i][0], prev[i - 1][0] if i > 0 else None, prev[i + 1][0] if i < n - 1 else None, ku, kd),
                (fresh[i][1], prev[i - 1][1] if i > 0 else None, prev[i + 1][1] if i < n - 1 else None, vu, vd))):
            want = oracle.assemble_context(H, W, n, i, p, fk, up_whole, dn_whole)
            got = oracle.assemble_context(H, W, n, i, p, fk, up_placed, dn_placed)
            assert not np.isnan(got).any(), (geo, i, t)
            assert np.array_equal(got, want), (geo, i, t)


def test_placing_keeps_the_other_rows():
    H, W, n, p, i = 16, 3, 4, 0.5, 1
    h, B, C = 4, 1, 2
    rng = np.random.default_rng(4)
    bufs = [rng.standard_normal((B, h * W, C)) for _ in range(4)]
    up_msg = rng.standard_normal((B, 2, 2 * W, C))
    dn_msg = rng.standard_normal((B, 2, 2 * W, C))
    ku, vu, kd, vd = oracle.place_boundary_messages(H, W, n, i, p, up_msg, dn_msg, *bufs)
    assert np.array_equal(ku[:, :2 * W], bufs[0][:, :2 * W]) and np.array_equal(ku[:, 2 * W:], up_msg[:, 0])
    assert np.array_equal(vu[:, :2 * W], bufs[1][:, :2 * W]) and np.array_equal(vu[:, 2 * W:], up_msg[:, 1])
    assert np.array_equal(kd[:, 2 * W:], bufs[2][:, 2 * W:]) and np.array_equal(kd[:, :2 * W], dn_msg[:, 0])
    assert np.array_equal(vd[:, 2 * W:], bufs[3][:, 2 * W:]) and np.array_equal(vd[:, :2 * W], dn_msg[:, 1])
    for a, b in zip(bufs, (ku, vu, kd, vd)):
        assert a is not b


# ---------------------------------------------------------------------------
# Planted mistakes: each must fail the checks above (CPU, monkeypatched)
# ---------------------------------------------------------------------------

def _battery():
    try:
        for n, h, W in ((3, 4, 2), (4, 3, 3), (2, 5, 1)):
            test_messages_carry_the_rows_the_neighbours_read(n, h, W)
        test_placed_messages_reproduce_the_whole_band_context(dict(H=16, W=4, n=4, p=0.5))
        test_placed_messages_reproduce_the_whole_band_context(dict(H=20, W=3, n=2, p=0.3))
    except AssertionError:
        return False
    return True


def test_unmodified_oracle_passes_the_boundary_battery():
    assert _battery()


def _msgs_shifted(H, W, n, i, p, k, v):        # rows one further into the band
    h = H // n
    up, dn = _ORIG_MSGS(H, W, n, i, p, k, v)
    r = None if up is None else up.shape[2] // W
    if up is not None and r < h:
        up = np.stack([k[:, W:(r + 1) * W], v[:, W:(r + 1) * W]], axis=1)
    return up, dn


def _msgs_swapped(H, W, n, i, p, k, v):        # directions exchanged
    up, dn = _ORIG_MSGS(H, W, n, i, p, k, v)
    if up is not None and dn is not None:
        return dn, up
    return up, dn


def _msgs_keys_twice(H, W, n, i, p, k, v):     # keys sent in place of values
    up, dn = _ORIG_MSGS(H, W, n, i, p, k, v)
    fix = lambda m: None if m is None else np.stack([m[:, 0], m[:, 0]], axis=1)
    return fix(up), fix(dn)


def _place_at_band_start(H, W, n, i, p, fu, fd, ku, vu, kd, vd):   # stale-above rows at the wrong end
    h, up, dn, _ = oracle.context_rows(H, n, i, p)
    ku, vu, kd, vd = (None if a is None else np.array(a, copy=True) for a in (ku, vu, kd, vd))
    if up > 0:
        ku[:, :up * W] = fu[:, 0]
        vu[:, :up * W] = fu[:, 1]
    if dn > 0:
        kd[:, :dn * W] = fd[:, 0]
        vd[:, :dn * W] = fd[:, 1]
    return ku, vu, kd, vd


_ORIG_MSGS = oracle.boundary_messages


@pytest.mark.parametrize("name,mutant", [
    ("boundary_messages", _msgs_shifted),
    ("boundary_messages", _msgs_swapped),
    ("boundary_messages", _msgs_keys_twice),
    ("place_boundary_messages", _place_at_band_start),
])
def test_planted_boundary_mistakes_are_caught(monkeypatch, name, mutant):
    monkeypatch.setattr(oracle, name, mutant)
    assert not _battery()


# ---------------------------------------------------------------------------
# Multi-hop messages (p > 1): every patch within reach gets the rows it reads
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("n,h,W", [(4, 3, 2), (6, 2, 3), (8, 4, 1), (3, 5, 2)])
def test_multihop_messages_carry_the_rows_each_patch_reads(n, h, W):
    from fractions import Fraction
    H = n * h
    for p in [q for q in (0.5, 1.0, 1.5, 2.3, float(n - 1)) if q <= max(1, n - 1)]:
        r = int(Fraction(str(p)) * h // 1)
        for i in range(n):
            k, v = _id_tensors(H, W, n, i)
            band = set(range(i * h * W, (i + 1) * h * W))
            for j in range(n):
                if j == i:
                    continue
                # brute force: image rows within r of patch j, every column
                ctx = {row * W + c for row in range(H) if j * h - r <= row < (j + 1) * h + r for c in range(W)}
                want = sorted(ctx & band)
                msg = oracle.multihop_message(H, W, n, i, p, j, k, v)
                if not want:
                    assert msg is None, (n, h, p, i, j)
                    continue
                assert msg is not None and msg.shape[2] == len(want), (n, h, p, i, j)
                assert (msg[0, 0, :, 0]).tolist() == [float(x) for x in want], (n, h, p, i, j)
                assert np.array_equal(msg[:, 1], -msg[:, 0])
                if abs(i - j) == 1 and p <= 1.0:
                    up_msg, dn_msg = oracle.boundary_messages(H, W, n, i, p, k, v)
                    assert np.array_equal(msg, up_msg if j < i else dn_msg)


@pytest.mark.parametrize("n,h,W,p", [(6, 3, 2, 1.5), (8, 2, 3, 2.5), (4, 4, 2, 3.0), (5, 3, 1, 0.7)])
def test_placed_multihop_messages_rebuild_the_stale_rows(n, h, W, p):
    H, B, C = n * h, 2, 3
    rng = np.random.default_rng(7)
    prev = [(rng.standard_normal((B, h * W, C)), rng.standard_normal((B, h * W, C))) for _ in range(n)]
    grid_k = np.concatenate([x[0] for x in prev], axis=1)
    grid_v = np.concatenate([x[1] for x in prev], axis=1)
    for i in range(n):
        _, up, dn, _ = oracle.context_rows_multihop(H, n, i, p)
        bufs = [np.full((B, up * W, C), np.nan), np.full((B, up * W, C), np.nan),
                np.full((B, dn * W, C), np.nan), np.full((B, dn * W, C), np.nan)]
        for j in range(n):
            if j == i:
                continue
            msg = oracle.multihop_message(H, W, n, j, p, i, *prev[j])
            assert (msg is None) == (oracle.multihop_message_rows(H, n, j, p, i)[0] == 0)
            if msg is not None:
                bufs = list(oracle.place_multihop_message(H, W, n, i, p, j, msg, *bufs))
        assert np.array_equal(bufs[0], grid_k[:, (i * h - up) * W:i * h * W])
        assert np.array_equal(bufs[1], grid_v[:, (i * h - up) * W:i * h * W])
        assert np.array_equal(bufs[2], grid_k[:, (i + 1) * h * W:((i + 1) * h + dn) * W])
        assert np.array_equal(bufs[3], grid_v[:, (i + 1) * h * W:((i + 1) * h + dn) * W])


def _multihop_battery():
    try:
        for n, h, W in ((4, 3, 2), (6, 2, 3)):
            test_multihop_messages_carry_the_rows_each_patch_reads(n, h, W)
        for n, h, W, p in ((6, 3, 2, 1.5), (8, 2, 3, 2.5)):
            test_placed_multihop_messages_rebuild_the_stale_rows(n, h, W, p)
    except AssertionError:
        return False
    return True


def test_unmodified_oracle_passes_the_multihop_battery():
    assert _multihop_battery()


_ORIG_HOP_ROWS = oracle.multihop_message_rows
_ORIG_HOP_MSG = oracle.multihop_message
_ORIG_HOP_PLACE = oracle.place_multihop_message


def _hop_rows_one_hop_short(H, n, i, p, j):       # (|i-j|) h subtracted instead of (|i-j|-1) h
    rows, first = _ORIG_HOP_ROWS(H, n, i, p, j)
    h = H // n
    return (max(0, rows - h) if abs(i - j) > 1 else rows), first


def _hop_msg_wrong_end(H, W, n, i, p, j, k, v):    # first rows where the last are read
    rows, first = oracle.multihop_message_rows(H, n, i, p, j)
    if rows == 0:
        return None
    h = H // n
    sl = slice((h - rows) * W, h * W) if first else slice(0, rows * W)
    return np.stack([k[:, sl], v[:, sl]], axis=1)


def _hop_place_unshifted(H, W, n, i, p, j, msg, ka, va, kb, vb):   # every message at the block's start
    rows, _ = oracle.multihop_message_rows(H, n, j, p, i)
    ka, va, kb, vb = (None if a is None else np.array(a, copy=True) for a in (ka, va, kb, vb))
    if rows:
        tk, tv = (ka, va) if j < i else (kb, vb)
        tk[:, :rows * W] = msg[:, 0]
        tv[:, :rows * W] = msg[:, 1]
    return ka, va, kb, vb


@pytest.mark.parametrize("name,mutant", [
    ("multihop_message_rows", _hop_rows_one_hop_short),
    ("multihop_message", _hop_msg_wrong_end),
    ("place_multihop_message", _hop_place_unshifted),
])
def test_planted_multihop_mistakes_are_caught(monkeypatch, name, mutant):
    import oracle.pcpp_oracle as mod
    monkeypatch.setattr(oracle, name, mutant)
    monkeypatch.setattr(mod, name, mutant)      # the oracle's own calls go through the module
    assert not _multihop_battery()
