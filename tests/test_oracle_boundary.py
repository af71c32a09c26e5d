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
