"""The C ABI library loads, exports every function include/pcpp.h declares,
and its host-side logic (Eq. 1 geometry, argument validation) behaves as
documented.  No compute call is made: every call here fails validation
before anything would be enqueued, or is host-only."""

import ctypes
import math
import os
import re

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pcpp.h")


def _declared():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(pcpp_[a-z0-9_]+)\s*\(", txt)))


def test_library_exports_every_declared_function():
    from paper_2412_02962_amd import pcpp
    names = _declared()
    assert len(names) >= 8
    lib = ctypes.CDLL(pcpp.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(pcpp.EXPORTED) == names


def test_version_and_strerror():
    from paper_2412_02962_amd import pcpp
    assert pcpp.pcpp_version() == 1
    for code in (0, -1, -2, -3, -4, -99):
        assert isinstance(pcpp.pcpp_strerror(code), str) and pcpp.pcpp_strerror(code)


def test_context_rows_agree_with_oracle_over_grid():
    # two independent implementations of Sec. 3.1 / Eq. 1 (C++ and Python)
    from paper_2412_02962_amd import pcpp
    ps = [0.0, 0.05, 0.1, 0.25, 0.29, 0.3, 0.33, 0.5, 0.67, 0.75, 0.8, 0.99, 1.0]
    for H in (1, 4, 8, 16, 30, 64, 100, 128, 240):
        for n in range(1, 9):
            if H % n:
                continue
            for i in range(n):
                for p in ps:
                    g = pcpp.make_geom(H, 7, n, i, p, 2)
                    h, up, dn, nkv = pcpp.pcpp_context_rows(g)
                    oh, oup, odn, rows = oracle.context_rows(H, n, i, p)
                    assert (h, up, dn, nkv) == (oh, oup, odn, rows * 7), (H, n, i, p)


@pytest.mark.parametrize("over", [
    dict(H=10, n_patches=4), dict(patch_idx=4), dict(patch_idx=-1), dict(partial=-0.1),
    dict(partial=1.5), dict(partial=math.nan), dict(n_patches=0), dict(W=0), dict(batch=0),
    dict(step=-1), dict(heads=0), dict(reserved=1),
])
def test_context_rows_rejects_invalid_geometry(over):
    from paper_2412_02962_amd import pcpp
    kw = dict(H=16, W=8, n_patches=4, patch_idx=1, partial=0.25, heads=2)
    kw.update(over)
    with pytest.raises(pcpp.PcppError) as e:
        pcpp.pcpp_context_rows(pcpp.make_geom(**kw))
    assert e.value.status == pcpp.PCPP_EINVAL


FAKE = 1 << 20  # an aligned non-null address; never dereferenced (validation fails first)


def _attn(pcpp, g, **ptrs):
    a = dict(q=FAKE, kf=FAKE, vf=FAKE, ku=FAKE, vu=FAKE, kd=FAKE, vd=FAKE, out=FAKE, ws=None, wsb=0)
    a.update(ptrs)
    return pcpp.lib().pcpp_partial_attention(ctypes.byref(g), a["q"], a["kf"], a["vf"], a["ku"], a["vu"],
                                             a["kd"], a["vd"], a["out"], a["ws"], a["wsb"], None)


def test_attention_validation_errors_before_launch():
    from paper_2412_02962_amd import pcpp
    g = pcpp.make_geom(128, 128, 8, 3, 0.25, 10)
    assert _attn(pcpp, pcpp.make_geom(128, 128, 8, 3, 0.25, 10, head_dim=128)) == pcpp.PCPP_ENOTSUP
    assert _attn(pcpp, pcpp.make_geom(128, 128, 8, 3, 0.25, 10, dtype=7)) == pcpp.PCPP_ENOTSUP
    assert _attn(pcpp, g, q=None) == pcpp.PCPP_EINVAL
    assert _attn(pcpp, g, out=None) == pcpp.PCPP_EINVAL
    assert _attn(pcpp, g, ku=None) == pcpp.PCPP_EINVAL        # needed: up = 4 rows
    assert _attn(pcpp, g, vd=None) == pcpp.PCPP_EINVAL
    assert _attn(pcpp, g, q=FAKE + 2) == pcpp.PCPP_EINVAL     # misaligned
    assert _attn(pcpp, pcpp.make_geom(128, 128, 8, 3, float("nan"), 10)) == pcpp.PCPP_EINVAL
    ws = pcpp.pcpp_partial_attention_workspace_size(g)
    if ws > 0:
        assert _attn(pcpp, g, ws=None, wsb=0) == pcpp.PCPP_EWORKSPACE
        assert _attn(pcpp, g, ws=FAKE, wsb=ws - 1) == pcpp.PCPP_EWORKSPACE


def test_workspace_size_is_zero_for_invalid_or_f32():
    from paper_2412_02962_amd import pcpp
    assert pcpp.pcpp_partial_attention_workspace_size(pcpp.make_geom(10, 8, 4, 0, 0.5, 2)) == 0
    assert pcpp.pcpp_partial_attention_workspace_size(
        pcpp.make_geom(16, 16, 4, 1, 0.25, 2, dtype=pcpp.PCPP_DTYPE_F32)) == 0


def test_gather_validation_errors_before_launch():
    from paper_2412_02962_amd import pcpp
    lib = pcpp.lib()
    g = pcpp.make_geom(16, 16, 4, 1, 0.25, 2)
    call = lambda *a: lib.pcpp_gather_context(ctypes.byref(g), *a, None)
    # nothing requested
    assert call(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, None, None) == pcpp.PCPP_EINVAL
    # one of the two outputs only
    assert call(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, None) == pcpp.PCPP_EINVAL
    # neighbour data missing while rows are needed
    assert call(FAKE, FAKE, None, FAKE, FAKE, FAKE, None, FAKE, FAKE) == pcpp.PCPP_EINVAL
    bad = pcpp.make_geom(16, 16, 4, 9, 0.25, 2)
    assert lib.pcpp_gather_context(ctypes.byref(bad), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                                   FAKE, None) == pcpp.PCPP_EINVAL


def test_binding_refuses_to_load_without_library(tmp_path, monkeypatch):
    import importlib.util
    src = os.path.join(ROOT, "paper_2412_02962_amd", "pcpp.py")
    dst = tmp_path / "pcpp.py"
    dst.write_text(open(src).read())
    spec = importlib.util.spec_from_file_location("pcpp_nolib", str(dst))
    mod = importlib.util.module_from_spec(spec)
    with pytest.raises(ImportError):
        spec.loader.exec_module(mod)


def _block_args(pcpp, **over):
    w = pcpp.pcpp_block_weights_t()
    for name, _ in pcpp.pcpp_block_weights_t._fields_[:-2]:
        setattr(w, name, FAKE)
    w.ff_inner = 2560
    w.gn_groups = 32
    a = dict(g=pcpp.make_geom(128, 128, 8, 3, 0.25, 10), w=w, x=FAKE, text=FAKE, nt=77, td=2048,
             ku=FAKE, vu=FAKE, kd=FAKE, vd=FAKE, y=FAKE, ko=None, vo=None, ws=FAKE, wsb=1 << 40)
    a.update(over)
    return a


def _block(pcpp, a):
    return pcpp.lib().pcpp_transformer_block(
        ctypes.byref(a["g"]), ctypes.byref(a["w"]), a["x"], a["text"], a["nt"], a["td"], a["ku"], a["vu"],
        a["kd"], a["vd"], a["y"], a["ko"], a["vo"], a["ws"], a["wsb"], None)


def test_block_validation_errors_before_launch():
    from paper_2412_02962_amd import pcpp
    E, N, W = pcpp.PCPP_EINVAL, pcpp.PCPP_ENOTSUP, pcpp.PCPP_EWORKSPACE
    assert _block(pcpp, _block_args(pcpp, g=pcpp.make_geom(128, 128, 8, 3, 0.25, 10, head_dim=80))) == N
    assert _block(pcpp, _block_args(pcpp, g=pcpp.make_geom(128, 128, 8, 3, 0.25, 10,
                                                           dtype=pcpp.PCPP_DTYPE_F32))) == N
    assert _block(pcpp, _block_args(pcpp, x=None)) == E
    assert _block(pcpp, _block_args(pcpp, text=None)) == E
    assert _block(pcpp, _block_args(pcpp, ku=None)) == E
    assert _block(pcpp, _block_args(pcpp, td=100)) == E           # not a multiple of 32
    assert _block(pcpp, _block_args(pcpp, nt=0)) == E
    a = _block_args(pcpp)
    a["w"].ff_inner = 100
    assert _block(pcpp, a) == E
    a = _block_args(pcpp)
    a["w"].gn_groups = 7                                             # 640 % 7 != 0
    assert _block(pcpp, a) == E
    a = _block_args(pcpp)
    a["w"].ff2_w = None
    assert _block(pcpp, a) == E
    a = _block_args(pcpp)
    a["w"].proj_in_w = FAKE + 8                                      # misaligned weight
    assert _block(pcpp, a) == E
    need = pcpp.pcpp_transformer_block_workspace_size(a["g"], _block_args(pcpp)["w"], 77, 2048)
    assert need > 0
    assert _block(pcpp, _block_args(pcpp, ws=None)) == W
    assert _block(pcpp, _block_args(pcpp, wsb=need - 1)) == W


def test_block_workspace_size_scales_with_batch_and_rejects_invalid():
    from paper_2412_02962_amd import pcpp
    w = _block_args(pcpp)["w"]
    one = pcpp.pcpp_transformer_block_workspace_size(pcpp.make_geom(128, 128, 8, 3, 0.25, 10), w, 77, 2048)
    two = pcpp.pcpp_transformer_block_workspace_size(pcpp.make_geom(128, 128, 8, 3, 0.25, 10, batch=2), w, 77,
                                                     2048)
    assert 0 < one < two <= 2 * one + 4096
    assert pcpp.pcpp_transformer_block_workspace_size(pcpp.make_geom(10, 128, 8, 3, 0.25, 10), w, 77, 2048) == 0


def test_boundary_bytes_follow_eq1_rows():
    from paper_2412_02962_amd import pcpp
    for (H, W, n, i, p, heads, B, dt, esize) in [(128, 128, 8, 3, 0.25, 10, 1, pcpp.PCPP_DTYPE_BF16, 2),
                                                 (128, 128, 8, 0, 0.25, 10, 2, pcpp.PCPP_DTYPE_BF16, 2),
                                                 (32, 48, 2, 1, 0.3, 3, 1, pcpp.PCPP_DTYPE_F32, 4),
                                                 (64, 64, 4, 2, 0.0, 1, 1, pcpp.PCPP_DTYPE_BF16, 2)]:
        g = pcpp.make_geom(H, W, n, i, p, heads, 64, B, 0, dt)
        h, up, dn, _ = oracle.context_rows(H, n, i, p)
        r = max(up, dn)
        assert pcpp.pcpp_boundary_bytes(g) == B * 2 * r * W * heads * 64 * esize
    assert pcpp.pcpp_boundary_bytes(pcpp.make_geom(10, 8, 4, 0, 0.5, 2)) == 0        # H % n != 0
    assert pcpp.pcpp_boundary_bytes(pcpp.make_geom(16, 8, 1, 0, 0.5, 2)) == 0        # one band: no neighbour


def test_layer_norm_validation_errors_before_launch():
    from paper_2412_02962_amd import pcpp
    lib = pcpp.lib()
    ln = lambda rows, C, eps, x, g, b, y: lib.pcpp_layer_norm(rows, C, eps, x, g, b, y, None)
    A = FAKE
    Y = FAKE + (1 << 30)
    assert ln(0, 640, 1e-5, A, A, A, Y) == pcpp.PCPP_EINVAL                # no rows
    assert ln((1 << 24) + 1, 640, 1e-5, A, A, A, Y) == pcpp.PCPP_EINVAL    # too many rows
    assert ln(16, 640, 0.0, A, A, A, Y) == pcpp.PCPP_EINVAL                # eps must be positive
    assert ln(16, 642, 1e-5, A, A, A, Y) == pcpp.PCPP_ENOTSUP              # channels not a multiple of 4
    assert ln(16, 4096, 1e-5, A, A, A, Y) == pcpp.PCPP_ENOTSUP             # channels beyond 2048
    assert ln(16, 640, 1e-5, None, A, A, Y) == pcpp.PCPP_EINVAL            # missing input
    assert ln(16, 640, 1e-5, A + 8, A, A, Y) == pcpp.PCPP_EINVAL           # misaligned input
    assert ln(16, 640, 1e-5, A, A, A, A + 64) == pcpp.PCPP_EINVAL          # output overlaps the input


def test_boundary_validation_errors_before_launch():
    from paper_2412_02962_amd import pcpp
    lib = pcpp.lib()
    g = pcpp.make_geom(16, 16, 4, 1, 0.25, 2)   # interior band, r = 1
    pack = lambda *a: lib.pcpp_pack_boundary(ctypes.byref(g), *a, None)
    unpack = lambda *a: lib.pcpp_unpack_boundary(ctypes.byref(g), *a, None)
    A, Bp = FAKE, FAKE + (1 << 30)
    assert pack(None, Bp, A + (1 << 31), A + (1 << 32)) == pcpp.PCPP_EINVAL      # keys missing
    assert pack(A, Bp, None, A + (1 << 32)) == pcpp.PCPP_EINVAL                  # message for band i-1 missing
    assert pack(A, Bp, A + 64, A + (1 << 32)) == pcpp.PCPP_EINVAL                # message overlaps the keys
    assert pack(A, Bp, A + (1 << 31), A + (1 << 31) + 64) == pcpp.PCPP_EINVAL    # messages overlap
    assert unpack(A, None, Bp, Bp + (1 << 26), Bp + (2 << 26), Bp + (3 << 26)) == pcpp.PCPP_EINVAL
    assert unpack(A, A + (1 << 26), Bp, Bp + 64, Bp + (2 << 26), Bp + (3 << 26)) == pcpp.PCPP_EINVAL
    # nothing to send or receive: a valid no-op without pointers
    none = pcpp.make_geom(16, 16, 4, 1, 0.0, 2)
    assert lib.pcpp_pack_boundary(ctypes.byref(none), None, None, None, None, None) == pcpp.PCPP_OK
    assert lib.pcpp_unpack_boundary(ctypes.byref(none), None, None, None, None, None, None, None) == pcpp.PCPP_OK
    bad = pcpp.make_geom(16, 16, 4, 4, 0.25, 2)
    assert lib.pcpp_pack_boundary(ctypes.byref(bad), A, Bp, FAKE, FAKE, None) == pcpp.PCPP_EINVAL


def test_multihop_geometry_and_validation():
    from paper_2412_02962_amd import pcpp
    lib = pcpp.lib()
    # p > 1 is rejected by the neighbour form and accepted (up to n - 1) by the multi-hop form
    g = pcpp.make_geom(64, 64, 8, 3, 1.5, 10)
    assert pcpp.pcpp_partial_attention_workspace_size(g) == 0
    assert pcpp.pcpp_partial_attention_multihop_workspace_size(g) > 0
    assert pcpp.pcpp_partial_attention_multihop_workspace_size(pcpp.make_geom(64, 64, 8, 3, 7.5, 10)) == 0
    call = lambda gg, *a: lib.pcpp_partial_attention_multihop(ctypes.byref(gg), *a, None)
    # rows above needed but missing
    assert call(g, FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 30) == pcpp.PCPP_EINVAL
    # misaligned output
    assert call(g, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE + 2, FAKE, 1 << 30) == pcpp.PCPP_EINVAL
    # workspace too small
    assert call(g, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 16) == pcpp.PCPP_EWORKSPACE


def test_multihop_message_bytes_match_the_oracle_rows():
    from paper_2412_02962_amd import pcpp
    for (H, W, n, p, heads, B) in [(64, 64, 8, 1.5, 2, 1), (48, 8, 6, 2.5, 1, 2), (32, 16, 4, 3.0, 1, 1),
                                   (64, 64, 8, 0.25, 2, 1), (16, 4, 2, 1.0, 1, 3)]:
        for i in range(n):
            g = pcpp.make_geom(H, W, n, i, p, heads, 64, B)
            for j in range(n):
                rows, _ = oracle.multihop_message_rows(H, n, i, p, j)
                rows_back, _ = oracle.multihop_message_rows(H, n, j, p, i)
                assert rows == rows_back                      # the same count in both directions
                assert pcpp.pcpp_multihop_message_bytes(g, j) == B * 2 * rows * W * heads * 64 * 2, (H, n, p, i, j)
            # p <= 1: the neighbour messages are the boundary messages
            if p <= 1.0 and 0 < i:
                assert pcpp.pcpp_multihop_message_bytes(g, i - 1) == pcpp.pcpp_boundary_bytes(g)
    g = pcpp.make_geom(64, 64, 8, 3, 1.5, 2)
    assert pcpp.pcpp_multihop_message_bytes(g, 8) == 0 and pcpp.pcpp_multihop_message_bytes(g, -1) == 0


def test_multihop_message_validation_errors_before_launch():
    from paper_2412_02962_amd import pcpp
    lib = pcpp.lib()
    g = pcpp.make_geom(64, 64, 8, 3, 1.5, 2)    # h = 8, r = 12: bands 1, 2, 4, 5 in reach
    pack = lambda peer, *a: lib.pcpp_pack_multihop(ctypes.byref(g), peer, *a, None)
    unpack = lambda peer, *a: lib.pcpp_unpack_multihop(ctypes.byref(g), peer, *a, None)
    A, Bp = FAKE, FAKE + (1 << 30)
    assert pack(8, A, Bp, A + (1 << 31)) == pcpp.PCPP_EINVAL              # no band 8
    assert pack(2, None, Bp, A + (1 << 31)) == pcpp.PCPP_EINVAL           # keys missing
    assert pack(2, A, Bp, None) == pcpp.PCPP_EINVAL                       # message missing
    assert pack(2, A, Bp, Bp + 64) == pcpp.PCPP_EINVAL                    # message overlaps the values
    assert pack(0, None, None, None) == pcpp.PCPP_OK                      # band 0 is out of reach
    assert pack(3, None, None, None) == pcpp.PCPP_OK                      # itself
    assert unpack(1, A, None, None, Bp, Bp + (1 << 26)) == pcpp.PCPP_EINVAL   # block above missing
    assert unpack(5, A, Bp, Bp + (1 << 26), None, None) == pcpp.PCPP_EINVAL   # block below missing
    assert unpack(1, A, Bp, Bp + 64, None, None) == pcpp.PCPP_EINVAL          # keys and values overlap
    assert unpack(1, Bp + 64, Bp, Bp + (1 << 26), None, None) == pcpp.PCPP_EINVAL  # message overlaps keys
    assert unpack(7, None, None, None, None, None) == pcpp.PCPP_OK
    f64 = pcpp.make_geom(64, 64, 8, 3, 1.5, 2, 64, 1, 0, 7)
    assert lib.pcpp_pack_multihop(ctypes.byref(f64), 2, A, Bp, A + (1 << 31), None) != pcpp.PCPP_OK


def test_resnet_geometry_and_validation():
    from paper_2412_02962_amd import pcpp
    lib = pcpp.lib()
    g = pcpp.make_resnet_geom(128, 128, 8, 3, 640, 640, 1280, 32, 1)
    ws = pcpp.pcpp_resnet_block_workspace_size(g)
    framed = 1 * 18 * 130 * 640 * 2
    assert ws >= 2 * framed + 16 * 128 * 640 * 2 + 640 * 4
    g2 = pcpp.make_resnet_geom(128, 128, 8, 3, 320, 640, 1280, 32, 1)
    assert pcpp.pcpp_resnet_block_workspace_size(g2) >= 16 * 128 * 640 * 4       # float32 shortcut
    bad = [pcpp.make_resnet_geom(100, 128, 8, 3, 640, 640),         # H % n
           pcpp.make_resnet_geom(128, 128, 8, 8, 640, 640),         # band index
           pcpp.make_resnet_geom(128, 128, 8, 3, 640, 640, 1284),   # T % 8
           pcpp.make_resnet_geom(128, 128, 8, 3, 640, 640, 1280, 48),   # groups do not divide
           pcpp.make_resnet_geom(128, 128, 8, 3, 640, 640, eps=0.0),
           pcpp.make_resnet_geom(128, 128, 8, 3, 640, 640, reserved=1)]
    for b in bad:
        assert pcpp.pcpp_resnet_block_workspace_size(b) == 0
    for c_in, c_out in ((96, 96), (640, 2624)):
        gg = pcpp.make_resnet_geom(64, 64, 4, 1, c_in, c_out, groups=32)
        assert pcpp.pcpp_resnet_block_workspace_size(gg) == 0
        assert lib.pcpp_resnet_block(ctypes.byref(gg), ctypes.byref(pcpp.pcpp_resnet_weights_t()), *([None] * 14),
                                     0, None) == pcpp.PCPP_ENOTSUP
    w = pcpp.make_resnet_weights({k: FAKE for k in pcpp.RESNET_PTR_FIELDS if not k.startswith("skip")})
    call = lambda gg, ww, *a: lib.pcpp_resnet_block(ctypes.byref(gg), ctypes.byref(ww), *a, None)
    big = 1 << 30
    ok_args = [FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, None, None, None, FAKE, None, None, FAKE, big]
    assert call(g, w, *ok_args[:-2], None, big) == pcpp.PCPP_EWORKSPACE
    assert call(g, w, *ok_args[:-2], FAKE, 16) == pcpp.PCPP_EWORKSPACE
    a = list(ok_args); a[2] = None                                   # band 3 needs the rows above
    assert call(g, w, *a) == pcpp.PCPP_EINVAL
    a = list(ok_args); a[0] = FAKE + 2                               # misaligned x
    assert call(g, w, *a) == pcpp.PCPP_EINVAL
    a = list(ok_args); a[6] = FAKE + 2                               # misaligned statistics
    assert call(g, w, *a) == pcpp.PCPP_EINVAL
    assert call(g2, w, *ok_args) == pcpp.PCPP_EINVAL                 # 320 -> 640 needs the shortcut weights
    a = list(ok_args); a[2] = FAKE + (1 << 28); a[11] = FAKE + (1 << 28) + 4096   # export over the rows above
    assert call(g, w, *a) == pcpp.PCPP_EINVAL


def test_guided_step_validation():
    from paper_2412_02962_amd import pcpp
    lib = pcpp.lib()
    call = lambda sp, n, *a: lib.pcpp_guided_step(ctypes.byref(sp), n, *a, None)
    ddpm = pcpp.make_step_params(pcpp.PCPP_STEP_DDPM, 5.0, alpha_t=0.99, alphabar_t=0.5, sigma_t=0.1)
    ddim = pcpp.make_step_params(pcpp.PCPP_STEP_DDIM, 5.0, alphabar_t=0.5, alphabar_prev=0.6)
    assert call(ddpm, 0, None, None, None, None, None) == pcpp.PCPP_OK          # nothing to do
    assert call(ddpm, 16, FAKE, None, FAKE, None, FAKE) == pcpp.PCPP_EINVAL
    assert call(ddim, 16, FAKE, FAKE, FAKE, FAKE, FAKE) == pcpp.PCPP_EINVAL       # DDIM takes no noise
    for bad in (pcpp.make_step_params(pcpp.PCPP_STEP_DDPM, 5.0, alpha_t=0.0, alphabar_t=0.5),
                pcpp.make_step_params(pcpp.PCPP_STEP_DDPM, 5.0, alpha_t=0.9, alphabar_t=1.0),
                pcpp.make_step_params(pcpp.PCPP_STEP_DDIM, 5.0, alphabar_t=0.5, alphabar_prev=0.0),
                pcpp.make_step_params(pcpp.PCPP_STEP_DDIM, float("nan"), alphabar_t=0.5, alphabar_prev=0.6),
                pcpp.make_step_params(2, 5.0),
                pcpp.make_step_params(pcpp.PCPP_STEP_DDIM, 5.0, alphabar_t=0.5, alphabar_prev=0.6, reserved=3)):
        assert call(bad, 16, FAKE, FAKE, FAKE, None, FAKE) == pcpp.PCPP_EINVAL
    assert call(ddpm, -1, FAKE, FAKE, FAKE, None, FAKE) == pcpp.PCPP_EINVAL


def test_conv3x3_geometry_and_validation():
    from paper_2412_02962_amd import pcpp
    lib = pcpp.lib()
    ok = pcpp.make_conv_geom(256, 256, 8, 3, 320, 320, 1, pcpp.PCPP_CONV_DOWN)
    assert pcpp.pcpp_conv3x3_workspace_size(ok) >= 1 * 34 * 258 * 320 * 2
    up = pcpp.make_conv_geom(64, 64, 8, 3, 1280, 1280, 1, pcpp.PCPP_CONV_UP)
    assert pcpp.pcpp_conv3x3_workspace_size(up) >= 1 * 18 * 130 * 1280 * 2
    for bad in (pcpp.make_conv_geom(24, 20, 8, 3, 64, 64, 1, pcpp.PCPP_CONV_DOWN),   # odd band height
                pcpp.make_conv_geom(16, 21, 4, 1, 64, 64, 1, pcpp.PCPP_CONV_DOWN),   # odd width
                pcpp.make_conv_geom(16, 20, 4, 4, 64, 64, 1, 0),                       # band index
                pcpp.make_conv_geom(16, 20, 4, 1, 64, 64, 1, 3),                       # mode
                pcpp.make_conv_geom(16, 20, 4, 1, 64, 64, 1, 0, 1)):                   # reserved
        assert pcpp.pcpp_conv3x3_workspace_size(bad) == 0
    ns = pcpp.make_conv_geom(16, 20, 4, 1, 4, 64, 1, 0)
    assert lib.pcpp_conv3x3(ctypes.byref(ns), FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE, 1 << 30, None) == \
        pcpp.PCPP_ENOTSUP
    g = pcpp.make_conv_geom(16, 20, 4, 1, 64, 64, 1, pcpp.PCPP_CONV_SAME)
    call = lambda *a: lib.pcpp_conv3x3(ctypes.byref(g), *a, None)
    assert call(FAKE, FAKE, None, FAKE, None, FAKE, FAKE, 1 << 30) == pcpp.PCPP_EINVAL      # row below missing
    assert call(FAKE, FAKE + 2, FAKE, FAKE, None, FAKE, FAKE, 1 << 30) == pcpp.PCPP_EINVAL  # misaligned
    assert call(FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE, 16) == pcpp.PCPP_EWORKSPACE
    d = pcpp.make_conv_geom(16, 20, 4, 1, 64, 64, 1, pcpp.PCPP_CONV_DOWN)
    assert lib.pcpp_conv3x3(ctypes.byref(d), FAKE, FAKE, None, FAKE, None, FAKE, FAKE, 16, None) == \
        pcpp.PCPP_EWORKSPACE                                                                  # no row below needed
    # pcpp_conv3x3_export: x, row_up, row_dn, w, bias, y, first_out, last_out, workspace, bytes
    ex = lambda *a: lib.pcpp_conv3x3_export(ctypes.byref(g), *a, None)
    A = [1 << k for k in range(21, 31)]  # distinct, far apart, aligned
    assert ex(A[0], A[1], A[2], A[3], None, A[4], A[0], None, A[7], 1 << 30) == pcpp.PCPP_EINVAL  # first_out on x
    assert ex(A[0], A[1], A[2], A[3], None, A[4], None, A[4], A[7], 1 << 30) == pcpp.PCPP_EINVAL  # last_out on y
    assert ex(A[0], A[1], A[2], A[3], None, A[4], A[5], A[5], A[7], 1 << 30) == pcpp.PCPP_EINVAL  # on each other
    assert ex(A[0], A[1], A[2], A[3], None, A[4], A[5] + 8, None, A[7], 1 << 30) == pcpp.PCPP_EINVAL  # misaligned
    assert ex(A[0], A[1], A[2], A[3], None, A[4], A[5], A[6], A[7], 16) == pcpp.PCPP_EWORKSPACE  # valid exports


def test_attention_plan_splits_only_on_whole_unmasked_xcds():
    """Key pieces are merged through one XCD's L2 only when workgroup w is
    known to run on XCD w % n_xcd: compute units in whole XCDs of 32 and a
    stream that may use all of them.  Otherwise the launch runs whole blocks
    (one piece each, no merging)."""
    from paper_2412_02962_amd import pcpp
    g = pcpp.make_geom(128, 128, 8, 3, 0.25, 10)           # 2048 queries x 3072 keys, 10 heads
    bq, k, wg = pcpp.pcpp_partial_attention_plan(g, 256, 256)
    blocks = 10 * math.ceil(2048 / bq)
    assert k > 1 and wg >= blocks * k                       # split: pieces of every block
    for cus, enabled in ((256, 255), (256, 128), (256, 0), (80, 80), (250, 250), (33, 33)):
        bq2, k2, wg2 = pcpp.pcpp_partial_attention_plan(g, cus, enabled)
        assert (bq2, k2, wg2) == (bq, 1, blocks), (cus, enabled)
    _, k4, _ = pcpp.pcpp_partial_attention_plan(g, 128, 128)  # a 4-XCD partition: still whole XCDs
    assert k4 > 1
    # one key tile per block cannot be split
    small = pcpp.make_geom(16, 16, 4, 1, 0.25, 2)
    assert pcpp.pcpp_partial_attention_plan(small, 256, 256)[1] == 1
    with pytest.raises(pcpp.PcppError):
        pcpp.pcpp_partial_attention_plan(g, -1, 0)
    with pytest.raises(pcpp.PcppError):
        pcpp.pcpp_partial_attention_plan(pcpp.make_geom(128, 128, 8, 3, 0.25, 10, dtype=pcpp.PCPP_DTYPE_F32), 256, 256)


def test_noalloc_attention_validates_before_any_gpu_work():
    """The allocation-free entry point checks its arguments like
    pcpp_partial_attention, and refuses geometries whose workspace exceeds
    its fixed device array, before touching the device."""
    from paper_2412_02962_amd import pcpp
    lib = pcpp.lib()
    fake = 1 << 40  # never dereferenced: every call below fails validation first
    g = pcpp.make_geom(128, 128, 8, 3, 0.25, 10)
    args = [fake] * 8
    assert lib.pcpp_partial_attention_noalloc(ctypes.byref(g), None, *args[1:], None) == pcpp.PCPP_EINVAL
    bad = pcpp.make_geom(128, 128, 8, 3, 1.5, 10)
    assert lib.pcpp_partial_attention_noalloc(ctypes.byref(bad), *args, None) == pcpp.PCPP_EINVAL
    d32 = pcpp.make_geom(128, 128, 8, 3, 0.25, 10, head_dim=32)
    assert lib.pcpp_partial_attention_noalloc(ctypes.byref(d32), *args, None) == pcpp.PCPP_ENOTSUP
    # 3840 px level 1, 2 bands: a workspace far above the fixed array
    big = pcpp.make_geom(240, 240, 2, 0, 0.3, 10)
    assert pcpp.pcpp_partial_attention_workspace_size(big) > pcpp.PCPP_NOALLOC_SCRATCH_BYTES
    assert lib.pcpp_partial_attention_noalloc(ctypes.byref(big), *args, None) == pcpp.PCPP_EWORKSPACE
    # the bench workload fits
    assert pcpp.pcpp_partial_attention_workspace_size(g) <= pcpp.PCPP_NOALLOC_SCRATCH_BYTES
