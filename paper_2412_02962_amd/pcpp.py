"""ctypes binding of libpcpp.so: the C ABI declared in include/pcpp.h, with
the same function names.  Argument marshalling only (device pointers from
torch tensors, the current HIP stream); every step of the computation runs
in the library's HIP kernels.  There is no fallback: if the shared library is
missing or does not load, importing this module raises."""

from __future__ import annotations

import ctypes
import os
from typing import Optional

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpcpp.so")

PCPP_OK = 0
PCPP_EINVAL = -1
PCPP_ENOTSUP = -2
PCPP_EWORKSPACE = -3
PCPP_EHIP = -4

PCPP_DTYPE_F32 = 0
PCPP_DTYPE_BF16 = 1


class PcppError(RuntimeError):
    def __init__(self, fn, status):
        self.status = status
        super().__init__(f"{fn} failed with status {status}: {pcpp_strerror(status)}")


class pcpp_geom_t(ctypes.Structure):
    _fields_ = [
        ("H", ctypes.c_int32), ("W", ctypes.c_int32),
        ("n_patches", ctypes.c_int32), ("patch_idx", ctypes.c_int32),
        ("partial", ctypes.c_double),
        ("heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
        ("batch", ctypes.c_int32), ("step", ctypes.c_int32),
        ("dtype", ctypes.c_int32), ("reserved", ctypes.c_int32),
    ]


_BLOCK_PTR_FIELDS = (
    "gn_gamma", "gn_beta", "proj_in_w", "proj_in_b", "ln1_gamma", "ln1_beta",
    "attn1_qkv_w", "attn1_out_w", "attn1_out_b", "ln2_gamma", "ln2_beta",
    "attn2_q_w", "attn2_kv_w", "attn2_out_w", "attn2_out_b", "ln3_gamma",
    "ln3_beta", "ff1_w", "ff1_b", "ff2_w", "ff2_b", "proj_out_w", "proj_out_b",
)


class pcpp_block_weights_t(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in _BLOCK_PTR_FIELDS] + [
        ("ff_inner", ctypes.c_int32), ("gn_groups", ctypes.c_int32)]


BASIC_BLOCK_PTR_FIELDS = (
    "ln1_gamma", "ln1_beta", "attn1_qkv_w", "attn1_out_w", "attn1_out_b", "ln2_gamma", "ln2_beta",
    "attn2_q_w", "attn2_kv_w", "attn2_out_w", "attn2_out_b", "ln3_gamma", "ln3_beta",
    "ff1_w", "ff1_b", "ff2_w", "ff2_b",
)


class pcpp_basic_block_weights_t(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in BASIC_BLOCK_PTR_FIELDS]


class pcpp_module_weights_t(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("gn_gamma", "gn_beta", "proj_in_w", "proj_in_b", "proj_out_w",
                                               "proj_out_b")] + [
        ("blocks", ctypes.POINTER(pcpp_basic_block_weights_t)), ("depth", ctypes.c_int32),
        ("ff_inner", ctypes.c_int32), ("gn_groups", ctypes.c_int32)]


class pcpp_resnet_geom_t(ctypes.Structure):
    _fields_ = [
        ("H", ctypes.c_int32), ("W", ctypes.c_int32),
        ("n_patches", ctypes.c_int32), ("patch_idx", ctypes.c_int32),
        ("c_in", ctypes.c_int32), ("c_out", ctypes.c_int32),
        ("temb_dim", ctypes.c_int32), ("groups", ctypes.c_int32),
        ("batch", ctypes.c_int32), ("eps", ctypes.c_float), ("reserved", ctypes.c_int32),
    ]


RESNET_PTR_FIELDS = (
    "gn1_gamma", "gn1_beta", "conv1_w", "conv1_b", "temb_w", "temb_b",
    "gn2_gamma", "gn2_beta", "conv2_w", "conv2_b", "skip_w", "skip_b",
)


class pcpp_resnet_weights_t(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in RESNET_PTR_FIELDS]


PCPP_CONV_SAME = 0
PCPP_CONV_DOWN = 1
PCPP_CONV_UP = 2


class pcpp_conv_geom_t(ctypes.Structure):
    _fields_ = [
        ("H", ctypes.c_int32), ("W", ctypes.c_int32),
        ("n_patches", ctypes.c_int32), ("patch_idx", ctypes.c_int32),
        ("c_in", ctypes.c_int32), ("c_out", ctypes.c_int32),
        ("batch", ctypes.c_int32), ("mode", ctypes.c_int32), ("reserved", ctypes.c_int32),
    ]


PCPP_STEP_DDPM = 0
PCPP_STEP_DDIM = 1


class pcpp_step_params_t(ctypes.Structure):
    _fields_ = [
        ("guidance", ctypes.c_float), ("alpha_t", ctypes.c_float), ("alphabar_t", ctypes.c_float),
        ("sigma_t", ctypes.c_float), ("alphabar_prev", ctypes.c_float),
        ("mode", ctypes.c_int32), ("reserved", ctypes.c_int32),
    ]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built: run __graft_entry__.build() "
                          "(or python paper_2412_02962_amd/build.py); there is no fallback path")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    gp = ctypes.POINTER(pcpp_geom_t)
    wp = ctypes.POINTER(pcpp_block_weights_t)
    i32p = ctypes.POINTER(ctypes.c_int32)
    sig = {
        "pcpp_version": (ctypes.c_int, []),
        "pcpp_strerror": (ctypes.c_char_p, [ctypes.c_int]),
        "pcpp_context_rows": (ctypes.c_int, [gp, i32p, i32p, i32p, i32p]),
        "pcpp_gather_context": (ctypes.c_int, [gp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]),
        "pcpp_partial_attention_workspace_size": (sz, [gp]),
        "pcpp_partial_attention_plan": (ctypes.c_int, [gp, i32, i32, vp, i32p, i32p, i32p]),
        "pcpp_partial_attention_noalloc": (ctypes.c_int, [gp, vp, vp, vp, vp, vp, vp, vp, vp, vp]),
        "pcpp_partial_attention": (ctypes.c_int, [gp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
        "pcpp_transformer_block_workspace_size": (sz, [gp, wp, i32, i32]),
        "pcpp_transformer_block": (ctypes.c_int, [gp, wp, vp, vp, i32, i32, vp, vp, vp, vp, vp, vp, vp,
                                                  vp, sz, vp]),
        "pcpp_transformer_block_sync_gn": (ctypes.c_int, [gp, wp, vp, vp, i32, i32, vp, vp, vp, vp, vp, vp,
                                                          vp, vp, vp, vp, sz, vp]),
        "pcpp_partial_attention_multihop_workspace_size": (sz, [gp]),
        "pcpp_partial_attention_multihop": (ctypes.c_int, [gp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
        "pcpp_boundary_bytes": (sz, [gp]),
        "pcpp_pack_boundary": (ctypes.c_int, [gp, vp, vp, vp, vp, vp]),
        "pcpp_unpack_boundary": (ctypes.c_int, [gp, vp, vp, vp, vp, vp, vp, vp]),
        "pcpp_multihop_message_bytes": (sz, [gp, i32]),
        "pcpp_pack_multihop": (ctypes.c_int, [gp, i32, vp, vp, vp, vp]),
        "pcpp_unpack_multihop": (ctypes.c_int, [gp, i32, vp, vp, vp, vp, vp, vp]),
        "pcpp_resnet_block_workspace_size": (sz, [ctypes.POINTER(pcpp_resnet_geom_t)]),
        "pcpp_resnet_block": (ctypes.c_int, [ctypes.POINTER(pcpp_resnet_geom_t),
                                             ctypes.POINTER(pcpp_resnet_weights_t)] + [vp] * 14 + [sz, vp]),
        "pcpp_guided_step": (ctypes.c_int, [ctypes.POINTER(pcpp_step_params_t), ctypes.c_int64,
                                            vp, vp, vp, vp, vp, vp]),
        "pcpp_transformer_module_workspace_size": (sz, [gp, ctypes.POINTER(pcpp_module_weights_t), i32, i32]),
        "pcpp_transformer_module": (ctypes.c_int, [gp, ctypes.POINTER(pcpp_module_weights_t), vp, vp, i32, i32,
                                                   vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
        "pcpp_concat_channels": (ctypes.c_int, [ctypes.c_int64, vp, i32, vp, i32, vp, vp]),
        "pcpp_layer_norm": (ctypes.c_int, [ctypes.c_int64, i32, ctypes.c_float, vp, vp, vp, vp, vp]),
        "pcpp_group_norm_workspace_size": (sz, [i32, i32, i32, i32]),
        "pcpp_group_norm": (ctypes.c_int, [i32, i32, i32, i32, ctypes.c_float, i32, vp, vp, vp, vp, i32, i32, vp, vp,
                                           vp, sz, vp]),
        "pcpp_conv3x3_workspace_size": (sz, [ctypes.POINTER(pcpp_conv_geom_t)]),
        "pcpp_conv3x3": (ctypes.c_int, [ctypes.POINTER(pcpp_conv_geom_t)] + [vp] * 7 + [sz, vp]),
        "pcpp_conv3x3_export": (ctypes.c_int, [ctypes.POINTER(pcpp_conv_geom_t)] + [vp] * 9 + [sz, vp]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    return lib


_lib = _load()
EXPORTED = (
    "pcpp_version", "pcpp_strerror", "pcpp_context_rows", "pcpp_gather_context",
    "pcpp_partial_attention_workspace_size", "pcpp_partial_attention", "pcpp_partial_attention_plan",
    "pcpp_partial_attention_noalloc",
    "pcpp_transformer_block_workspace_size", "pcpp_transformer_block",
    "pcpp_boundary_bytes", "pcpp_pack_boundary", "pcpp_unpack_boundary", "pcpp_transformer_block_sync_gn",
    "pcpp_partial_attention_multihop_workspace_size", "pcpp_partial_attention_multihop",
    "pcpp_multihop_message_bytes", "pcpp_pack_multihop", "pcpp_unpack_multihop",
    "pcpp_resnet_block_workspace_size", "pcpp_resnet_block", "pcpp_guided_step",
    "pcpp_conv3x3_workspace_size", "pcpp_conv3x3", "pcpp_conv3x3_export",
    "pcpp_transformer_module_workspace_size", "pcpp_transformer_module",
    "pcpp_concat_channels", "pcpp_layer_norm", "pcpp_group_norm_workspace_size", "pcpp_group_norm",
)


def lib():
    return _lib


def make_geom(H, W, n_patches, patch_idx, partial, heads, head_dim=64, batch=1, step=0,
              dtype=PCPP_DTYPE_BF16, reserved=0) -> pcpp_geom_t:
    return pcpp_geom_t(H, W, n_patches, patch_idx, float(partial), heads, head_dim, batch, step,
                       dtype, reserved)


def _ptr(t) -> Optional[int]:
    """Device address of a tensor (or a raw int address); None -> NULL."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is not None:
        return stream if isinstance(stream, int) else stream.cuda_stream
    import torch  # device memory and streams only
    return torch.cuda.current_stream().cuda_stream


def _check(fn, st):
    if st != PCPP_OK:
        raise PcppError(fn, st)


def pcpp_version() -> int:
    return _lib.pcpp_version()


def pcpp_strerror(status: int) -> str:
    return _lib.pcpp_strerror(status).decode()


def pcpp_context_rows(g: pcpp_geom_t):
    """(h, up, dn, n_kv) of Eq. 1; raises PcppError on invalid geometry."""
    h, up, dn, nkv = (ctypes.c_int32() for _ in range(4))
    _check("pcpp_context_rows", _lib.pcpp_context_rows(ctypes.byref(g), ctypes.byref(h), ctypes.byref(up),
                                                       ctypes.byref(dn), ctypes.byref(nkv)))
    return h.value, up.value, dn.value, nkv.value


def pcpp_gather_context(g, k_fresh, v_fresh, k_up, v_up, k_dn, v_dn, idx_out, k_ctx, v_ctx, stream=None):
    _check("pcpp_gather_context", _lib.pcpp_gather_context(
        ctypes.byref(g), _ptr(k_fresh), _ptr(v_fresh), _ptr(k_up), _ptr(v_up), _ptr(k_dn), _ptr(v_dn),
        _ptr(idx_out), _ptr(k_ctx), _ptr(v_ctx), _stream(stream)))


def pcpp_partial_attention_workspace_size(g) -> int:
    return _lib.pcpp_partial_attention_workspace_size(ctypes.byref(g))


def pcpp_partial_attention_plan(g, cus=0, cus_enabled=0, stream=None):
    """(queries per block, pieces per block, workgroups) of the bf16 attention's
    launch: on a device of `cus` compute units with `cus_enabled` usable, or
    (cus = 0) on the current device with the CU mask of `stream`."""
    bq, k, wg = (ctypes.c_int32() for _ in range(3))
    st = _stream(stream) if cus == 0 else None
    _check("pcpp_partial_attention_plan", _lib.pcpp_partial_attention_plan(
        ctypes.byref(g), cus, cus_enabled, st, ctypes.byref(bq), ctypes.byref(k), ctypes.byref(wg)))
    return bq.value, k.value, wg.value


def pcpp_partial_attention(g, q, k_fresh, v_fresh, k_up, v_up, k_dn, v_dn, out, workspace=None,
                           ws_bytes=0, stream=None):
    _check("pcpp_partial_attention", _lib.pcpp_partial_attention(
        ctypes.byref(g), _ptr(q), _ptr(k_fresh), _ptr(v_fresh), _ptr(k_up), _ptr(v_up), _ptr(k_dn),
        _ptr(v_dn), _ptr(out), _ptr(workspace), ws_bytes, _stream(stream)))


PCPP_NOALLOC_SCRATCH_BYTES = 32 * 1024 * 1024


def pcpp_partial_attention_noalloc(g, q, k_fresh, v_fresh, k_up, v_up, k_dn, v_dn, out, stream=None):
    _check("pcpp_partial_attention_noalloc", _lib.pcpp_partial_attention_noalloc(
        ctypes.byref(g), _ptr(q), _ptr(k_fresh), _ptr(v_fresh), _ptr(k_up), _ptr(v_up), _ptr(k_dn),
        _ptr(v_dn), _ptr(out), _stream(stream)))


def make_block_weights(tensors: dict, ff_inner: int, gn_groups: int) -> pcpp_block_weights_t:
    w = pcpp_block_weights_t()
    for name in _BLOCK_PTR_FIELDS:
        setattr(w, name, _ptr(tensors.get(name)))
    w.ff_inner = ff_inner
    w.gn_groups = gn_groups
    return w


def pcpp_transformer_block_workspace_size(g, w, n_text, text_dim) -> int:
    return _lib.pcpp_transformer_block_workspace_size(ctypes.byref(g), ctypes.byref(w), n_text, text_dim)


def pcpp_transformer_block(g, w, x, text, n_text, text_dim, k_up, v_up, k_dn, v_dn, y, k_fresh_out,
                           v_fresh_out, workspace, ws_bytes, stream=None):
    _check("pcpp_transformer_block", _lib.pcpp_transformer_block(
        ctypes.byref(g), ctypes.byref(w), _ptr(x), _ptr(text), n_text, text_dim, _ptr(k_up), _ptr(v_up),
        _ptr(k_dn), _ptr(v_dn), _ptr(y), _ptr(k_fresh_out), _ptr(v_fresh_out), _ptr(workspace), ws_bytes,
        _stream(stream)))


def pcpp_boundary_bytes(g) -> int:
    return _lib.pcpp_boundary_bytes(ctypes.byref(g))


def pcpp_pack_boundary(g, k_fresh, v_fresh, send_up, send_dn, stream=None):
    _check("pcpp_pack_boundary", _lib.pcpp_pack_boundary(
        ctypes.byref(g), _ptr(k_fresh), _ptr(v_fresh), _ptr(send_up), _ptr(send_dn), _stream(stream)))


def pcpp_unpack_boundary(g, recv_up, recv_dn, k_up, v_up, k_dn, v_dn, stream=None):
    _check("pcpp_unpack_boundary", _lib.pcpp_unpack_boundary(
        ctypes.byref(g), _ptr(recv_up), _ptr(recv_dn), _ptr(k_up), _ptr(v_up), _ptr(k_dn), _ptr(v_dn),
        _stream(stream)))


def pcpp_transformer_block_sync_gn(g, w, x, text, n_text, text_dim, k_up, v_up, k_dn, v_dn, gn_bands, gn_own, y,
                                   k_fresh_out, v_fresh_out, workspace, ws_bytes, stream=None):
    _check("pcpp_transformer_block_sync_gn", _lib.pcpp_transformer_block_sync_gn(
        ctypes.byref(g), ctypes.byref(w), _ptr(x), _ptr(text), n_text, text_dim, _ptr(k_up), _ptr(v_up),
        _ptr(k_dn), _ptr(v_dn), _ptr(gn_bands), _ptr(gn_own), _ptr(y), _ptr(k_fresh_out), _ptr(v_fresh_out),
        _ptr(workspace), ws_bytes, _stream(stream)))


def pcpp_partial_attention_multihop_workspace_size(g) -> int:
    return _lib.pcpp_partial_attention_multihop_workspace_size(ctypes.byref(g))


def pcpp_partial_attention_multihop(g, q, k_fresh, v_fresh, k_above, v_above, k_below, v_below, out,
                                    workspace=None, ws_bytes=0, stream=None):
    _check("pcpp_partial_attention_multihop", _lib.pcpp_partial_attention_multihop(
        ctypes.byref(g), _ptr(q), _ptr(k_fresh), _ptr(v_fresh), _ptr(k_above), _ptr(v_above), _ptr(k_below),
        _ptr(v_below), _ptr(out), _ptr(workspace), ws_bytes, _stream(stream)))


def pcpp_multihop_message_bytes(g, peer) -> int:
    return _lib.pcpp_multihop_message_bytes(ctypes.byref(g), peer)


def pcpp_pack_multihop(g, peer, k_fresh, v_fresh, send, stream=None):
    _check("pcpp_pack_multihop", _lib.pcpp_pack_multihop(
        ctypes.byref(g), peer, _ptr(k_fresh), _ptr(v_fresh), _ptr(send), _stream(stream)))


def pcpp_unpack_multihop(g, peer, recv, k_above, v_above, k_below, v_below, stream=None):
    _check("pcpp_unpack_multihop", _lib.pcpp_unpack_multihop(
        ctypes.byref(g), peer, _ptr(recv), _ptr(k_above), _ptr(v_above), _ptr(k_below), _ptr(v_below),
        _stream(stream)))


def make_resnet_geom(H, W, n_patches, patch_idx, c_in, c_out, temb_dim=1280, groups=32, batch=1, eps=1e-5,
                     reserved=0) -> pcpp_resnet_geom_t:
    return pcpp_resnet_geom_t(H, W, n_patches, patch_idx, c_in, c_out, temb_dim, groups, batch, float(eps),
                              reserved)


def make_resnet_weights(tensors: dict) -> pcpp_resnet_weights_t:
    w = pcpp_resnet_weights_t()
    for name in RESNET_PTR_FIELDS:
        setattr(w, name, _ptr(tensors.get(name)))
    return w


def pcpp_resnet_block_workspace_size(g) -> int:
    return _lib.pcpp_resnet_block_workspace_size(ctypes.byref(g))


def pcpp_resnet_block(g, w, x, temb, edges1_up, edges1_dn, edges2_up, edges2_dn, gn1_bands, gn1_own, gn2_bands,
                      gn2_own, y, edges1_out, edges2_out, workspace, ws_bytes, stream=None):
    _check("pcpp_resnet_block", _lib.pcpp_resnet_block(
        ctypes.byref(g), ctypes.byref(w), _ptr(x), _ptr(temb), _ptr(edges1_up), _ptr(edges1_dn), _ptr(edges2_up),
        _ptr(edges2_dn), _ptr(gn1_bands), _ptr(gn1_own), _ptr(gn2_bands), _ptr(gn2_own), _ptr(y), _ptr(edges1_out),
        _ptr(edges2_out), _ptr(workspace), ws_bytes, _stream(stream)))


def make_step_params(mode, guidance, alpha_t=1.0, alphabar_t=0.5, sigma_t=0.0, alphabar_prev=1.0,
                     reserved=0) -> pcpp_step_params_t:
    return pcpp_step_params_t(float(guidance), float(alpha_t), float(alphabar_t), float(sigma_t),
                              float(alphabar_prev), mode, reserved)


def pcpp_guided_step(sp, n, x_t, eps_uncond, eps_cond, z, x_prev, stream=None):
    _check("pcpp_guided_step", _lib.pcpp_guided_step(
        ctypes.byref(sp), n, _ptr(x_t), _ptr(eps_uncond), _ptr(eps_cond), _ptr(z), _ptr(x_prev), _stream(stream)))


def make_conv_geom(H, W, n_patches, patch_idx, c_in, c_out, batch=1, mode=PCPP_CONV_SAME,
                   reserved=0) -> pcpp_conv_geom_t:
    return pcpp_conv_geom_t(H, W, n_patches, patch_idx, c_in, c_out, batch, mode, reserved)


def pcpp_conv3x3_workspace_size(g) -> int:
    return _lib.pcpp_conv3x3_workspace_size(ctypes.byref(g))


def pcpp_conv3x3(g, x, row_up, row_dn, w, bias, y, workspace, ws_bytes, stream=None):
    _check("pcpp_conv3x3", _lib.pcpp_conv3x3(
        ctypes.byref(g), _ptr(x), _ptr(row_up), _ptr(row_dn), _ptr(w), _ptr(bias), _ptr(y), _ptr(workspace),
        ws_bytes, _stream(stream)))


def pcpp_conv3x3_export(g, x, row_up, row_dn, w, bias, y, first_out, last_out, workspace, ws_bytes,
                        stream=None):
    _check("pcpp_conv3x3_export", _lib.pcpp_conv3x3_export(
        ctypes.byref(g), _ptr(x), _ptr(row_up), _ptr(row_dn), _ptr(w), _ptr(bias), _ptr(y), _ptr(first_out),
        _ptr(last_out), _ptr(workspace), ws_bytes, _stream(stream)))


def make_module_weights(module: dict, blocks: list, ff_inner: int, gn_groups: int):
    """(pcpp_module_weights_t, keep-alive array) from device tensors: module
    holds gn_gamma .. proj_out_b, blocks[j] basic block j's tensors."""
    arr = (pcpp_basic_block_weights_t * len(blocks))()
    for j, bt in enumerate(blocks):
        for name in BASIC_BLOCK_PTR_FIELDS:
            setattr(arr[j], name, _ptr(bt.get(name)))
    w = pcpp_module_weights_t()
    for name in ("gn_gamma", "gn_beta", "proj_in_w", "proj_in_b", "proj_out_w", "proj_out_b"):
        setattr(w, name, _ptr(module.get(name)))
    w.blocks = ctypes.cast(arr, ctypes.POINTER(pcpp_basic_block_weights_t))
    w.depth = len(blocks)
    w.ff_inner = ff_inner
    w.gn_groups = gn_groups
    return w, arr


def _ptr_array(ts):
    if ts is None:
        return None
    return (ctypes.c_void_p * len(ts))(*[_ptr(t) for t in ts])


def pcpp_transformer_module_workspace_size(g, w, n_text, text_dim) -> int:
    return _lib.pcpp_transformer_module_workspace_size(ctypes.byref(g), ctypes.byref(w), n_text, text_dim)


def pcpp_transformer_module(g, w, x, text, n_text, text_dim, k_up, v_up, k_dn, v_dn, gn_bands, gn_own, y,
                            k_fresh_out, v_fresh_out, workspace, ws_bytes, stream=None):
    """k_up .. v_fresh_out: lists of per-basic-block tensors (or None)."""
    arrs = [_ptr_array(a) for a in (k_up, v_up, k_dn, v_dn, k_fresh_out, v_fresh_out)]
    _check("pcpp_transformer_module", _lib.pcpp_transformer_module(
        ctypes.byref(g), ctypes.byref(w), _ptr(x), _ptr(text), n_text, text_dim,
        *[None if a is None else ctypes.cast(a, ctypes.c_void_p) for a in arrs[:4]],
        _ptr(gn_bands), _ptr(gn_own), _ptr(y),
        *[None if a is None else ctypes.cast(a, ctypes.c_void_p) for a in arrs[4:]],
        _ptr(workspace), ws_bytes, _stream(stream)))


def pcpp_concat_channels(rows, a, ca, b, cb, out, stream=None):
    _check("pcpp_concat_channels", _lib.pcpp_concat_channels(rows, _ptr(a), ca, _ptr(b), cb, _ptr(out),
                                                              _stream(stream)))


def pcpp_layer_norm(rows, channels, eps, x, gamma, beta, y, stream=None):
    _check("pcpp_layer_norm", _lib.pcpp_layer_norm(rows, channels, eps, _ptr(x), _ptr(gamma), _ptr(beta), _ptr(y),
                                                    _stream(stream)))


def pcpp_group_norm_workspace_size(batch, tokens, channels, groups) -> int:
    return _lib.pcpp_group_norm_workspace_size(batch, tokens, channels, groups)


def pcpp_group_norm(batch, tokens, channels, groups, eps, silu, x, gamma, beta, y, workspace, ws_bytes, stream=None,
                    bands=None, n_bands=1, band=0, own_out=None):
    _check("pcpp_group_norm", _lib.pcpp_group_norm(batch, tokens, channels, groups, eps, silu, _ptr(x), _ptr(gamma),
                                                    _ptr(beta), _ptr(bands), n_bands, band, _ptr(own_out), _ptr(y),
                                                    _ptr(workspace), ws_bytes, _stream(stream)))
