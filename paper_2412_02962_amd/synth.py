"""Seeded synthetic inputs for the PCPP hot path.

This module only draws numbers and lays them out; it holds none of the
method's arithmetic (no context selection, no attention, no normalisation).
Both the GPU path's tests and the CPU oracle consume what it returns, so it
imports nothing else from this package and nothing from the oracle.

Workload shapes follow the SDXL U-Net's self-attention layers: an image of
R x R pixels has an R/8 latent, whose first transformer level runs on an
(R/16) x (R/16) token grid with 640 channels (10 heads of 64) and whose
second level runs on (R/32) x (R/32) tokens with 1280 channels (20 heads).
The patch split follows Sec. 3.1: n row bands of height h = H/n, full width.

Every tensor is drawn on the full token grid, patch by patch, from its own
counter-keyed stream (seed, patch, tensor kind), so patch j's arrays are the
same whichever patch is the local one.  Fresh activations are N(0, 1); the
stale copy a neighbour holds from the previous step is fresh + sigma * N(0, 1)
with sigma = 0.05 (the small step-to-step change the method relies on,
abstract and Sec. 2.2).
"""

from __future__ import annotations

import dataclasses
import os
from typing import Dict, Optional

import numpy as np

BASE_SEED = 2412029620

DTYPE_F32 = "f32"
DTYPE_BF16 = "bf16"


@dataclasses.dataclass(frozen=True)
class AttnConfig:
    """Geometry of one partially conditioned self-attention call."""

    name: str
    H: int            # token-grid height of this layer
    W: int            # token-grid width
    n: int            # number of row patches
    i: int            # 0-based local patch index (row band i, top band is 0)
    p: float          # partial value: fraction of a neighbour's height used
    heads: int
    d: int            # head dim
    dtype: str
    seed_id: int
    batch: int = 1
    step: int = 0

    @property
    def C(self) -> int:
        return self.heads * self.d

    @property
    def h(self) -> int:
        return self.H // self.n

    @property
    def n_q(self) -> int:
        return self.h * self.W


@dataclasses.dataclass(frozen=True)
class BlockConfig:
    """One SDXL-shaped transformer block (GroupNorm, proj_in, self-attn,
    cross-attn, GEGLU feed-forward, proj_out) around a partial self-attn."""

    name: str
    attn: AttnConfig
    n_text: int = 77
    text_dim: int = 2048
    ff_inner: int = 2560
    gn_groups: int = 32
    seed_id: int = 5


def _cfg(name, H, W, n, i, p, heads, d, dtype, seed_id):
    return AttnConfig(name=name, H=H, W=W, n=n, i=i, p=p, heads=heads, d=d,
                      dtype=dtype, seed_id=seed_id)


# The five workloads: a tiny fp32 case, and SDXL level-1 / level-2 shapes at
# 1024 px and 2048 px.  The 2048 px level-1 case is run at p = 0.25 and 0.5.
ATTN_CONFIGS: Dict[str, AttnConfig] = {
    c.name: c
    for c in [
        _cfg("tiny_f32", 16, 16, 4, 1, 0.25, 2, 64, DTYPE_F32, 1),
        _cfg("sdxl1024_l1", 64, 64, 4, 1, 0.25, 10, 64, DTYPE_BF16, 2),
        _cfg("sdxl2048_l1_p25", 128, 128, 8, 3, 0.25, 10, 64, DTYPE_BF16, 3),
        _cfg("sdxl2048_l1_p50", 128, 128, 8, 3, 0.5, 10, 64, DTYPE_BF16, 3),
        _cfg("sdxl2048_l2_edge", 64, 64, 8, 0, 0.25, 20, 64, DTYPE_BF16, 4),
    ]
}

# The paper's own band splits (Sec. 5.1: two devices at p = 0.3, four at
# p = 0.8) on SDXL's two self-attention grids (level 1: R/16 square, 640
# channels; level 2: R/32 square, 1280 channels) at 1024, 2048 and 3840 px.
# Two bands: band 0 (each band is an edge band); four bands: interior band 1.
PAPER_GEOMETRIES: Dict[str, AttnConfig] = {}
for _res in (1024, 2048, 3840):
    for _lvl, _div, _heads in ((1, 16, 10), (2, 32, 20)):
        for _n, _p, _i in ((2, 0.3, 0), (4, 0.8, 1)):
            _name = f"paper_{_res}_l{_lvl}_n{_n}_p{_p}"
            PAPER_GEOMETRIES[_name] = _cfg(_name, _res // _div, _res // _div, _n, _i, _p, _heads, 64, DTYPE_BF16,
                                           60 + _res // 1024 * 4 + _lvl * 2 + _n // 2)

BLOCK_CONFIG = BlockConfig(
    name="sdxl2048_block",
    attn=_cfg("sdxl2048_block_attn", 128, 128, 8, 3, 0.25, 10, 64, DTYPE_BF16, 5),
)

# The same block at the second transformer level (64 x 64 tokens of 1280
# channels, 20 heads, feed-forward 4 x 1280), interior band 3 of 8.
BLOCK_CONFIG_L2 = BlockConfig(
    name="sdxl2048_l2_block",
    attn=_cfg("sdxl2048_l2_block_attn", 64, 64, 8, 3, 0.25, 20, 64, DTYPE_BF16, 6),
    ff_inner=5120,
    seed_id=6,
)

# Input variants.
#   "unit"      : Q, K, V ~ N(0,1); the kernel's 1/sqrt(d) makes logits unit-std
#   "prescaled" : Q, K, V ~ N(0,1)/sqrt(d) as well (near-uniform softmax)
#   "sharp"     : Q ~ 4 N(0,1) (logits four times wider)
#   "stale_eq_fresh": no step-to-step drift (stale copies equal fresh ones)
VARIANTS = ("unit", "prescaled", "sharp", "stale_eq_fresh")

_KIND = {"q": 1, "k": 2, "v": 3, "k_drift": 4, "v_drift": 5, "q_drift": 6}


def _stream(seed: int, *key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, *key])))


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round to bfloat16 (round to nearest even via float32) and return the
    16-bit patterns as uint16.  NaN inputs are not expected here."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    u = f.view(np.uint32)
    # finite values stay below 2^32 after adding the rounding bias
    u = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return u.astype(np.uint16)


def store(x: np.ndarray, dtype: str) -> np.ndarray:
    """Cast a float64 draw to its stored form: float32, or bf16 bit patterns."""
    if dtype == DTYPE_F32:
        return np.ascontiguousarray(x, dtype=np.float32)
    if dtype == DTYPE_BF16:
        return bf16_bits(x)
    raise ValueError(dtype)


def patch_tensor(cfg: AttnConfig, patch: int, kind: str, stale: bool,
                 variant: str = "unit", seed: Optional[int] = None) -> np.ndarray:
    """float64 [batch, h*W, C] draw of tensor `kind` ('q', 'k' or 'v') for row
    band `patch`, fresh (this step) or stale (the previous step's copy)."""
    if variant not in VARIANTS:
        raise ValueError(variant)
    s = BASE_SEED + cfg.seed_id if seed is None else seed
    shape = (cfg.batch, cfg.h * cfg.W, cfg.C)
    x = _stream(s, patch, _KIND[kind]).standard_normal(shape)
    if stale and variant != "stale_eq_fresh":
        x = x + 0.05 * _stream(s, patch, _KIND[kind + "_drift"]).standard_normal(shape)
    if variant == "prescaled":
        x = x / np.sqrt(cfg.d)
    elif variant == "sharp" and kind == "q":
        x = 4.0 * x
    return x


def attention_inputs(cfg: AttnConfig, variant: str = "unit",
                     seed: Optional[int] = None) -> Dict[str, Optional[np.ndarray]]:
    """Stored-dtype inputs of one partial-attention call on patch cfg.i.

    Returns q, k_fresh, v_fresh: the local patch's fresh tensors
    [batch, h*W, C]; k_up, v_up: the whole stale patch above (or None for the
    top patch); k_dn, v_dn: the whole stale patch below (or None for the
    bottom patch).  Which rows of the neighbours are read is the method's
    business, not the generator's.
    """
    i = cfg.i
    out: Dict[str, Optional[np.ndarray]] = {}
    out["q"] = store(patch_tensor(cfg, i, "q", False, variant, seed), cfg.dtype)
    out["k_fresh"] = store(patch_tensor(cfg, i, "k", False, variant, seed), cfg.dtype)
    out["v_fresh"] = store(patch_tensor(cfg, i, "v", False, variant, seed), cfg.dtype)
    for tag, j in (("up", i - 1), ("dn", i + 1)):
        if 0 <= j < cfg.n:
            out["k_" + tag] = store(patch_tensor(cfg, j, "k", True, variant, seed), cfg.dtype)
            out["v_" + tag] = store(patch_tensor(cfg, j, "v", True, variant, seed), cfg.dtype)
        else:
            out["k_" + tag] = None
            out["v_" + tag] = None
    return out


# --------------------------------------------------------------------------
# Transformer-block inputs (random-init weights of the SDXL block shapes).
# --------------------------------------------------------------------------

BLOCK_WEIGHT_NAMES = (
    "gn_gamma", "gn_beta",
    "proj_in_w", "proj_in_b",
    "ln1_gamma", "ln1_beta",
    "attn1_qkv_w",
    "attn1_out_w", "attn1_out_b",
    "ln2_gamma", "ln2_beta",
    "attn2_q_w", "attn2_kv_w",
    "attn2_out_w", "attn2_out_b",
    "ln3_gamma", "ln3_beta",
    "ff1_w", "ff1_b",
    "ff2_w", "ff2_b",
    "proj_out_w", "proj_out_b",
)


def block_weight_shapes(bc: BlockConfig) -> Dict[str, tuple]:
    C = bc.attn.C
    F = bc.ff_inner
    T = bc.text_dim
    return {
        "gn_gamma": (C,), "gn_beta": (C,),
        "proj_in_w": (C, C), "proj_in_b": (C,),
        "ln1_gamma": (C,), "ln1_beta": (C,),
        # rows [0,C) = W_q, [C,2C) = W_k, [2C,3C) = W_v   (nn.Linear layout: [out, in])
        "attn1_qkv_w": (3 * C, C),
        "attn1_out_w": (C, C), "attn1_out_b": (C,),
        "ln2_gamma": (C,), "ln2_beta": (C,),
        "attn2_q_w": (C, C),
        # rows [0,C) = W_k, [C,2C) = W_v over the text features
        "attn2_kv_w": (2 * C, T),
        "attn2_out_w": (C, C), "attn2_out_b": (C,),
        "ln3_gamma": (C,), "ln3_beta": (C,),
        # rows [0,F) = value half, [F,2F) = gate half of GEGLU
        "ff1_w": (2 * F, C), "ff1_b": (2 * F,),
        "ff2_w": (C, F), "ff2_b": (C,),
        "proj_out_w": (C, C), "proj_out_b": (C,),
    }


def block_inputs(bc: BlockConfig = BLOCK_CONFIG, seed: Optional[int] = None,
                 batch: int = 1) -> Dict[str, Optional[np.ndarray]]:
    """bf16 inputs of one transformer-block call on patch bc.attn.i.

    x [batch, h*W, C] ~ N(0,1); text [batch, n_text, text_dim] ~ N(0,1);
    linear weights ~ N(0, 1/fan_in); biases ~ 0.02 N(0,1); norm scales
    ~ 1 + 0.1 N(0,1), shifts ~ 0.1 N(0,1); the neighbours' stale K and V
    (whole patches above / below, [batch, h*W, C]) ~ N(0,1), the scale of the
    block's own K/V projections of a layer-normed input.
    """
    cfg = bc.attn
    s = BASE_SEED + bc.seed_id if seed is None else seed
    C = cfg.C
    nq = cfg.h * cfg.W
    out: Dict[str, Optional[np.ndarray]] = {}
    out["x"] = bf16_bits(_stream(s, 100).standard_normal((batch, nq, C)))
    out["text"] = bf16_bits(_stream(s, 101).standard_normal((batch, bc.n_text, bc.text_dim)))
    for idx, (name, shape) in enumerate(block_weight_shapes(bc).items()):
        g = _stream(s, 200 + idx)
        if name.endswith("_w"):
            w = g.standard_normal(shape) / np.sqrt(shape[1])
        elif name.endswith("_b") or name.endswith("_beta"):
            w = (0.02 if name.endswith("_b") else 0.1) * g.standard_normal(shape)
        else:  # *_gamma
            w = 1.0 + 0.1 * g.standard_normal(shape)
        out[name] = bf16_bits(w)
    for tag, j, key in (("up", cfg.i - 1, 300), ("dn", cfg.i + 1, 310)):
        if 0 <= j < cfg.n:
            out["k_" + tag] = bf16_bits(_stream(s, key).standard_normal((batch, nq, C)))
            out["v_" + tag] = bf16_bits(_stream(s, key + 1).standard_normal((batch, nq, C)))
        else:
            out["k_" + tag] = None
            out["v_" + tag] = None
    return out


# ---------------------------------------------------------------------------
# ResNet block and the latent update of a step
# ---------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class ResnetConfig:
    """One band of an SDXL ResNet block: token grid H x W split in n bands,
    band i, c_in -> c_out channels, a T-wide time embedding."""
    name: str
    H: int
    W: int
    n: int
    i: int
    c_in: int
    c_out: int
    temb_dim: int = 1280
    groups: int = 32
    batch: int = 1
    seed_id: int = 80

    @property
    def h(self) -> int:
        return self.H // self.n


# SDXL's ResNets at the 2048 px image's first transformer level (128 x 128
# tokens of 640 channels, 8 bands): the plain one, and the first one of the
# level, which widens 320 channels to 640.
RESNET_CONFIGS = {
    "sdxl2048_l1_res640": ResnetConfig("sdxl2048_l1_res640", 128, 128, 8, 3, 640, 640, seed_id=80),
    "sdxl2048_l1_res320_640": ResnetConfig("sdxl2048_l1_res320_640", 128, 128, 8, 3, 320, 640, seed_id=81),
    # the other levels of the 2048 px image: 256 x 256 tokens of 320 channels
    # (no attention there), 64 x 64 tokens of 1280 channels (and the ResNet
    # entering it from 640 channels)
    "sdxl2048_l0_res320": ResnetConfig("sdxl2048_l0_res320", 256, 256, 8, 3, 320, 320, seed_id=89),
    "sdxl2048_l2_res1280": ResnetConfig("sdxl2048_l2_res1280", 64, 64, 8, 3, 1280, 1280, seed_id=90),
    "sdxl2048_l2_res640_1280": ResnetConfig("sdxl2048_l2_res640_1280", 64, 64, 8, 3, 640, 1280, seed_id=91),
    # the up path's first ResNet of each level, on the concatenation with the skip
    "sdxl2048_l2_res2560_1280": ResnetConfig("sdxl2048_l2_res2560_1280", 64, 64, 8, 3, 2560, 1280, seed_id=92),
    "sdxl2048_l1_res1920_640": ResnetConfig("sdxl2048_l1_res1920_640", 128, 128, 8, 3, 1920, 640, seed_id=93),
    "sdxl2048_l0_res960_320": ResnetConfig("sdxl2048_l0_res960_320", 256, 256, 8, 3, 960, 320, seed_id=94),
}


def resnet_weight_shapes(rc: ResnetConfig) -> Dict[str, tuple]:
    s = {
        "gn1_gamma": (rc.c_in,), "gn1_beta": (rc.c_in,),
        "conv1_w": (rc.c_out, 3, 3, rc.c_in), "conv1_b": (rc.c_out,),
        "temb_w": (rc.c_out, rc.temb_dim), "temb_b": (rc.c_out,),
        "gn2_gamma": (rc.c_out,), "gn2_beta": (rc.c_out,),
        "conv2_w": (rc.c_out, 3, 3, rc.c_out), "conv2_b": (rc.c_out,),
    }
    if rc.c_in != rc.c_out:
        s["skip_w"] = (rc.c_out, rc.c_in)
        s["skip_b"] = (rc.c_out,)
    return s


def resnet_inputs(rc: ResnetConfig, seed: Optional[int] = None) -> Dict[str, Optional[np.ndarray]]:
    """bf16 inputs of one ResNet-block call on band rc.i.

    x [B, h*W, c_in] ~ N(0, 1); temb [B, T] ~ N(0, 1); weights ~ N(0,
    1/fan_in) (fan_in = 9 c for a 3x3 kernel); biases ~ 0.02 N(0, 1); norm
    scales ~ 1 + 0.1 N(0, 1), shifts ~ 0.1 N(0, 1).  The neighbours' edge
    rows of the two convolution inputs ([B, 2, W, c], None at the image's
    edges) are N(0, 1) clipped below at -0.28, the range of SiLU's outputs.
    """
    s = BASE_SEED + rc.seed_id if seed is None else seed
    B, W = rc.batch, rc.W
    out: Dict[str, Optional[np.ndarray]] = {}
    out["x"] = bf16_bits(_stream(s, 400).standard_normal((B, rc.h * W, rc.c_in)))
    out["temb"] = bf16_bits(_stream(s, 401).standard_normal((B, rc.temb_dim)))
    for idx, (name, shape) in enumerate(resnet_weight_shapes(rc).items()):
        g = _stream(s, 500 + idx)
        if name.endswith("_w"):
            w = g.standard_normal(shape) / np.sqrt(np.prod(shape[1:]))
        elif name.endswith("_b") or name.endswith("_beta"):
            w = (0.02 if name.endswith("_b") else 0.1) * g.standard_normal(shape)
        else:
            w = 1.0 + 0.1 * g.standard_normal(shape)
        out[name] = bf16_bits(w)
    for k, (tag, c) in enumerate((("edges1", rc.c_in), ("edges2", rc.c_out))):
        for side, j in (("up", rc.i - 1), ("dn", rc.i + 1)):
            key = f"{tag}_{side}"
            if 0 <= j < rc.n:
                e = _stream(s, 600 + 2 * k + (side == "dn")).standard_normal((B, 2, W, c))
                out[key] = bf16_bits(np.maximum(e, -0.28))
            else:
                out[key] = None
    return out


def step_inputs(n: int, seed: int, with_noise: bool = True) -> Dict[str, Optional[np.ndarray]]:
    """float32 latent-update inputs: x_t, the two guidance branches' noise
    predictions and (optionally) the DDPM noise z, each n values ~ N(0, 1)."""
    out: Dict[str, Optional[np.ndarray]] = {}
    for k, name in enumerate(("x_t", "eps_uncond", "eps_cond", "z")):
        out[name] = _stream(seed, 700 + k).standard_normal(n).astype(np.float32)
    if not with_noise:
        out["z"] = None
    return out


def conv_inputs(H: int, W: int, n: int, i: int, c_in: int, c_out: int, batch: int, seed: int
                ) -> Dict[str, Optional[np.ndarray]]:
    """bf16 inputs of one 3x3 band convolution: x [B, h*W, c_in] ~ N(0, 1),
    the rows above / below the band [B, W, c_in] ~ N(0, 1) (None at the
    image's edges), weights [c_out, 3, 3, c_in] ~ N(0, 1/(9 c_in)), bias
    ~ 0.02 N(0, 1)."""
    s = BASE_SEED + seed
    h = H // n
    out: Dict[str, Optional[np.ndarray]] = {
        "x": bf16_bits(_stream(s, 800).standard_normal((batch, h * W, c_in))),
        "row_up": bf16_bits(_stream(s, 801).standard_normal((batch, W, c_in))) if i > 0 else None,
        "row_dn": bf16_bits(_stream(s, 802).standard_normal((batch, W, c_in))) if i < n - 1 else None,
        "w": bf16_bits(_stream(s, 803).standard_normal((c_out, 3, 3, c_in)) / np.sqrt(9 * c_in)),
        "b": bf16_bits(0.02 * _stream(s, 804).standard_normal(c_out)),
    }
    return out


# SDXL's resolution changes at 2048 px, 8 bands, band 3: the downsampler from
# level 0 (256 x 256 tokens, 320 channels) and the upsamplers into level 1
# and level 0, as (H, W, n, i, c_in, c_out, mode: 0 same, 1 down, 2 up).
CONV_CONFIGS = {
    "sdxl2048_down_l0": (256, 256, 8, 3, 320, 320, 1),
    "sdxl2048_up_l2": (64, 64, 8, 3, 1280, 1280, 2),
    "sdxl2048_up_l1": (128, 128, 8, 3, 640, 640, 2),
}


MODULE_WEIGHT_NAMES = ("gn_gamma", "gn_beta", "proj_in_w", "proj_in_b", "proj_out_w", "proj_out_b")


def module_inputs(bc: BlockConfig, depth: int, seed: Optional[int] = None, batch: int = 1):
    """bf16 inputs of one transformer-module call of the given depth: x, text
    and the module's own weights as block_inputs draws them for `seed`; basic
    block j's weights and stale neighbour K/V as block_inputs draws them for
    seed + 1000 + j.  Returns (x, text, module_weights, [block_weights],
    [(k_up, v_up, k_dn, v_dn)])."""
    s = BASE_SEED + bc.seed_id if seed is None else seed
    base = block_inputs(bc, seed=s, batch=batch)
    module = {k: base[k] for k in MODULE_WEIGHT_NAMES}
    blocks, stale = [], []
    for j in range(depth):
        bj = block_inputs(bc, seed=s + 1000 + j, batch=batch)
        blocks.append({k: bj[k] for k in BLOCK_WEIGHT_NAMES if k not in MODULE_WEIGHT_NAMES})
        stale.append((bj["k_up"], bj["v_up"], bj["k_dn"], bj["v_dn"]))
    return base["x"], base["text"], module, blocks, stale


# ---------------------------------------------------------------------------
# An SDXL-shaped U-Net on one band: topology and seeded random weights / stale
# neighbour data (shapes and draws only)
# ---------------------------------------------------------------------------

LATENT_PAD = 64   # the 4 latent channels, zero-padded to the convolution's granularity


@dataclasses.dataclass(frozen=True)
class UNetSpec:
    """channels / depths per level (depth 0: no attention at that level),
    the latent grid H0 x W0 split in n bands (band i), p of the attention."""
    name: str
    channels: tuple
    depths: tuple
    H0: int
    W0: int
    n: int
    i: int
    p: float = 0.25
    batch: int = 1
    temb_dim: int = 1280
    text_dim: int = 2048
    n_text: int = 77
    groups: int = 32
    seed_id: int = 120


UNET_SDXL_2048 = UNetSpec("sdxl2048_unet", (320, 640, 1280), (0, 2, 10), 256, 256, 8, 3)
UNET_TINY = UNetSpec("tiny_unet", (64, 128, 128), (0, 1, 1), 32, 16, 2, 1, p=0.5, temb_dim=64, text_dim=64,
                     n_text=7, seed_id=121)


def unet_layers(sp: UNetSpec):
    """SDXL's order of layers on one band: conv_in; per level two (ResNet
    [+ module]) pairs and a downsampler except at the last level; the middle
    (ResNet, module, ResNet); per level on the way up three (ResNet on the
    concatenation with a skip [+ module]) pairs and an upsampler except at
    level 0; the output GroupNorm + SiLU and conv_out.  Each entry: name,
    kind ('conv', 'resnet', 'module', 'gn'), grid H x W of its input, c_in,
    c_out, mode / depth, and whether its output is pushed as a skip or a skip
    is popped and concatenated to its input first."""
    L = []
    ch = sp.channels
    H, W = sp.H0, sp.W0
    c = ch[0]
    L.append(dict(name="conv_in", kind="conv", H=H, W=W, c_in=LATENT_PAD, c_out=c, mode=0, push=True))
    skip_ch = [c]
    for lv in range(len(ch)):
        for r in range(2):
            L.append(dict(name=f"down{lv}_res{r}", kind="resnet", H=H, W=W, c_in=c, c_out=ch[lv], level=lv,
                          push=sp.depths[lv] == 0))
            c = ch[lv]
            if sp.depths[lv]:
                L.append(dict(name=f"down{lv}_mod{r}", kind="module", H=H, W=W, c_in=c, c_out=c, level=lv,
                              depth=sp.depths[lv], push=True))
            skip_ch.append(c)
        if lv < len(ch) - 1:
            L.append(dict(name=f"down{lv}_ds", kind="conv", H=H, W=W, c_in=c, c_out=c, mode=1, push=True))
            H, W = H // 2, W // 2
            skip_ch.append(c)
    top = len(ch) - 1
    L.append(dict(name="mid_res0", kind="resnet", H=H, W=W, c_in=c, c_out=c, level=top))
    if sp.depths[top]:
        L.append(dict(name="mid_mod", kind="module", H=H, W=W, c_in=c, c_out=c, level=top, depth=sp.depths[top]))
    L.append(dict(name="mid_res1", kind="resnet", H=H, W=W, c_in=c, c_out=c, level=top))
    for lv in reversed(range(len(ch))):
        for r in range(3):
            sc = skip_ch.pop()
            L.append(dict(name=f"up{lv}_res{r}", kind="resnet", H=H, W=W, c_in=c + sc, c_out=ch[lv], level=lv,
                          pop=True, skip_c=sc))
            c = ch[lv]
            if sp.depths[lv]:
                L.append(dict(name=f"up{lv}_mod{r}", kind="module", H=H, W=W, c_in=c, c_out=c, level=lv,
                              depth=sp.depths[lv]))
        if lv > 0:
            L.append(dict(name=f"up{lv}_us", kind="conv", H=H, W=W, c_in=c, c_out=c, mode=2))
            H, W = 2 * H, 2 * W
    L.append(dict(name="out_gn", kind="gn", H=H, W=W, c_in=c, c_out=c))
    L.append(dict(name="conv_out", kind="conv", H=H, W=W, c_in=c, c_out=LATENT_PAD, mode=0))
    return L


def _w(g, shape, fan_in):
    return bf16_bits(g.standard_normal(shape) / np.sqrt(fan_in))


def _band_stats(g, n: int, B: int, G: int, count: float) -> np.ndarray:
    """Plausible (count, mean, M2) of every band's GroupNorm input, [n, B, G, 3]
    float32: means 0.1 N(0, 1), variances 0.8 + 0.4 U(0, 1)."""
    st = np.empty((n, B, G, 3))
    st[..., 0] = count
    st[..., 1] = 0.1 * g.standard_normal((n, B, G))
    st[..., 2] = count * (0.8 + 0.4 * g.random((n, B, G)))
    return st.astype(np.float32)


def unet_band_inputs(sp: UNetSpec, sync_gn: bool = False):
    """Seeded bf16 weights of every layer, the band's stale neighbour data
    for every layer, the padded latent band, the time embedding and the text:
    (weights, stale, latent, temb, text).  Draw recipe as the single layers'
    (weights N(0, 1/fan_in), biases 0.02 N, norm scales 1 + 0.1 N, shifts
    0.1 N, neighbour rows / K / V N(0, 1)); conv_in's weights are zero on the
    60 padding channels, conv_out's outputs beyond the first 4 are zero.
    With sync_gn, every GroupNorm also gets every band's statistics
    (_band_stats; entry i is replaced by the band's own in the step)."""
    s = BASE_SEED + sp.seed_id
    B = sp.batch

    def one(idx, ly):
        """Weights and stale data of layer idx, from the layer's own streams."""
        weights, stale = {}, {}
        g = _stream(s, 1000 + idx)
        h = ly["H"] // sp.n
        W, ci, co = ly["W"], ly["c_in"], ly["c_out"]
        up = sp.i > 0
        dn = sp.i < sp.n - 1
        rnd = lambda shape: bf16_bits(g.standard_normal(shape))
        if ly["kind"] == "conv":
            w = g.standard_normal((co, 3, 3, ci)) / np.sqrt(9 * ci)
            if ly["name"] == "conv_in":
                w[:, :, :, 4:] = 0.0
            if ly["name"] == "conv_out":
                w[4:] = 0.0
            b = 0.02 * g.standard_normal(co)
            if ly["name"] == "conv_out":
                b[4:] = 0.0
            weights[ly["name"]] = {"w": bf16_bits(w), "b": bf16_bits(b)}
            rows_up = rnd((B, W, ci)) if up else None
            rows_dn = rnd((B, W, ci)) if dn and ly["mode"] != 1 else None
            stale[ly["name"]] = {"row_up": rows_up, "row_dn": rows_dn}
        elif ly["kind"] == "resnet":
            rc = ResnetConfig(ly["name"], ly["H"], W, sp.n, sp.i, ci, co, temb_dim=sp.temb_dim, groups=sp.groups,
                              batch=B, seed_id=0)
            d = resnet_inputs(rc, seed=s + 2000 + idx)
            weights[ly["name"]] = {k: d[k] for k in resnet_weight_shapes(rc)}
            stale[ly["name"]] = {k: d[k] for k in ("edges1_up", "edges1_dn", "edges2_up", "edges2_dn")}
            if sync_gn:
                gs = _stream(s, 4000 + idx)
                stale[ly["name"]]["gn1_bands"] = _band_stats(gs, sp.n, B, sp.groups, h * W * ci / sp.groups)
                stale[ly["name"]]["gn2_bands"] = _band_stats(gs, sp.n, B, sp.groups, h * W * co / sp.groups)
        elif ly["kind"] == "module":
            heads = co // 64
            bc = BlockConfig(ly["name"], AttnConfig(name=ly["name"], H=ly["H"], W=W, n=sp.n, i=sp.i, p=sp.p,
                                                     heads=heads, d=64, dtype=DTYPE_BF16, seed_id=0),
                             n_text=sp.n_text, text_dim=sp.text_dim, ff_inner=4 * co, gn_groups=sp.groups, seed_id=0)
            _, _, module, blocks, st = module_inputs(bc, ly["depth"], seed=s + 3000 + 37 * idx, batch=B)
            weights[ly["name"]] = {"module": module, "blocks": blocks, "ff_inner": 4 * co, "heads": heads}
            stale[ly["name"]] = st
            if sync_gn:
                stale[ly["name"] + ":gn_bands"] = _band_stats(_stream(s, 4000 + idx), sp.n, B, sp.groups,
                                                              h * W * ci / sp.groups)
        else:  # the output GroupNorm
            weights[ly["name"]] = {"gamma": bf16_bits(1.0 + 0.1 * g.standard_normal(co)),
                                   "beta": bf16_bits(0.1 * g.standard_normal(co))}
            stale[ly["name"]] = {"gn_bands": _band_stats(_stream(s, 4000 + idx), sp.n, B, sp.groups,
                                                         h * W * co / sp.groups) if sync_gn else None}
        return weights, stale

    # Layers are independent draws: fill them on a few threads (numpy's
    # generators and array arithmetic release the GIL on large arrays); the
    # values do not depend on the order.
    import concurrent.futures
    layers = unet_layers(sp)
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        parts = list(ex.map(lambda a: one(*a), list(enumerate(layers))))
    weights, stale = {}, {}
    for w_, s_ in parts:
        weights.update(w_)
        stale.update(s_)
    g = _stream(s, 999)
    h0 = sp.H0 // sp.n
    lat = np.zeros((B, h0 * sp.W0, LATENT_PAD))
    lat[:, :, :4] = g.standard_normal((B, h0 * sp.W0, 4))
    temb = bf16_bits(g.standard_normal((B, sp.temb_dim)))
    text = bf16_bits(g.standard_normal((B, sp.n_text, sp.text_dim)))
    return weights, stale, bf16_bits(lat), temb, text
