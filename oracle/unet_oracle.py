"""CPU float64 oracle for the rest of one per-band U-Net step: the 3x3
convolution with its halo rows, the SDXL-shaped ResNet block around two of
them, and the guided reverse-diffusion update.

TEST INFRASTRUCTURE ONLY, like the rest of this package: only the test
suite, the smoke check and the benchmark's CPU-baseline leg may use it, and
it shares no code with the GPU library.

Citations are to arXiv 2412.02962: Sec. 3.1 (classifier-free guidance,
Eq. 2; the reverse step, Eq. 3 and Eq. 4), Sec. 3.3 (the U-Net's layers are
attention, convolution and GroupNorm; convolutions keep DistriFusion's
exchange of boundary pixels), Sec. 4 (SDXL with a 50-step DDIM sampler and
guidance scale 5).

Readings (also in the design notes):
  R19 a 3x3 convolution of band i reads one row above and one row below the
      band: the neighbours' boundary rows of the convolution input as they
      were exchanged at the previous step (stale), zeros at the image's top
      and bottom and at its left and right edges.
  R20 ResNet block (SDXL's): GroupNorm (32 groups, eps 1e-5) -> SiLU ->
      conv 3x3 -> + linear(SiLU(time embedding)) per channel -> GroupNorm ->
      SiLU -> conv 3x3 -> + shortcut (the input, or a 1x1 convolution of it
      when the channel count changes).
  R21 the reverse step is Eq. 3 and Eq. 4 with beta_t = 1 - alpha_t; the
      DDIM sampler the experiments use is Song et al.'s deterministic update
      (eta = 0).
"""

from __future__ import annotations

import math
from typing import Dict, Optional, Tuple

import numpy as np

from .pcpp_oracle import group_norm, group_norm_synchronized, group_stats, linear


def silu(x: np.ndarray) -> np.ndarray:
    """SiLU(x) = x * sigmoid(x)."""
    return x / (1.0 + np.exp(-x))


# ---------------------------------------------------------------------------
# 3x3 convolution of one row band (Sec. 3.3: boundary pixels from neighbours)
# ---------------------------------------------------------------------------

def pad_band(x: np.ndarray, W: int, halo_up: Optional[np.ndarray],
             halo_dn: Optional[np.ndarray]) -> np.ndarray:
    """The band's input x [B, h*W, C] framed for a 3x3 convolution:
    [B, h+2, W+2, C] with the row above (halo_up [B, W, C], or zeros) on
    top, the row below (halo_dn, or zeros) at the bottom and zero columns at
    both sides (R19)."""
    B, N, C = x.shape
    h = N // W
    out = np.zeros((B, h + 2, W + 2, C))
    out[:, 1:h + 1, 1:W + 1] = x.reshape(B, h, W, C)
    if halo_up is not None:
        out[:, 0, 1:W + 1] = halo_up
    if halo_dn is not None:
        out[:, h + 1, 1:W + 1] = halo_dn
    return out


def conv3x3_band(x: np.ndarray, W: int, w: np.ndarray, b: Optional[np.ndarray],
                 halo_up: Optional[np.ndarray], halo_dn: Optional[np.ndarray]) -> np.ndarray:
    """out[b, y, x, o] = bias[o] + sum over taps (ky, kx) and channels c of
    w[o, ky, kx, c] * in[b, y + ky - 1, x + kx - 1, c], `in` being the framed
    band (pad_band).  w is [C_out, 3, 3, C_in] (tap-major, channel-minor).
    Returns [B, h*W, C_out]."""
    B, N, C = x.shape
    h = N // W
    xp = pad_band(x, W, halo_up, halo_dn)
    out = np.zeros((B, h, W, w.shape[0]))
    for ky in range(3):
        for kx in range(3):
            out += xp[:, ky:ky + h, kx:kx + W, :] @ w[:, ky, kx, :].T
    if b is not None:
        out += b
    return out.reshape(B, N, w.shape[0])


def conv3x3_band_mode(x: np.ndarray, W: int, w: np.ndarray, b: Optional[np.ndarray],
                      row_up: Optional[np.ndarray], row_dn: Optional[np.ndarray], mode: str) -> np.ndarray:
    """The U-Net's three 3x3 convolutions on a band x [B, h*W, C_in] (R19):
    'same'  stride 1 (ResNets, conv_in, conv_out): rows row_up / row_dn
            [B, W, C_in] (the neighbours' adjacent rows, or zeros) frame the band;
    'down'  stride 2, padding 1 (SDXL's downsampler): output (y, x) reads
            input rows 2y-1 .. 2y+1 and columns 2x-1 .. 2x+1, so only the row
            above is read; h and W even; output [B, (h/2)*(W/2), C_out];
    'up'    nearest 2x upsampling, then stride 1 (SDXL's upsampler): every
            input token becomes a 2 x 2 block, the neighbours' rows are
            upsampled the same way; output [B, (2h)*(2W), C_out]."""
    B, N, C = x.shape
    h = N // W
    if mode == "same":
        return conv3x3_band(x, W, w, b, row_up, row_dn)
    if mode == "down":
        xp = pad_band(x, W, row_up, None)           # [B, h+2, W+2, C]
        ho, wo = h // 2, W // 2
        out = np.zeros((B, ho, wo, w.shape[0]))
        for ky in range(3):
            for kx in range(3):
                out += xp[:, ky:ky + 2 * ho:2, kx:kx + 2 * wo:2, :] @ w[:, ky, kx, :].T
        if b is not None:
            out += b
        return out.reshape(B, ho * wo, w.shape[0])
    if mode == "up":
        g = np.repeat(np.repeat(x.reshape(B, h, W, C), 2, axis=1), 2, axis=2).reshape(B, 4 * N, C)
        up2 = lambda r: None if r is None else np.repeat(r, 2, axis=1)
        return conv3x3_band(g, 2 * W, w, b, up2(row_up), up2(row_dn))
    raise ValueError(mode)


def edge_rows(a: np.ndarray, W: int) -> np.ndarray:
    """What a band exports for its neighbours' next 3x3 convolution: its
    first and last rows of the convolution input a [B, h*W, C], as
    [B, 2, W, C] (row 0, then row h-1)."""
    B, N, C = a.shape
    h = N // W
    g = a.reshape(B, h, W, C)
    return np.stack([g[:, 0], g[:, h - 1]], axis=1)


# ---------------------------------------------------------------------------
# ResNet block (R20)
# ---------------------------------------------------------------------------

RESNET_GN_EPS = 1e-5


def resnet_block(W: int, wts: Dict[str, np.ndarray], x: np.ndarray, temb: np.ndarray,
                 edges1_up: Optional[np.ndarray], edges1_dn: Optional[np.ndarray],
                 edges2_up: Optional[np.ndarray], edges2_dn: Optional[np.ndarray],
                 groups: int = 32, i: int = 0,
                 gn1_band_stats: Optional[np.ndarray] = None,
                 gn2_band_stats: Optional[np.ndarray] = None, stats_out: Optional[list] = None):
    """One SDXL-shaped ResNet block on a row band, float64.

    x [B, h*W, C_in]; temb [B, T] (the step's time embedding).  edges*_up is
    the band above's export of the convolution input (edge_rows, [B, 2, W, C],
    its row 1 = its last row is read), edges*_dn the band below's (its row 0
    is read); None at the image's edge.  With gn*_band_stats [n, B, G, 3] the
    GroupNorm is the synchronized one (every band's statistics, this band's
    own, index i, in its place).
    Returns (y [B, h*W, C_out], edges1, edges2): the output and this band's
    own exports of the two convolution inputs.  stats_out, if a list, gets
    this band's own statistics of the two GroupNorm inputs (group_stats).
    """
    def gn(t, gamma, beta, stats):
        if stats is None:
            return group_norm(t, groups, gamma, beta, eps=RESNET_GN_EPS)
        return group_norm_synchronized(t, groups, gamma, beta, stats, i, eps=RESNET_GN_EPS)

    if stats_out is not None:
        stats_out.append(group_stats(x, groups))
    a1 = silu(gn(x, wts["gn1_gamma"], wts["gn1_beta"], gn1_band_stats))
    hid = conv3x3_band(a1, W, wts["conv1_w"], wts["conv1_b"],
                       None if edges1_up is None else edges1_up[:, 1],
                       None if edges1_dn is None else edges1_dn[:, 0])
    hid = hid + linear(silu(temb), wts["temb_w"], wts["temb_b"])[:, None, :]
    if stats_out is not None:
        stats_out.append(group_stats(hid, groups))
    a2 = silu(gn(hid, wts["gn2_gamma"], wts["gn2_beta"], gn2_band_stats))
    hid = conv3x3_band(a2, W, wts["conv2_w"], wts["conv2_b"],
                       None if edges2_up is None else edges2_up[:, 1],
                       None if edges2_dn is None else edges2_dn[:, 0])
    skip = x if "skip_w" not in wts else linear(x, wts["skip_w"], wts["skip_b"])
    return skip + hid, edge_rows(a1, W), edge_rows(a2, W)


# ---------------------------------------------------------------------------
# Guided reverse step (Eq. 2, Eq. 3, Eq. 4; R21)
# ---------------------------------------------------------------------------

def guided_noise(eps_uncond: np.ndarray, eps_cond: np.ndarray, s: float) -> np.ndarray:
    """Eq. 2: the unconditional prediction plus s times the difference of the
    conditional and the unconditional one."""
    return eps_uncond + s * (eps_cond - eps_uncond)


def reverse_step_ddpm(x_t: np.ndarray, eps_uncond: np.ndarray, eps_cond: np.ndarray, s: float,
                      alpha_t: float, alphabar_t: float, sigma_t: float,
                      z: Optional[np.ndarray]) -> np.ndarray:
    """Eq. 3 then Eq. 4: mu = (x_t - beta_t / sqrt(1 - alphabar_t) * eps) /
    sqrt(alpha_t) with beta_t = 1 - alpha_t, then x_{t-1} = mu + sigma_t z."""
    e = guided_noise(eps_uncond, eps_cond, s)
    mu = (x_t - (1.0 - alpha_t) / math.sqrt(1.0 - alphabar_t) * e) / math.sqrt(alpha_t)
    return mu if z is None else mu + sigma_t * z


def reverse_step_ddim(x_t: np.ndarray, eps_uncond: np.ndarray, eps_cond: np.ndarray, s: float,
                      alphabar_t: float, alphabar_prev: float) -> np.ndarray:
    """Deterministic DDIM (Song et al., eta = 0) with the guided noise of
    Eq. 2: the predicted clean sample x0 = (x_t - sqrt(1 - alphabar_t) eps) /
    sqrt(alphabar_t), re-noised to the previous level: sqrt(alphabar_prev) x0
    + sqrt(1 - alphabar_prev) eps."""
    e = guided_noise(eps_uncond, eps_cond, s)
    x0 = (x_t - math.sqrt(1.0 - alphabar_t) * e) / math.sqrt(alphabar_t)
    return math.sqrt(alphabar_prev) * x0 + math.sqrt(1.0 - alphabar_prev) * e


def scaled_linear_alphabar(n_train: int = 1000, beta_start: float = 0.00085,
                           beta_end: float = 0.012) -> np.ndarray:
    """SDXL's training noise schedule: betas on a line in sqrt space from
    beta_start to beta_end, alphabar_t = prod_{s <= t} (1 - beta_s)."""
    betas = np.linspace(math.sqrt(beta_start), math.sqrt(beta_end), n_train) ** 2
    return np.cumprod(1.0 - betas)


def resnet_weight_shapes(c_in: int, c_out: int, temb_dim: int) -> Dict[str, Tuple[int, ...]]:
    """Shapes of the ResNet block's weights, in the layout the oracle and the
    library use: linears [out, in], 3x3 kernels [C_out, 3, 3, C_in]."""
    s = {
        "gn1_gamma": (c_in,), "gn1_beta": (c_in,),
        "conv1_w": (c_out, 3, 3, c_in), "conv1_b": (c_out,),
        "temb_w": (c_out, temb_dim), "temb_b": (c_out,),
        "gn2_gamma": (c_out,), "gn2_beta": (c_out,),
        "conv2_w": (c_out, 3, 3, c_out), "conv2_b": (c_out,),
    }
    if c_in != c_out:
        s["skip_w"] = (c_out, c_in)
        s["skip_b"] = (c_out,)
    return s


# ---------------------------------------------------------------------------
# One band's U-Net forward (SDXL's order of layers), float64
# ---------------------------------------------------------------------------

def unet_band_step(layers, n: int, i: int, p: float, groups: int, weights, stale,
                   latent: np.ndarray, temb: np.ndarray, text: np.ndarray, sync_gn: bool = False,
                   exports: Optional[dict] = None) -> np.ndarray:
    """The noise prediction of band i: the layers in order (`layers`, a list
    of dicts: name, kind 'conv' / 'resnet' / 'module' / 'gn', input grid H x
    W, channels, conv mode, module depth, push / pop of skip connections),
    each with its weights and the band's stale neighbour data of the previous
    step (convolution rows, ResNet edge rows, every basic block's K/V).  The
    up path concatenates its state with the skip along the channels before
    its ResNets.  GroupNorms use the band's own statistics, or with sync_gn
    the synchronized ones (every band's statistics from stale: a ResNet's
    gn1_bands / gn2_bands, stale[module + ':gn_bands'], the head's gn_bands).
    latent [B, h*W, 64] (4 channels, zero-padded); returns [B, h*W, 64].
    exports, if a dict, gets per layer what the neighbours read at the next
    step (Sec. 3.2): a convolution's first and last input rows, a ResNet's
    edges1 / edges2, a module's per-block K and V, and the band's own
    GroupNorm statistics ('gn', a list in the layer's order)."""
    from .pcpp_oracle import group_norm as _gn, group_norm_synchronized as _gns, transformer_module as _module
    modes = {0: "same", 1: "down", 2: "up"}
    hcur = latent
    skips = []
    for ly in layers:
        name, kind, W = ly["name"], ly["kind"], ly["W"]
        w = weights[name]
        if kind == "conv":
            st = stale[name]
            if exports is not None:
                rows = hcur.reshape(hcur.shape[0], -1, W, hcur.shape[2])
                exports[name] = {"first": rows[:, 0], "last": rows[:, -1]}
            out = conv3x3_band_mode(hcur, W, w["w"], w["b"], st["row_up"], st["row_dn"], modes[ly["mode"]])
        elif kind == "resnet":
            if ly.get("pop"):
                hcur = np.concatenate([hcur, skips.pop()], axis=-1)
            st = stale[name]
            stats = []
            out, e1, e2 = resnet_block(W, w, hcur, temb, st["edges1_up"], st["edges1_dn"], st["edges2_up"],
                                       st["edges2_dn"], groups=groups, i=i,
                                       gn1_band_stats=st["gn1_bands"] if sync_gn else None,
                                       gn2_band_stats=st["gn2_bands"] if sync_gn else None, stats_out=stats)
            if exports is not None:
                exports[name] = {"edges1": e1, "edges2": e2, "gn": stats}
        elif kind == "module":
            out, ks, vs = _module(ly["H"], W, n, i, p, w["heads"], w["module"], w["blocks"], hcur, text,
                                  stale[name], gn_groups=groups,
                                  gn_band_stats=stale[name + ":gn_bands"] if sync_gn else None)
            if exports is not None:
                exports[name] = {"k": ks, "v": vs, "gn": [group_stats(hcur, groups)]}
        else:
            if exports is not None:
                exports[name] = {"gn": [group_stats(hcur, groups)]}
            if sync_gn:
                out = silu(_gns(hcur, groups, w["gamma"], w["beta"], stale[name]["gn_bands"], i, eps=RESNET_GN_EPS))
            else:
                out = silu(_gn(hcur, groups, w["gamma"], w["beta"], eps=RESNET_GN_EPS))
        if ly.get("push"):
            skips.append(out)
        hcur = out
    return hcur


def image_step(layers, n: int, p: float, groups: int, weights, prev, latents, temb: np.ndarray,
               text: np.ndarray, sync_gn: bool = False):
    """One denoising step of the whole image under PCPP (Sec. 3.1-3.3): every
    band i runs unet_band_step with the stale data its neighbours exported
    at the previous step (Sec. 3.2: the step's exchange).  prev[j] is band
    j's exports of that step, or prev is None before the first step: then
    nothing has been received and, as in Fig. 1 where no synchronous warm-up
    step runs, the bands are computed separately: the attention takes no
    stale rows (p = 0 for this step), the convolutions see zero rows beyond
    the band (the zero padding of an image of its own) and the GroupNorms
    the band's own statistics (the others have count 0).  latents[i] is band
    i's [B, h*W, 64] input.  Returns (outputs, exports), one per band.
    Band i reads from band i-1 the last rows it exported (convolutions: its
    last input row; ResNets: its edge rows, of which the last is used; the
    attention: its K/V, of which the last r rows are used) and from band i+1
    the first ones; with sync_gn every band's statistics of every GroupNorm.
    """
    def nb_export(j, name):
        if j < 0 or j >= n or prev is None or prev[j] is None:
            return None
        return prev[j][name]

    outs, exps = [], []
    for i in range(n):
        B = latents[i].shape[0]
        stale = {}
        for ly in layers:
            name, kind, H, W, ci, co = ly["name"], ly["kind"], ly["H"], ly["W"], ly["c_in"], ly["c_out"]
            h = H // n
            up, dn = nb_export(i - 1, name), nb_export(i + 1, name)

            def gn_stack(k):  # [n, B, G, 3]: entry j = band j's k-th statistics (count 0 if none)
                st = np.zeros((n, B, groups, 3))
                for j in range(n):
                    e = nb_export(j, name)
                    if e is not None:
                        st[j] = e["gn"][k]
                return st

            if kind == "conv":
                zero = np.zeros((B, W, ci))
                stale[name] = {"row_up": (up["last"] if up else zero) if i > 0 else None,
                               "row_dn": (dn["first"] if dn else zero) if i < n - 1 and ly["mode"] != 1 else None}
            elif kind == "resnet":
                z1, z2 = np.zeros((B, 2, W, ci)), np.zeros((B, 2, W, co))
                stale[name] = {"edges1_up": (up["edges1"] if up else z1) if i > 0 else None,
                               "edges1_dn": (dn["edges1"] if dn else z1) if i < n - 1 else None,
                               "edges2_up": (up["edges2"] if up else z2) if i > 0 else None,
                               "edges2_dn": (dn["edges2"] if dn else z2) if i < n - 1 else None}
                if sync_gn:
                    stale[name]["gn1_bands"], stale[name]["gn2_bands"] = gn_stack(0), gn_stack(1)
            elif kind == "module":
                st = []
                for j in range(ly["depth"]):
                    ku = up["k"][j] if up else None
                    vu = up["v"][j] if up else None
                    kd = dn["k"][j] if dn else None
                    vd = dn["v"][j] if dn else None
                    st.append((ku, vu, kd, vd))
                stale[name] = st
                if sync_gn:
                    stale[name + ":gn_bands"] = gn_stack(0)
            else:
                stale[name] = {"gn_bands": gn_stack(0) if sync_gn else None}
        ex = {}
        p_step = p if prev is not None else 0.0
        outs.append(unet_band_step(layers, n, i, p_step, groups, weights, stale, latents[i], temb, text,
                                   sync_gn=sync_gn, exports=ex))
        exps.append(ex)
    return outs, exps
