"""CPU float64 oracle for the PCPP per-patch hot path.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this module.  It shares no code with
the GPU library: it imports nothing from the package and the package imports
nothing from here.

Everything is computed in float64 from the stored inputs (float32 values, or
bfloat16 bit patterns widened exactly), with plain loops or single library
primitives (numpy matmul, exp, scipy erf), in the order the paper states.

Citations are to arXiv 2412.02962 (Partially Conditioned Patch Parallelism):
Sec. 3.1 (Formulation, Eq. 1), Sec. 3.2 (Communication with only
neighbouring patches), Sec. 3.3 (Partially conditioned attention, Fig. 3).

Readings of points the paper leaves open (each also listed in the design
notes):
  R1  patches are row bands, patch 1 is the top band; the API is 0-based, so
      the paper's patch i is index i-1 here.
  R2  the number of context rows taken from a neighbour is
      r = min(h, floor(p*h + 1e-9)) when p*h is not a whole number.
  R3  p lies in [0, 1] for the neighbour form; the multi-hop form
      (context_rows_multihop) takes p up to max(1, n - 1), r image rows past
      each band edge, clipped to the image.
  R4  the exchanged tensors are the neighbours' key and value projections
      (Sec. 3.3: K and V are extended with stale keys and values), never Q.
  R6  the local patch's rows are always fresh; its own stale copy is unused.
  R7  edge patches get one-sided context, no wrap-around and no padding.
  R8  scaled dot-product attention uses scale 1/sqrt(d), no mask or bias.
  R11 the result does not depend on the diffusion step t; the warm-up steps
      (full-image attention) are the case n = 1.
  R15 block constants: GroupNorm 32 groups eps 1e-6 with affine; LayerNorm
      eps 1e-5 with affine; exact (erf) GELU; GEGLU = value * GELU(gate)
      with the value in the first half of the projection.
"""

from __future__ import annotations

import math
from typing import Dict, Optional, Tuple

import numpy as np
from scipy.special import erf

CTX_EPS = 1e-9


# ---------------------------------------------------------------------------
# Stored values -> float64
# ---------------------------------------------------------------------------

def from_bf16_bits(u16: np.ndarray) -> np.ndarray:
    """Widen bfloat16 bit patterns (uint16) to float64 exactly."""
    u = np.asarray(u16, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def as_f64(x: Optional[np.ndarray], dtype: str) -> Optional[np.ndarray]:
    """Stored tensor (float32, or uint16 bf16 bits) -> float64."""
    if x is None:
        return None
    if dtype == "bf16":
        return from_bf16_bits(x)
    return np.asarray(x, dtype=np.float64)


# ---------------------------------------------------------------------------
# Sec. 3.1 and Eq. 1: which rows form the neighbouring context
# ---------------------------------------------------------------------------

def context_rows(H: int, n: int, i: int, p: float) -> Tuple[int, int, int, int]:
    """Patch height and context row counts for 0-based patch i.

    Sec. 3.1: the H x W map is cut into n horizontal bands of h = H/n rows.
    Eq. 1: a patch is conditioned on the lower p*h rows of the patch above it
    (absent for the top patch) and the upper p*h rows of the patch below it
    (absent for the bottom patch).  Reading R2 fixes the row count when p*h
    is fractional.

    Returns (h, up, dn, rows): rows above taken from patch i-1, rows below
    taken from patch i+1, and the total rows of the key/value context.
    """
    if n <= 0 or H % n != 0:
        raise ValueError("H must be a positive multiple of n")
    if not (0 <= i < n):
        raise ValueError("patch index out of range")
    if not (0.0 <= p <= 1.0):  # also rejects NaN
        raise ValueError("p must lie in [0, 1]")
    h = H // n
    r = min(h, int(math.floor(p * h + CTX_EPS)))
    up = r if i > 0 else 0
    dn = r if i < n - 1 else 0
    return h, up, dn, up + h + dn


def context_token_ids(H: int, W: int, n: int, i: int, p: float) -> np.ndarray:
    """Global token ids (row*W + col) of the key/value context, ascending.

    The context rows of patch i are [i*h - up, (i+1)*h + dn): the neighbour
    rows above, the patch itself, the neighbour rows below (Eq. 1 plus the
    local patch, Sec. 3.3), each with every column.
    """
    h, up, dn, rows = context_rows(H, n, i, p)
    ids = []
    for row in range(i * h - up, (i + 1) * h + dn):
        for col in range(W):
            ids.append(row * W + col)
    return np.asarray(ids, dtype=np.int32)


def assemble_context(H: int, W: int, n: int, i: int, p: float,
                     fresh: np.ndarray, up: Optional[np.ndarray],
                     dn: Optional[np.ndarray]) -> np.ndarray:
    """Key (or value) tensor of the context, [B, rows*W, C] in token order.

    fresh: this patch's tensor of the current step, [B, h*W, C].
    up / dn: the stale tensor of the whole patch above / below, [B, h*W, C]
    (Sec. 3.2: the previous step's activations held in the receive buffers).
    The lower `up` rows of the patch above and the upper `dn` rows of the
    patch below are used (Eq. 1).
    """
    h, n_up, n_dn, _ = context_rows(H, n, i, p)
    parts = []
    if n_up > 0:
        parts.append(up[:, (h - n_up) * W:h * W, :])
    parts.append(fresh)
    if n_dn > 0:
        parts.append(dn[:, 0:n_dn * W, :])
    return np.concatenate(parts, axis=1)


def context_rows_multihop(H: int, n: int, i: int, p: float) -> Tuple[int, int, int, int]:
    """Row counts when p may exceed 1 (Sec. 6: context beyond the immediate
    neighbours).  Eq. 1 read with the patch boundaries dropped: the r =
    floor(p*h) image rows directly above the patch and directly below it,
    clipped to the image (reading R2 for the floor).  Returns (h, up, dn,
    rows); equals context_rows for p <= 1."""
    if n <= 0 or H % n != 0:
        raise ValueError("H must be a positive multiple of n")
    if not (0 <= i < n):
        raise ValueError("patch index out of range")
    if not (0.0 <= p <= max(1, n - 1)):
        raise ValueError("p must lie in [0, max(1, n - 1)]")
    h = H // n
    r = int(math.floor(p * h + CTX_EPS))
    up = min(r, i * h)
    dn = min(r, (n - 1 - i) * h)
    return h, up, dn, up + h + dn


def partial_attention_multihop(H: int, W: int, n: int, i: int, p: float, heads: int,
                               q: np.ndarray, k_fresh: np.ndarray, v_fresh: np.ndarray,
                               k_above: Optional[np.ndarray], v_above: Optional[np.ndarray],
                               k_below: Optional[np.ndarray], v_below: Optional[np.ndarray]):
    """Partially conditioned attention with the stale rows given compactly:
    k_above [B, up*W, C] = image rows i*h-up .. i*h-1, k_below [B, dn*W, C]
    = rows (i+1)*h .. (i+1)*h+dn-1 (context_rows_multihop)."""
    h, up, dn, _ = context_rows_multihop(H, n, i, p)
    kc = np.concatenate(([k_above] if up else []) + [k_fresh] + ([k_below] if dn else []), axis=1)
    vc = np.concatenate(([v_above] if up else []) + [v_fresh] + ([v_below] if dn else []), axis=1)
    return mha(q, kc, vc, heads)


# ---------------------------------------------------------------------------
# Sec. 3.2 with Eq. 1: the rows a patch's neighbours read from it
# ---------------------------------------------------------------------------

def boundary_messages(H: int, W: int, n: int, i: int, p: float,
                      k_fresh: np.ndarray, v_fresh: np.ndarray):
    """What patch i sends its two neighbours for their next step.

    Sec. 3.2: a patch exchanges its activations only with the neighbouring
    patches, which use them one step later as stale context.  Eq. 1 (seen
    from the neighbours): patch i-1 is conditioned on the upper rows of
    patch i, as many as patch i-1's own geometry takes from below; patch
    i+1 on the lower rows of patch i, as many as it takes from above.  Only
    those rows need to travel (the p-aware form of the exchange; the paper
    sends whole patches).

    k_fresh, v_fresh: [B, h*W, C].  Returns (to_up, to_dn), each
    [B, 2, rows*W, C] (keys, then values), or None when that neighbour does
    not exist or takes no rows.
    """
    h = H // n
    to_up = to_dn = None
    if i > 0:
        rows = context_rows(H, n, i - 1, p)[2]  # what patch i-1 takes from below
        if rows > 0:
            to_up = np.stack([k_fresh[:, :rows * W, :], v_fresh[:, :rows * W, :]], axis=1)
    if i < n - 1:
        rows = context_rows(H, n, i + 1, p)[1]  # what patch i+1 takes from above
        if rows > 0:
            to_dn = np.stack([k_fresh[:, (h - rows) * W:h * W, :], v_fresh[:, (h - rows) * W:h * W, :]],
                             axis=1)
    return to_up, to_dn


def place_boundary_messages(H: int, W: int, n: int, i: int, p: float,
                            from_up: Optional[np.ndarray], from_dn: Optional[np.ndarray],
                            k_up: np.ndarray, v_up: np.ndarray,
                            k_dn: np.ndarray, v_dn: np.ndarray):
    """Receiver side of boundary_messages for patch i.

    from_up was built by patch i-1 (its lower rows), from_dn by patch i+1
    (its upper rows).  They are written where Eq. 1 reads them: the last
    `up` rows of the stale buffer of the patch above, the first `dn` rows of
    that of the patch below.  Returns new (k_up, v_up, k_dn, v_dn); the
    inputs are not modified and their other rows are kept.
    """
    h, up, dn, _ = context_rows(H, n, i, p)
    k_up, v_up, k_dn, v_dn = (None if a is None else np.array(a, copy=True) for a in (k_up, v_up, k_dn, v_dn))
    if up > 0:
        k_up[:, (h - up) * W:h * W, :] = from_up[:, 0]
        v_up[:, (h - up) * W:h * W, :] = from_up[:, 1]
    if dn > 0:
        k_dn[:, :dn * W, :] = from_dn[:, 0]
        v_dn[:, :dn * W, :] = from_dn[:, 1]
    return k_up, v_up, k_dn, v_dn


def multihop_message_rows(H: int, n: int, i: int, p: float, j: int) -> Tuple[int, bool]:
    """How many rows of patch i patch j reads with multi-hop context
    (context_rows_multihop), and whether they are patch i's first rows
    (j above i) or its last rows (j below i)."""
    h = H // n
    if j == i or not (0 <= j < n):
        return 0, j < i
    _, up_j, dn_j, _ = context_rows_multihop(H, n, j, p)
    if j < i:   # patch j's context below reaches into patch i from its top
        return max(0, min(h, (j + 1) * h + dn_j - i * h)), True
    # patch j's context above reaches into patch i from its bottom
    return max(0, (i + 1) * h - max(i * h, j * h - up_j)), False


def multihop_message(H: int, W: int, n: int, i: int, p: float, j: int,
                     k_fresh: np.ndarray, v_fresh: np.ndarray) -> Optional[np.ndarray]:
    """What patch i sends patch j with multi-hop context: the rows of patch
    i that patch j's context holds, [B, 2, rows*W, C] (keys, then values), or
    None.  For |i - j| = 1 and p <= 1 these are boundary_messages."""
    rows, first = multihop_message_rows(H, n, i, p, j)
    if rows == 0:
        return None
    h = H // n
    sl = slice(0, rows * W) if first else slice((h - rows) * W, h * W)
    return np.stack([k_fresh[:, sl], v_fresh[:, sl]], axis=1)


def place_multihop_message(H: int, W: int, n: int, i: int, p: float, j: int, msg: np.ndarray,
                           k_above: np.ndarray, v_above: np.ndarray,
                           k_below: np.ndarray, v_below: np.ndarray):
    """Receiver side for patch i: writes patch j's message into copies of
    the compact stale blocks (rows i*h-up .. i*h-1 above, (i+1)*h ..
    (i+1)*h+dn-1 below) at the image rows it holds.  Returns the new
    (k_above, v_above, k_below, v_below)."""
    h, up, dn, _ = context_rows_multihop(H, n, i, p)
    rows, _ = multihop_message_rows(H, n, j, p, i)
    ka, va, kb, vb = (None if a is None else np.array(a, copy=True) for a in (k_above, v_above, k_below, v_below))
    if rows == 0:
        return ka, va, kb, vb
    if j < i:   # patch j's last rows: image rows (j+1)*h - rows .. (j+1)*h - 1
        off = (j + 1) * h - rows - (i * h - up)
        ka[:, off * W:(off + rows) * W] = msg[:, 0]
        va[:, off * W:(off + rows) * W] = msg[:, 1]
    else:       # patch j's first rows: image rows j*h .. j*h + rows - 1
        off = j * h - (i + 1) * h
        kb[:, off * W:(off + rows) * W] = msg[:, 0]
        vb[:, off * W:(off + rows) * W] = msg[:, 1]
    return ka, va, kb, vb


# ---------------------------------------------------------------------------
# Sec. 3.3: multi-head scaled dot-product attention over the context
# ---------------------------------------------------------------------------

def mha(q: np.ndarray, k: np.ndarray, v: np.ndarray, heads: int,
        return_probs: bool = False):
    """Multi-head scaled dot-product attention, float64.

    q [B, Nq, C], k and v [B, Nkv, C], C = heads * d, head a owns channels
    [a*d, (a+1)*d).  For every query: s_j = q.k_j / sqrt(d), softmax over j
    (max subtracted, R8), output = sum_j softmax_j * v_j.
    Returns O [B, Nq, C] (and the probabilities [B, heads, Nq, Nkv]).
    """
    B, nq, C = q.shape
    d = C // heads
    out = np.empty((B, nq, C), dtype=np.float64)
    probs = np.empty((B, heads, nq, k.shape[1])) if return_probs else None
    for b in range(B):
        for a in range(heads):
            qa = q[b, :, a * d:(a + 1) * d]
            ka = k[b, :, a * d:(a + 1) * d]
            va = v[b, :, a * d:(a + 1) * d]
            s = (qa @ ka.T) / math.sqrt(d)
            m = s.max(axis=1, keepdims=True)
            w = np.exp(s - m)
            pa = w / w.sum(axis=1, keepdims=True)
            out[b, :, a * d:(a + 1) * d] = pa @ va
            if return_probs:
                probs[b, a] = pa
    return (out, probs) if return_probs else out


def partial_attention(H: int, W: int, n: int, i: int, p: float, heads: int,
                      q: np.ndarray, k_fresh: np.ndarray, v_fresh: np.ndarray,
                      k_up: Optional[np.ndarray], v_up: Optional[np.ndarray],
                      k_dn: Optional[np.ndarray], v_dn: Optional[np.ndarray],
                      return_probs: bool = False):
    """Partially conditioned self-attention of patch i (Sec. 3.3, Fig. 3).

    Queries come from the local patch only; keys and values are the local
    fresh ones extended with the stale boundary slices of the neighbours
    given by Eq. 1.  All arrays float64.
    """
    kc = assemble_context(H, W, n, i, p, k_fresh, k_up, k_dn)
    vc = assemble_context(H, W, n, i, p, v_fresh, v_up, v_dn)
    return mha(q, kc, vc, heads, return_probs)


# ---------------------------------------------------------------------------
# Transformer block around the partial self-attention (SDXL-shaped; the
# paper names Attention, Convolution and Group Norm as the U-Net's layers,
# Sec. 3.3, and uses SDXL as the model, Sec. 4).
# ---------------------------------------------------------------------------

def group_norm(x: np.ndarray, groups: int, gamma: np.ndarray, beta: np.ndarray,
               eps: float = 1e-6) -> np.ndarray:
    """GroupNorm over the patch's tokens: x [B, N, C]; channels split into
    `groups` contiguous groups; statistics over (tokens x group channels),
    two passes (mean, then mean squared deviation, biased)."""
    B, N, C = x.shape
    cg = C // groups
    y = np.empty_like(x)
    for b in range(B):
        for g in range(groups):
            blk = x[b, :, g * cg:(g + 1) * cg]
            mean = blk.mean()
            var = ((blk - mean) ** 2).mean()
            y[b, :, g * cg:(g + 1) * cg] = (blk - mean) / math.sqrt(var + eps)
    return y * gamma + beta


def group_stats(x: np.ndarray, groups: int) -> np.ndarray:
    """Per image and group of a patch's tokens x [B, N, C]: (count, mean,
    M2) with M2 the sum of squared deviations from the mean; [B, groups, 3]."""
    B, N, C = x.shape
    cg = C // groups
    st = np.empty((B, groups, 3))
    for b in range(B):
        for g in range(groups):
            blk = x[b, :, g * cg:(g + 1) * cg]
            mean = blk.mean()
            st[b, g] = (blk.size, mean, ((blk - mean) ** 2).sum())
    return st


def group_norm_synchronized(x: np.ndarray, groups: int, gamma: np.ndarray, beta: np.ndarray,
                            band_stats: np.ndarray, i: int, eps: float = 1e-6) -> np.ndarray:
    """GroupNorm of patch i with statistics over the whole image.

    Sec. 3.3 keeps DistriFusion's synchronized GroupNorm: the statistics
    come from every patch, exchanged among all devices.  band_stats
    [n, B, groups, 3] holds each patch's (count, mean, M2) (the other
    patches' from the previous step, as exchanged); entry i is replaced by
    this patch's own statistics of x.  The whole-image mean is the
    count-weighted mean of the patch means, and the whole-image M2 is the sum
    of the patch M2 plus count * (patch mean - whole mean)^2 (law of total
    variance); variance = M2 / count (biased).
    """
    st = np.array(band_stats, dtype=np.float64, copy=True)
    st[i] = group_stats(x, groups)
    n_all = st[..., 0].sum(axis=0)                          # [B, G]
    mean = (st[..., 0] * st[..., 1]).sum(axis=0) / n_all
    m2 = (st[..., 2] + st[..., 0] * (st[..., 1] - mean[None]) ** 2).sum(axis=0)
    var = m2 / n_all
    B, N, C = x.shape
    cg = C // groups
    y = np.empty_like(x)
    for b in range(B):
        for g in range(groups):
            blk = x[b, :, g * cg:(g + 1) * cg]
            y[b, :, g * cg:(g + 1) * cg] = (blk - mean[b, g]) / math.sqrt(var[b, g] + eps)
    return y * gamma + beta


def layer_norm(x: np.ndarray, gamma: np.ndarray, beta: np.ndarray,
               eps: float = 1e-5) -> np.ndarray:
    """LayerNorm over the channel axis (last), biased variance."""
    mean = x.mean(axis=-1, keepdims=True)
    var = ((x - mean) ** 2).mean(axis=-1, keepdims=True)
    return (x - mean) / np.sqrt(var + eps) * gamma + beta


def linear(x: np.ndarray, w: np.ndarray, b: Optional[np.ndarray] = None) -> np.ndarray:
    """y = x w^T (+ b), w in [out, in] layout."""
    y = x @ w.T
    return y if b is None else y + b


def gelu(x: np.ndarray) -> np.ndarray:
    """Exact GELU: x * Phi(x) = 0.5 x (1 + erf(x / sqrt(2)))."""
    return 0.5 * x * (1.0 + erf(x / math.sqrt(2.0)))


def geglu(x: np.ndarray, w: np.ndarray, b: np.ndarray) -> np.ndarray:
    """GEGLU: project to 2F, value = first F, gate = last F, value*GELU(gate)."""
    hcat = linear(x, w, b)
    f = hcat.shape[-1] // 2
    return hcat[..., :f] * gelu(hcat[..., f:])


def transformer_block(H: int, W: int, n: int, i: int, p: float, heads: int,
                      wts: Dict[str, np.ndarray], x: np.ndarray, text: np.ndarray,
                      k_up: Optional[np.ndarray], v_up: Optional[np.ndarray],
                      k_dn: Optional[np.ndarray], v_dn: Optional[np.ndarray],
                      gn_groups: int = 32, gn_band_stats: Optional[np.ndarray] = None):
    """One SDXL-shaped transformer block on patch i, float64.

    x [B, h*W, C] (the patch's tokens), text [B, n_text, text_dim].
    Order: GroupNorm (patch-local statistics) -> proj_in -> LayerNorm ->
    Q, K, V of the local patch -> partial self-attention with the
    neighbours' stale K/V (Sec. 3.3) -> out-proj + residual -> LayerNorm ->
    cross-attention to the text -> out-proj + residual -> LayerNorm ->
    GEGLU feed-forward + residual -> proj_out + the block input.
    Returns (y, k_fresh, v_fresh): the output and the patch's own K and V,
    which the neighbours read as stale context at the next step (Sec. 3.2).
    With gn_band_stats [n, B, groups, 3] the GroupNorm is the synchronized
    one (group_norm_synchronized) instead of the patch-local one.
    """
    C = x.shape[-1]
    if gn_band_stats is None:
        t = group_norm(x, gn_groups, wts["gn_gamma"], wts["gn_beta"])
    else:
        t = group_norm_synchronized(x, gn_groups, wts["gn_gamma"], wts["gn_beta"], gn_band_stats, i)
    hid = linear(t, wts["proj_in_w"], wts["proj_in_b"])

    n1 = layer_norm(hid, wts["ln1_gamma"], wts["ln1_beta"])
    wqkv = wts["attn1_qkv_w"]
    q = linear(n1, wqkv[0:C])
    k = linear(n1, wqkv[C:2 * C])
    v = linear(n1, wqkv[2 * C:3 * C])
    a = partial_attention(H, W, n, i, p, heads, q, k, v, k_up, v_up, k_dn, v_dn)
    hid = hid + linear(a, wts["attn1_out_w"], wts["attn1_out_b"])

    n2 = layer_norm(hid, wts["ln2_gamma"], wts["ln2_beta"])
    q2 = linear(n2, wts["attn2_q_w"])
    wkv = wts["attn2_kv_w"]
    k2 = linear(text, wkv[0:C])
    v2 = linear(text, wkv[C:2 * C])
    a2 = mha(q2, k2, v2, heads)
    hid = hid + linear(a2, wts["attn2_out_w"], wts["attn2_out_b"])

    n3 = layer_norm(hid, wts["ln3_gamma"], wts["ln3_beta"])
    hid = hid + linear(geglu(n3, wts["ff1_w"], wts["ff1_b"]), wts["ff2_w"], wts["ff2_b"])

    y = linear(hid, wts["proj_out_w"], wts["proj_out_b"]) + x
    return y, k, v


MODULE_BLOCK_KEYS = ("ln1_gamma", "ln1_beta", "attn1_qkv_w", "attn1_out_w", "attn1_out_b",
                     "ln2_gamma", "ln2_beta", "attn2_q_w", "attn2_kv_w", "attn2_out_w", "attn2_out_b",
                     "ln3_gamma", "ln3_beta", "ff1_w", "ff1_b", "ff2_w", "ff2_b")


def transformer_module(H: int, W: int, n: int, i: int, p: float, heads: int,
                       module_wts: Dict[str, np.ndarray], block_wts, x: np.ndarray, text: np.ndarray,
                       stale, gn_groups: int = 32, gn_band_stats: Optional[np.ndarray] = None):
    """SDXL's transformer module of depth d = len(block_wts) on patch i,
    float64: GroupNorm -> proj_in -> d basic blocks -> proj_out + the module
    input.  Basic block j: LayerNorm -> Q, K, V of the local patch -> partial
    self-attention with the neighbours' stale K/V of that block (stale[j] =
    (k_up, v_up, k_dn, v_dn), Sec. 3.3) -> out-proj + residual -> LayerNorm ->
    cross-attention to the text -> out-proj + residual -> LayerNorm -> GEGLU
    feed-forward + residual.  module_wts holds gn_gamma, gn_beta, proj_in_w,
    proj_in_b, proj_out_w, proj_out_b; block_wts[j] the MODULE_BLOCK_KEYS.
    Returns (y, [K_j], [V_j]): every block's own K and V, what the neighbours
    read at the next step."""
    C = x.shape[-1]
    if gn_band_stats is None:
        t = group_norm(x, gn_groups, module_wts["gn_gamma"], module_wts["gn_beta"])
    else:
        t = group_norm_synchronized(x, gn_groups, module_wts["gn_gamma"], module_wts["gn_beta"], gn_band_stats, i)
    hid = linear(t, module_wts["proj_in_w"], module_wts["proj_in_b"])
    ks, vs = [], []
    for bw, (k_up, v_up, k_dn, v_dn) in zip(block_wts, stale):
        n1 = layer_norm(hid, bw["ln1_gamma"], bw["ln1_beta"])
        q = linear(n1, bw["attn1_qkv_w"][0:C])
        k = linear(n1, bw["attn1_qkv_w"][C:2 * C])
        v = linear(n1, bw["attn1_qkv_w"][2 * C:3 * C])
        hid = hid + linear(partial_attention(H, W, n, i, p, heads, q, k, v, k_up, v_up, k_dn, v_dn),
                           bw["attn1_out_w"], bw["attn1_out_b"])
        n2 = layer_norm(hid, bw["ln2_gamma"], bw["ln2_beta"])
        k2 = linear(text, bw["attn2_kv_w"][0:C])
        v2 = linear(text, bw["attn2_kv_w"][C:2 * C])
        hid = hid + linear(mha(linear(n2, bw["attn2_q_w"]), k2, v2, heads), bw["attn2_out_w"], bw["attn2_out_b"])
        n3 = layer_norm(hid, bw["ln3_gamma"], bw["ln3_beta"])
        hid = hid + linear(geglu(n3, bw["ff1_w"], bw["ff1_b"]), bw["ff2_w"], bw["ff2_b"])
        ks.append(k)
        vs.append(v)
    return linear(hid, module_wts["proj_out_w"], module_wts["proj_out_b"]) + x, ks, vs
