// C ABI entry points of the PCPP library: argument validation, Eq. 1
// geometry, and kernel launches on the caller's stream.
//
// Everything here runs on the host.  Validation completes before anything
// is enqueued, so an error return leaves the outputs untouched.

#include <math.h>
#include <stdint.h>
#include <stdlib.h>

#include "../../include/pcpp.h"
#include "api_internal.h"
#include "kernels.h"

#define PCPP_EXPORT extern "C" __attribute__((visibility("default")))

namespace pcpp {

// Sec. 3.1: h = H/n.  Eq. 1: r = p*h rows from each existing neighbour; a
// fractional p*h is floored (the small epsilon keeps decimal fractions such
// as p = 0.29, h = 100 at their exact value).
int validate_geom(const pcpp_geom_t* g, Geo* out) { return validate_geom_hops(g, false, out); }

// With multi_hop, p may exceed 1: context reaching past the neighbours (the
// extension Sec. 6 hypothesises for many bands), up to the whole image at
// p = n - 1.  r = floor(p*h + 1e-9) rows above and below the band, clipped
// to the image.
int validate_geom_hops(const pcpp_geom_t* g, bool multi_hop, Geo* out) {
    if (g == nullptr) return PCPP_EINVAL;
    if (g->reserved != 0) return PCPP_EINVAL;
    if (g->n_patches < 1 || g->H < 1 || g->W < 1) return PCPP_EINVAL;
    if (g->H % g->n_patches != 0) return PCPP_EINVAL;
    if (g->patch_idx < 0 || g->patch_idx >= g->n_patches) return PCPP_EINVAL;
    const double p_max = multi_hop ? (double)(g->n_patches - 1 > 1 ? g->n_patches - 1 : 1) : 1.0;
    if (!(g->partial >= 0.0 && g->partial <= p_max)) return PCPP_EINVAL;  // NaN fails too
    if (g->heads < 1 || g->head_dim < 1 || g->batch < 1 || g->step < 0) return PCPP_EINVAL;
    if ((int64_t)g->H * g->W > INT32_MAX / 2) return PCPP_EINVAL;
    if ((int64_t)g->heads * g->head_dim > (1 << 20)) return PCPP_EINVAL;
    Geo r;
    r.h = g->H / g->n_patches;
    const double rows = floor(g->partial * (double)r.h + 1e-9);
    if (multi_hop) {
        const int64_t ctx = (int64_t)rows;
        const int64_t above = (int64_t)g->patch_idx * r.h, below = (int64_t)(g->n_patches - 1 - g->patch_idx) * r.h;
        r.up = (int32_t)(ctx < above ? ctx : above);
        r.dn = (int32_t)(ctx < below ? ctx : below);
    } else {
        const int32_t ctx = rows >= (double)r.h ? r.h : (int32_t)rows;
        r.up = g->patch_idx > 0 ? ctx : 0;
        r.dn = g->patch_idx < g->n_patches - 1 ? ctx : 0;
    }
    r.nq = r.h * g->W;
    r.n_kv = (r.up + r.h + r.dn) * g->W;
    r.C = g->heads * g->head_dim;
    r.esize = g->dtype == PCPP_DTYPE_BF16 ? 2 : 4;
    if (out) *out = r;
    return PCPP_OK;
}

KvSource make_kv_source(const pcpp_geom_t* g, const Geo& r, const void* k_fresh, const void* v_fresh,
                        const void* k_up, const void* v_up, const void* k_dn, const void* v_dn) {
    KvSource s;
    const int64_t band = (int64_t)r.nq * r.C;  // elements of one whole band
    const int64_t skip_up = (int64_t)(r.h - r.up) * g->W * r.C * r.esize;
    s.k[0] = (r.up > 0 && k_up) ? (const char*)k_up + skip_up : nullptr;
    s.v[0] = (r.up > 0 && v_up) ? (const char*)v_up + skip_up : nullptr;
    s.k[1] = k_fresh;
    s.v[1] = v_fresh;
    s.k[2] = r.dn > 0 ? k_dn : nullptr;
    s.v[2] = r.dn > 0 ? v_dn : nullptr;
    s.bstride[0] = s.bstride[1] = s.bstride[2] = band;
    s.end0 = r.up * g->W;
    s.end1 = (r.up + r.h) * g->W;
    s.n_kv = r.n_kv;
    return s;
}

// Key/value sources from compact stale rows: the up rows directly above the
// band and the dn rows directly below it, each [B, rows*W, C].
KvSource make_kv_source_compact(const pcpp_geom_t* g, const Geo& r, const void* k_fresh, const void* v_fresh,
                                const void* k_above, const void* v_above, const void* k_below,
                                const void* v_below) {
    KvSource s;
    s.k[0] = r.up > 0 ? k_above : nullptr;
    s.v[0] = r.up > 0 ? v_above : nullptr;
    s.k[1] = k_fresh;
    s.v[1] = v_fresh;
    s.k[2] = r.dn > 0 ? k_below : nullptr;
    s.v[2] = r.dn > 0 ? v_below : nullptr;
    s.bstride[0] = (int64_t)r.up * g->W * r.C;
    s.bstride[1] = (int64_t)r.nq * r.C;
    s.bstride[2] = (int64_t)r.dn * g->W * r.C;
    s.end0 = r.up * g->W;
    s.end1 = (r.up + r.h) * g->W;
    s.n_kv = r.n_kv;
    return s;
}

static bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Shared argument checks of the attention entry points.
int check_attention(const pcpp_geom_t* g, Geo* r, const void* q, const void* k_fresh,
                           const void* v_fresh, const void* k_up, const void* v_up, const void* k_dn,
                           const void* v_dn, const void* out) {
    int st = validate_geom(g, r);
    if (st != PCPP_OK) return st;
    if (g->dtype != PCPP_DTYPE_BF16 && g->dtype != PCPP_DTYPE_F32) return PCPP_ENOTSUP;
    if (g->head_dim != 64) return PCPP_ENOTSUP;
    if (!q || !k_fresh || !v_fresh || !out) return PCPP_EINVAL;
    if (r->up > 0 && (!k_up || !v_up)) return PCPP_EINVAL;
    if (r->dn > 0 && (!k_dn || !v_dn)) return PCPP_EINVAL;
    if (g->heads > 65535 || g->batch > 65535) return PCPP_EINVAL;
    const void* ptrs[8] = {q, k_fresh, v_fresh, k_up, v_up, k_dn, v_dn, out};
    for (const void* p : ptrs)
        if (p && !aligned16(p)) return PCPP_EINVAL;
    return PCPP_OK;
}

AttnParams make_attn_params(const pcpp_geom_t* g, const Geo& r, const void* q, void* out,
                            const KvSource& kv) {
    AttnParams p;
    p.q = q;
    p.out = out;
    p.q_bstride = (int64_t)r.nq * r.C;
    p.nq = r.nq;
    p.C = r.C;
    p.heads = g->heads;
    p.batch = g->batch;
    p.kv = kv;
    p.scale = (float)(1.0 / sqrt((double)g->head_dim));
    p.scale_log2 = (float)(1.4426950408889634 / sqrt((double)g->head_dim));
    return p;
}

}  // namespace pcpp

using namespace pcpp;

PCPP_EXPORT int pcpp_version(void) { return PCPP_VERSION; }

PCPP_EXPORT const char* pcpp_strerror(int status) {
    switch (status) {
        case PCPP_OK: return "ok";
        case PCPP_EINVAL: return "invalid argument (geometry, partial value, pointer or alignment)";
        case PCPP_ENOTSUP: return "unsupported head_dim, dtype or shape";
        case PCPP_EWORKSPACE: return "workspace missing or too small";
        case PCPP_EHIP: return "HIP runtime or kernel launch failure";
        default: return "unknown status";
    }
}

PCPP_EXPORT int pcpp_context_rows(const pcpp_geom_t* g, int32_t* h, int32_t* up, int32_t* dn,
                                  int32_t* n_kv) {
    Geo r;
    int st = validate_geom(g, &r);
    if (st != PCPP_OK) return st;
    if (h) *h = r.h;
    if (up) *up = r.up;
    if (dn) *dn = r.dn;
    if (n_kv) *n_kv = r.n_kv;
    return PCPP_OK;
}

PCPP_EXPORT int pcpp_gather_context(const pcpp_geom_t* g, const void* k_fresh, const void* v_fresh,
                                    const void* k_up, const void* v_up, const void* k_dn,
                                    const void* v_dn, int32_t* idx_out, void* k_ctx, void* v_ctx,
                                    void* stream) {
    Geo r;
    int st = validate_geom(g, &r);
    if (st != PCPP_OK) return st;
    if (g->dtype != PCPP_DTYPE_BF16 && g->dtype != PCPP_DTYPE_F32) return PCPP_ENOTSUP;
    if ((k_ctx == nullptr) != (v_ctx == nullptr)) return PCPP_EINVAL;
    if (k_ctx == nullptr && idx_out == nullptr) return PCPP_EINVAL;  // nothing to do
    if (k_ctx != nullptr) {
        if (!k_fresh || !v_fresh) return PCPP_EINVAL;
        if (r.up > 0 && (!k_up || !v_up)) return PCPP_EINVAL;
        if (r.dn > 0 && (!k_dn || !v_dn)) return PCPP_EINVAL;
    }
    if (g->batch > 65535) return PCPP_EINVAL;
    GatherParams p;
    p.src = make_kv_source(g, r, k_fresh, v_fresh, k_up, v_up, k_dn, v_dn);
    p.k_ctx = k_ctx;
    p.v_ctx = v_ctx;
    p.idx = idx_out;
    p.idx_base = (g->patch_idx * r.h - r.up) * g->W;
    p.C = r.C;
    p.batch = g->batch;
    p.esize = r.esize;
    return launch_gather(p, (hipStream_t)stream) == hipSuccess ? PCPP_OK : PCPP_EHIP;
}

PCPP_EXPORT size_t pcpp_partial_attention_workspace_size(const pcpp_geom_t* g) {
    Geo r;
    if (validate_geom(g, &r) != PCPP_OK) return 0;
    if (g->dtype != PCPP_DTYPE_BF16 || g->head_dim != 64) return 0;
    KvSource kv = make_kv_source(g, r, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr);
    return attention_bf16_ws_bytes(make_attn_params(g, r, nullptr, nullptr, kv));
}

PCPP_EXPORT int pcpp_partial_attention_plan(const pcpp_geom_t* g, int32_t cus, int32_t cus_enabled, void* stream,
                                            int32_t* block_queries, int32_t* pieces, int32_t* workgroups) {
    Geo r;
    int st = validate_geom(g, &r);
    if (st != PCPP_OK) return st;
    if (g->dtype != PCPP_DTYPE_BF16 || g->head_dim != 64) return PCPP_ENOTSUP;
    if (cus < 0 || (cus > 0 && cus_enabled < 0)) return PCPP_EINVAL;
    DeviceLayout d;
    if (cus > 0) {
        d = layout_for(cus, cus_enabled);
    } else {
        d = device_layout((hipStream_t)stream);
        if (device_cus() <= 0) return PCPP_EHIP;
    }
    KvSource kv = make_kv_source(g, r, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr);
    const AttnPlanInfo pi = attention_bf16_plan(make_attn_params(g, r, nullptr, nullptr, kv), d);
    if (block_queries) *block_queries = pi.block_queries;
    if (pieces) *pieces = pi.pieces;
    if (workgroups) *workgroups = pi.workgroups;
    return PCPP_OK;
}

PCPP_EXPORT size_t pcpp_partial_attention_multihop_workspace_size(const pcpp_geom_t* g) {
    Geo r;
    if (validate_geom_hops(g, true, &r) != PCPP_OK) return 0;
    if (g->dtype != PCPP_DTYPE_BF16 || g->head_dim != 64) return 0;
    KvSource kv = make_kv_source_compact(g, r, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr);
    return attention_bf16_ws_bytes(make_attn_params(g, r, nullptr, nullptr, kv));
}

PCPP_EXPORT int pcpp_partial_attention_multihop(const pcpp_geom_t* g, const void* q, const void* k_fresh,
                                                const void* v_fresh, const void* k_above, const void* v_above,
                                                const void* k_below, const void* v_below, void* out,
                                                void* workspace, size_t ws_bytes, void* stream) {
    Geo r;
    int st = validate_geom_hops(g, true, &r);
    if (st != PCPP_OK) return st;
    if (g->dtype != PCPP_DTYPE_BF16 && g->dtype != PCPP_DTYPE_F32) return PCPP_ENOTSUP;
    if (g->head_dim != 64) return PCPP_ENOTSUP;
    if (!q || !k_fresh || !v_fresh || !out) return PCPP_EINVAL;
    if (r.up > 0 && (!k_above || !v_above)) return PCPP_EINVAL;
    if (r.dn > 0 && (!k_below || !v_below)) return PCPP_EINVAL;
    if (g->heads > 65535 || g->batch > 65535) return PCPP_EINVAL;
    const void* ptrs[8] = {q, k_fresh, v_fresh, k_above, v_above, k_below, v_below, out};
    for (const void* p : ptrs)
        if (p && !aligned16(p)) return PCPP_EINVAL;
    KvSource kv = make_kv_source_compact(g, r, k_fresh, v_fresh, k_above, v_above, k_below, v_below);
    AttnParams p = make_attn_params(g, r, q, out, kv);
    hipError_t e;
    if (g->dtype == PCPP_DTYPE_BF16) {
        const size_t need = attention_bf16_ws_bytes(p);
        if (workspace == nullptr || ws_bytes < need) return PCPP_EWORKSPACE;
        if (!aligned16(workspace)) return PCPP_EINVAL;
        e = launch_attention_bf16(p, workspace, ws_bytes, (hipStream_t)stream);
    } else {
        e = launch_attention_f32(p, (hipStream_t)stream);
    }
    return e == hipSuccess ? PCPP_OK : PCPP_EHIP;
}

PCPP_EXPORT int pcpp_partial_attention(const pcpp_geom_t* g, const void* q, const void* k_fresh,
                                       const void* v_fresh, const void* k_up, const void* v_up,
                                       const void* k_dn, const void* v_dn, void* out, void* workspace,
                                       size_t ws_bytes, void* stream) {
    Geo r;
    int st = check_attention(g, &r, q, k_fresh, v_fresh, k_up, v_up, k_dn, v_dn, out);
    if (st != PCPP_OK) return st;
    KvSource kv = make_kv_source(g, r, k_fresh, v_fresh, k_up, v_up, k_dn, v_dn);
    AttnParams p = make_attn_params(g, r, q, out, kv);
    hipError_t e;
    if (g->dtype == PCPP_DTYPE_BF16) {
        const size_t need = attention_bf16_ws_bytes(p);
        if (workspace == nullptr || ws_bytes < need) return PCPP_EWORKSPACE;
        if (!aligned16(workspace)) return PCPP_EINVAL;
        e = launch_attention_bf16(p, workspace, ws_bytes, (hipStream_t)stream);
    } else {
        e = launch_attention_f32(p, (hipStream_t)stream);
    }
    return e == hipSuccess ? PCPP_OK : PCPP_EHIP;
}

// ---------------------------------------------------------------------------
// p-aware boundary messages (Sec. 3.2 with Eq. 1)
// ---------------------------------------------------------------------------

namespace {

// Rows a neighbour of band i reads from it: ctx rows of the neighbour's own
// geometry (the same r for every band of one layer).
int32_t neighbour_rows(const Geo& r) { return r.up > r.dn ? r.up : r.dn; }

bool ranges_overlap(const void* a, int64_t na, const void* b, int64_t nb) {
    if (!a || !b || na <= 0 || nb <= 0) return false;
    const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
    return x < y + (uintptr_t)nb && y < x + (uintptr_t)na;
}

}  // namespace

PCPP_EXPORT size_t pcpp_boundary_bytes(const pcpp_geom_t* g) {
    Geo r;
    if (validate_geom(g, &r) != PCPP_OK) return 0;
    if (g->dtype != PCPP_DTYPE_BF16 && g->dtype != PCPP_DTYPE_F32) return 0;
    return (size_t)g->batch * 2 * (size_t)neighbour_rows(r) * g->W * r.C * r.esize;
}

PCPP_EXPORT int pcpp_pack_boundary(const pcpp_geom_t* g, const void* k_fresh, const void* v_fresh,
                                   void* send_up, void* send_dn, void* stream) {
    Geo r;
    int st = validate_geom(g, &r);
    if (st != PCPP_OK) return st;
    if (g->dtype != PCPP_DTYPE_BF16 && g->dtype != PCPP_DTYPE_F32) return PCPP_ENOTSUP;
    if (g->batch > 65535) return PCPP_EINVAL;
    const bool to_up = r.up > 0, to_dn = r.dn > 0;  // band i-1 / i+1 exists and reads rows
    if (!to_up && !to_dn) return PCPP_OK;
    if (!k_fresh || !v_fresh) return PCPP_EINVAL;
    if ((to_up && !send_up) || (to_dn && !send_dn)) return PCPP_EINVAL;
    const int64_t row = (int64_t)g->W * r.C * r.esize;  // bytes of one token row
    const int64_t band = row * r.h;
    const int64_t run = row * neighbour_rows(r);
    const int64_t msg = 2 * run * g->batch;
    const int64_t fresh_all = band * g->batch;
    for (const void* out : {(const void*)(to_up ? send_up : nullptr), (const void*)(to_dn ? send_dn : nullptr)})
        if (ranges_overlap(out, msg, k_fresh, fresh_all) || ranges_overlap(out, msg, v_fresh, fresh_all))
            return PCPP_EINVAL;
    if (to_up && to_dn && ranges_overlap(send_up, msg, send_dn, msg)) return PCPP_EINVAL;
    CopyParams p;
    p.n_seg = 0;
    p.batch = g->batch;
    auto add = [&](const void* src, int64_t src_off, void* dst, int64_t dst_off) {
        CopySeg& s = p.seg[p.n_seg++];
        s.src = (const char*)src + src_off;
        s.dst = (char*)dst + dst_off;
        s.src_bstride = band;
        s.dst_bstride = 2 * run;
        s.bytes = run;
    };
    if (to_up) {  // the band above reads this band's first r rows
        add(k_fresh, 0, send_up, 0);
        add(v_fresh, 0, send_up, run);
    }
    if (to_dn) {  // the band below reads this band's last r rows
        add(k_fresh, band - run, send_dn, 0);
        add(v_fresh, band - run, send_dn, run);
    }
    return launch_seg_copy(p, r.esize, (hipStream_t)stream) == hipSuccess ? PCPP_OK : PCPP_EHIP;
}

PCPP_EXPORT int pcpp_unpack_boundary(const pcpp_geom_t* g, const void* recv_up, const void* recv_dn,
                                     void* k_up, void* v_up, void* k_dn, void* v_dn, void* stream) {
    Geo r;
    int st = validate_geom(g, &r);
    if (st != PCPP_OK) return st;
    if (g->dtype != PCPP_DTYPE_BF16 && g->dtype != PCPP_DTYPE_F32) return PCPP_ENOTSUP;
    if (g->batch > 65535) return PCPP_EINVAL;
    const bool from_up = r.up > 0, from_dn = r.dn > 0;
    if ((from_up && (!recv_up || !k_up || !v_up)) || (from_dn && (!recv_dn || !k_dn || !v_dn)))
        return PCPP_EINVAL;
    if (!from_up && !from_dn) return PCPP_OK;
    const int64_t row = (int64_t)g->W * r.C * r.esize;
    const int64_t band = row * r.h;
    const int64_t run = row * neighbour_rows(r);
    const int64_t msg = 2 * run * g->batch;
    const int64_t stale_all = band * g->batch;
    const void* recvs[2] = {from_up ? recv_up : nullptr, from_dn ? recv_dn : nullptr};
    void* outs[4] = {from_up ? k_up : nullptr, from_up ? v_up : nullptr, from_dn ? k_dn : nullptr,
                     from_dn ? v_dn : nullptr};
    for (int a = 0; a < 4; ++a) {
        for (const void* in : recvs)
            if (ranges_overlap(outs[a], stale_all, in, msg)) return PCPP_EINVAL;
        for (int c = a + 1; c < 4; ++c)
            if (ranges_overlap(outs[a], stale_all, outs[c], stale_all)) return PCPP_EINVAL;
    }
    CopyParams p;
    p.n_seg = 0;
    p.batch = g->batch;
    auto add = [&](const void* src, int64_t src_off, void* dst, int64_t dst_off) {
        CopySeg& s = p.seg[p.n_seg++];
        s.src = (const char*)src + src_off;
        s.dst = (char*)dst + dst_off;
        s.src_bstride = 2 * run;
        s.dst_bstride = band;
        s.bytes = run;
    };
    if (from_up) {  // the band above sent its last r rows: they close the stale buffer
        add(recv_up, 0, k_up, band - run);
        add(recv_up, run, v_up, band - run);
    }
    if (from_dn) {  // the band below sent its first r rows: they open the stale buffer
        add(recv_dn, 0, k_dn, 0);
        add(recv_dn, run, v_dn, 0);
    }
    return launch_seg_copy(p, r.esize, (hipStream_t)stream) == hipSuccess ? PCPP_OK : PCPP_EHIP;
}

// ---------------------------------------------------------------------------
// Multi-hop messages (p > 1, the context beyond the neighbours of Sec. 6)
// ---------------------------------------------------------------------------

namespace {

// Rows bands i and j exchange, the same in both directions: band j's
// context (r rows past its edge) reaches r - (|i-j|-1)*h rows into band i,
// at most the whole band.  The clip of the context to the image never cuts
// these rows, they lie inside it.
int64_t hop_rows(const pcpp_geom_t* g, const Geo& r, int32_t peer) {
    const int64_t d = peer > g->patch_idx ? peer - g->patch_idx : g->patch_idx - peer;
    if (d == 0) return 0;
    const int64_t ctx = (int64_t)floor(g->partial * (double)r.h + 1e-9);
    const int64_t rows = ctx - (d - 1) * r.h;
    return rows < 0 ? 0 : (rows > r.h ? r.h : rows);
}

int validate_peer(const pcpp_geom_t* g, int32_t peer, Geo* r) {
    int st = validate_geom_hops(g, true, r);
    if (st != PCPP_OK) return st;
    if (peer < 0 || peer >= g->n_patches) return PCPP_EINVAL;
    if (g->dtype != PCPP_DTYPE_BF16 && g->dtype != PCPP_DTYPE_F32) return PCPP_ENOTSUP;
    if (g->batch > 65535) return PCPP_EINVAL;
    return PCPP_OK;
}

}  // namespace

PCPP_EXPORT size_t pcpp_multihop_message_bytes(const pcpp_geom_t* g, int32_t peer) {
    Geo r;
    if (validate_peer(g, peer, &r) != PCPP_OK) return 0;
    return (size_t)g->batch * 2 * (size_t)hop_rows(g, r, peer) * g->W * r.C * r.esize;
}

PCPP_EXPORT int pcpp_pack_multihop(const pcpp_geom_t* g, int32_t peer, const void* k_fresh,
                                   const void* v_fresh, void* send, void* stream) {
    Geo r;
    int st = validate_peer(g, peer, &r);
    if (st != PCPP_OK) return st;
    const int64_t rows = hop_rows(g, r, peer);
    if (rows == 0) return PCPP_OK;
    if (!k_fresh || !v_fresh || !send) return PCPP_EINVAL;
    const int64_t row = (int64_t)g->W * r.C * r.esize;
    const int64_t band = row * r.h;
    const int64_t run = row * rows;
    const int64_t msg = 2 * run * g->batch;
    if (ranges_overlap(send, msg, k_fresh, band * g->batch) || ranges_overlap(send, msg, v_fresh, band * g->batch))
        return PCPP_EINVAL;
    // a band above reads this band's first rows, a band below its last rows
    const int64_t src_off = peer < g->patch_idx ? 0 : band - run;
    CopyParams p;
    p.n_seg = 2;
    p.batch = g->batch;
    for (int s = 0; s < 2; ++s) {
        p.seg[s].src = (const char*)(s == 0 ? k_fresh : v_fresh) + src_off;
        p.seg[s].dst = (char*)send + s * run;
        p.seg[s].src_bstride = band;
        p.seg[s].dst_bstride = 2 * run;
        p.seg[s].bytes = run;
    }
    return launch_seg_copy(p, r.esize, (hipStream_t)stream) == hipSuccess ? PCPP_OK : PCPP_EHIP;
}

PCPP_EXPORT int pcpp_unpack_multihop(const pcpp_geom_t* g, int32_t peer, const void* recv, void* k_above,
                                     void* v_above, void* k_below, void* v_below, void* stream) {
    Geo r;
    int st = validate_peer(g, peer, &r);
    if (st != PCPP_OK) return st;
    const int64_t rows = hop_rows(g, r, peer);
    if (rows == 0) return PCPP_OK;
    const bool above = peer < g->patch_idx;
    void* kd = above ? k_above : k_below;
    void* vd = above ? v_above : v_below;
    if (!recv || !kd || !vd) return PCPP_EINVAL;
    const int64_t row = (int64_t)g->W * r.C * r.esize;
    const int64_t run = row * rows;
    const int64_t block = row * (above ? r.up : r.dn);  // one image of the compact stale block
    const int64_t msg = 2 * run * g->batch;
    if (ranges_overlap(kd, block * g->batch, vd, block * g->batch) ||
        ranges_overlap(recv, msg, kd, block * g->batch) || ranges_overlap(recv, msg, vd, block * g->batch))
        return PCPP_EINVAL;
    // The block above holds image rows i*h-up .. i*h-1 and receives the last
    // rows of band j; the block below holds (i+1)*h .. (i+1)*h+dn-1 and
    // receives the first rows of band j.
    const int64_t i = g->patch_idx, j = peer, h = r.h;
    const int64_t dst_row = above ? (j + 1) * h - rows - (i * h - r.up) : (j - i - 1) * h;
    CopyParams p;
    p.n_seg = 2;
    p.batch = g->batch;
    for (int s = 0; s < 2; ++s) {
        p.seg[s].src = (const char*)recv + s * run;
        p.seg[s].dst = (char*)(s == 0 ? kd : vd) + dst_row * row;
        p.seg[s].src_bstride = 2 * run;
        p.seg[s].dst_bstride = block;
        p.seg[s].bytes = run;
    }
    return launch_seg_copy(p, r.esize, (hipStream_t)stream) == hipSuccess ? PCPP_OK : PCPP_EHIP;
}
