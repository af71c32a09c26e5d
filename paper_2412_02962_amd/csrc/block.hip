// pcpp_transformer_block / pcpp_transformer_module: SDXL's transformer
// module (depth 1: the block) on one band,
// built from the library's kernels (GroupNorm, LayerNorm, MFMA GEMMs with
// fused epilogues, and the attention kernel used twice: partially
// conditioned self-attention over the band plus its neighbours' stale
// boundary rows, Sec. 3.3 of arXiv 2412.02962, and cross-attention to the
// text features).
//
// Data flow (per call, all images of the batch stacked as GEMM rows):
//   t   = GroupNorm(x)                         bf16
//   h   = t Wpi^T + b                          fp32 residual stream
//   n   = LayerNorm(h)                         bf16
//   q,k,v = n Wqkv^T                           bf16 (k, v also exported)
//   a   = PartialAttention(q, k, v, stale)     bf16
//   h  += a Wo^T + b                           fp32 (epilogue residual)
//   n   = LayerNorm(h);  q2 = n Wq2^T;  k2,v2 = text Wkv^T
//   a   = Attention(q2, k2, v2);  h += a Wo2^T + b
//   n   = LayerNorm(h);  u = GEGLU(n Wff1^T + b)   (epilogue value*GELU(gate))
//   h  += u Wff2^T + b
//   y   = h Wpo^T + b + x                      bf16 (h rounded to bf16 by FF-out)

#include <stdint.h>

#include "../../include/pcpp.h"
#include "api_internal.h"
#include "gemm.h"
#include "kernels.h"

#define PCPP_EXPORT extern "C" __attribute__((visibility("default")))

namespace pcpp {

namespace {

struct BlockLayout {
    size_t t16, hid, q16, k16, v16, a16, kv2, u16, attn_ws, gn, split, total;
    size_t attn_ws_bytes, split_bytes;
    int kv_slots;  // basic blocks whose text K/V one launch computes
    bool kv_grouped;
};

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

int validate_block(const pcpp_geom_t* g, int32_t ff_inner, int32_t gn_groups, int32_t n_text, int32_t text_dim,
                   Geo* r) {
    int st = validate_geom(g, r);
    if (st != PCPP_OK) return st;
    if (g->dtype != PCPP_DTYPE_BF16 || g->head_dim != 64) return PCPP_ENOTSUP;
    if (n_text < 1 || text_dim < 32 || text_dim % 32 != 0) return PCPP_EINVAL;
    if (ff_inner < 64 || ff_inner % 64 != 0) return PCPP_EINVAL;
    if (gn_groups < 1 || r->C % gn_groups != 0) return PCPP_EINVAL;
    if (!norm_shapes_ok(r->C, gn_groups)) return PCPP_ENOTSUP;  // LayerNorm keeps a row in registers
    if (g->heads > 65535 || g->batch > 65535) return PCPP_EINVAL;
    return PCPP_OK;
}

AttnParams self_attn_params(const pcpp_geom_t* g, const Geo& r, const void* q, void* out, const void* k,
                            const void* v, const void* k_up, const void* v_up, const void* k_dn, const void* v_dn,
                            void*) {
    return make_attn_params(g, r, q, out, make_kv_source(g, r, k, v, k_up, v_up, k_dn, v_dn));
}

// Cross-attention: one key segment of n_text tokens per image.
AttnParams cross_attn_params(const pcpp_geom_t* g, const Geo& r, const void* q, void* out, const void* k2,
                             const void* v2, int32_t n_text) {
    KvSource kv;
    kv.k[0] = kv.k[2] = nullptr;
    kv.v[0] = kv.v[2] = nullptr;
    kv.k[1] = k2;
    kv.v[1] = v2;
    kv.bstride[0] = kv.bstride[1] = kv.bstride[2] = (int64_t)n_text * r.C;
    kv.end0 = 0;
    kv.end1 = n_text;
    kv.n_kv = n_text;
    return make_attn_params(g, r, q, out, kv);
}

// The text K/V of up to GEMM_MAX_WSEG basic blocks come from one grouped
// product (text_dim % 64 == 0; else one product per block into one slot).
BlockLayout layout(const pcpp_geom_t* g, const Geo& r, int32_t ff_inner, int32_t gn_groups, int32_t n_text,
                   int32_t text_dim, int32_t depth) {
    BlockLayout L;
    const size_t rows = (size_t)g->batch * r.nq;
    const size_t C = r.C;
    const size_t ps = attention_bf16_ws_bytes(self_attn_params(g, r, nullptr, nullptr, nullptr, nullptr,
                                                                 nullptr, nullptr, nullptr, nullptr, nullptr));
    const size_t pc = attention_bf16_ws_bytes(cross_attn_params(g, r, nullptr, nullptr, nullptr, nullptr, n_text));
    L.attn_ws_bytes = ps > pc ? ps : pc;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        size_t o = off;
        off += align256(bytes);
        return o;
    };
    L.t16 = take(rows * C * 2);
    L.hid = take(rows * C * 4);
    L.q16 = take(rows * C * 2);
    L.k16 = take(rows * C * 2);
    L.v16 = take(rows * C * 2);
    L.a16 = take(rows * C * 2);
    L.kv_grouped = text_dim % 64 == 0;
    L.kv_slots = L.kv_grouped ? (depth < GEMM_MAX_WSEG ? depth : GEMM_MAX_WSEG) : 1;
    L.kv2 = take((size_t)L.kv_slots * 2 * g->batch * n_text * C * 2);
    L.u16 = take(rows * (size_t)ff_inner * 2);
    L.attn_ws = take(L.attn_ws_bytes);
    L.gn = take(group_norm_ws_bytes(g->batch, gn_groups, r.nq));
    // One split-K region serves every GEMM of the call in turn (stream order):
    // the largest any of them can use.
    const int M = (int)rows, Ci = (int)C;
    const size_t sizes[] = {gemm_split_ws_bytes(M, Ci, Ci, false), gemm_split_ws_bytes(M, 3 * Ci, Ci, false),
                            gemm_split_ws_bytes(M, Ci, ff_inner, false)};
    L.split_bytes = 0;
    for (size_t b : sizes) L.split_bytes = b > L.split_bytes ? b : L.split_bytes;
    for (int nb = 1; nb <= L.kv_slots; ++nb) {  // every chunk size, the last one may be short
        const size_t b = gemm_split_ws_bytes(g->batch * n_text, nb * 2 * Ci, text_dim, false);
        L.split_bytes = b > L.split_bytes ? b : L.split_bytes;
    }
    L.split = L.split_bytes ? take(L.split_bytes) : 0;
    L.total = off;
    return L;
}

GemmParams gemm(const void* a, int64_t lda, bool a_f32, const void* wt, const void* bias, int M, int N, int K,
                void* out, int64_t ldo, bool out_f32) {
    GemmParams p;
    p.a = a;
    p.lda = lda;
    p.a_f32 = a_f32 ? 1 : 0;
    p.w = (const __bf16*)wt;
    p.bias = (const __bf16*)bias;
    p.M = M;
    p.N = N;
    p.K = K;
    p.geglu = 0;
    p.F = 0;
    p.resid = nullptr;
    p.ldr = 0;
    p.resid_f32 = 0;
    p.out[0] = out;
    p.out[1] = p.out[2] = nullptr;
    p.seg = N;
    p.ldo = ldo;
    p.out_f32 = out_f32 ? 1 : 0;
    p.out_bf16 = nullptr;
    return p;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

}  // namespace

}  // namespace pcpp

using namespace pcpp;

namespace {

// The module's own weights (GroupNorm, proj_in, proj_out) and sizes.
struct ModuleW {
    const void *gn_gamma, *gn_beta, *proj_in_w, *proj_in_b, *proj_out_w, *proj_out_b;
    int32_t ff_inner, gn_groups;
};

ModuleW module_of(const pcpp_block_weights_t* w) {
    return ModuleW{w->gn_gamma, w->gn_beta, w->proj_in_w, w->proj_in_b, w->proj_out_w, w->proj_out_b, w->ff_inner,
                   w->gn_groups};
}

pcpp_basic_block_weights_t basic_of(const pcpp_block_weights_t* w) {
    pcpp_basic_block_weights_t b;
    b.ln1_gamma = w->ln1_gamma;
    b.ln1_beta = w->ln1_beta;
    b.attn1_qkv_w = w->attn1_qkv_w;
    b.attn1_out_w = w->attn1_out_w;
    b.attn1_out_b = w->attn1_out_b;
    b.ln2_gamma = w->ln2_gamma;
    b.ln2_beta = w->ln2_beta;
    b.attn2_q_w = w->attn2_q_w;
    b.attn2_kv_w = w->attn2_kv_w;
    b.attn2_out_w = w->attn2_out_w;
    b.attn2_out_b = w->attn2_out_b;
    b.ln3_gamma = w->ln3_gamma;
    b.ln3_beta = w->ln3_beta;
    b.ff1_w = w->ff1_w;
    b.ff1_b = w->ff1_b;
    b.ff2_w = w->ff2_w;
    b.ff2_b = w->ff2_b;
    return b;
}

// GroupNorm -> proj_in -> depth basic blocks -> proj_out + x.  Basic block j
// reads the stale neighbour K/V k_up[j] .. v_dn[j] and exports its own K/V
// to k_out[j] / v_out[j] (either array, or an entry, may be null: then the
// workspace holds them).
int run_module(const pcpp_geom_t* g, const ModuleW& mw, const pcpp_basic_block_weights_t* blocks, int depth,
               const void* x, const void* text, int32_t n_text, int32_t text_dim, const void* const* k_up,
               const void* const* v_up, const void* const* k_dn, const void* const* v_dn, const float* gn_bands,
               float* gn_own, void* y, void* const* k_out, void* const* v_out, void* workspace, size_t ws_bytes,
               void* stream) {
    Geo r;
    int st = validate_block(g, mw.ff_inner, mw.gn_groups, n_text, text_dim, &r);
    if (st != PCPP_OK) return st;
    if (depth < 1 || depth > 64 || blocks == nullptr) return PCPP_EINVAL;
    const void* mptrs[] = {mw.gn_gamma, mw.gn_beta, mw.proj_in_w, mw.proj_in_b, mw.proj_out_w, mw.proj_out_b};
    for (const void* p : mptrs)
        if (p == nullptr || !aligned16(p)) return PCPP_EINVAL;
    if (!x || !text || !y || !aligned16(x) || !aligned16(text) || !aligned16(y)) return PCPP_EINVAL;
    if ((r.up > 0 && (!k_up || !v_up)) || (r.dn > 0 && (!k_dn || !v_dn))) return PCPP_EINVAL;
    for (int j = 0; j < depth; ++j) {
        const pcpp_basic_block_weights_t& w = blocks[j];
        const void* wptrs[] = {w.ln1_gamma, w.ln1_beta, w.attn1_qkv_w, w.attn1_out_w, w.attn1_out_b, w.ln2_gamma,
                               w.ln2_beta, w.attn2_q_w, w.attn2_kv_w, w.attn2_out_w, w.attn2_out_b, w.ln3_gamma,
                               w.ln3_beta, w.ff1_w, w.ff1_b, w.ff2_w, w.ff2_b};
        for (const void* p : wptrs)
            if (p == nullptr || !aligned16(p)) return PCPP_EINVAL;
        if (r.up > 0 && (!k_up[j] || !v_up[j] || !aligned16(k_up[j]) || !aligned16(v_up[j]))) return PCPP_EINVAL;
        if (r.dn > 0 && (!k_dn[j] || !v_dn[j] || !aligned16(k_dn[j]) || !aligned16(v_dn[j]))) return PCPP_EINVAL;
        if (k_out && k_out[j] && !aligned16(k_out[j])) return PCPP_EINVAL;
        if (v_out && v_out[j] && !aligned16(v_out[j])) return PCPP_EINVAL;
    }
    const BlockLayout L = layout(g, r, mw.ff_inner, mw.gn_groups, n_text, text_dim, depth);
    if (workspace == nullptr || ws_bytes < L.total) return PCPP_EWORKSPACE;
    if (!aligned16(workspace)) return PCPP_EINVAL;

    hipStream_t s = (hipStream_t)stream;
    char* ws = (char*)workspace;
    const int B = g->batch, N = r.nq, C = r.C, F = mw.ff_inner, T = n_text;
    const int rows = B * N;
    __bf16* t16 = (__bf16*)(ws + L.t16);
    float* hid = (float*)(ws + L.hid);
    __bf16* q16 = (__bf16*)(ws + L.q16);
    __bf16* a16 = (__bf16*)(ws + L.a16);
    __bf16* kv2 = (__bf16*)(ws + L.kv2);
    const int64_t kv_elems = (int64_t)B * T * C;  // one K or V of the text
    __bf16* u16 = (__bf16*)(ws + L.u16);
    void* attn_ws = ws + L.attn_ws;
    void* split_ws = L.split_bytes ? ws + L.split : nullptr;
    // Every plain GEMM may split K over the shared region, and the attention
    // launches merge key pieces through theirs: the GroupNorm statistics
    // launch below clears both sets of counters, so the workspace needs no
    // clearing between calls.
    auto gemm_s = [&](GemmParams mm) {
        mm.split_ws = split_ws;
        mm.split_ws_bytes = L.split_bytes;
        return launch_gemm(mm, s);
    };
    auto gemm_pair_s = [&](GemmParams a, GemmParams b) {
        a.split_ws = b.split_ws = split_ws;
        a.split_ws_bytes = b.split_ws_bytes = L.split_bytes;
        return launch_gemm_pair(a, b, s);
    };
    // Text K/V of blocks j.. (the rest of its chunk of kv_slots blocks): one
    // product over their stacked weights, block u's K at slot 2u, V at 2u + 1.
    auto text_kv = [&](int j) {
        const int nb = depth - j < L.kv_slots ? depth - j : L.kv_slots;
        GemmParams kv = gemm(text, text_dim, false, blocks[j].attn2_kv_w, nullptr, B * T, nb * 2 * C, text_dim, kv2, C,
                             false);
        kv.seg = C;
        kv.seg_stride = kv_elems;
        kv.w_seg_rows = 2 * C;
        for (int u = 0; u < nb; ++u) kv.w_seg[u] = (const __bf16*)blocks[j + u].attn2_kv_w;
        return kv;
    };
    hipError_t e = hipSuccess;
#define PCPP_CHECK(call)                  \
    do {                                  \
        e = (call);                       \
        if (e != hipSuccess) return PCPP_EHIP; \
    } while (0)

    // GroupNorm over the band's tokens, then proj_in into the fp32 stream.
    GroupNormParams gp;
    gp.x = (const __bf16*)x;
    gp.y = t16;
    gp.gamma = (const __bf16*)mw.gn_gamma;
    gp.beta = (const __bf16*)mw.gn_beta;
    gp.stats = (float*)(ws + L.gn);
    gp.B = B;
    gp.N = N;
    gp.C = C;
    gp.G = mw.gn_groups;
    gp.eps = 1e-6f;
    gp.bands = gn_bands;
    gp.n_bands = g->n_patches;
    gp.band = g->patch_idx;
    gp.own_out = gn_own;
    gp.zero = (int*)split_ws;
    gp.n_zero = split_ws ? GEMM_SPLIT_COUNTERS : 0;
    // The attention launches' work counters too: the workspace may hold
    // anything on entry (a caller may share it with calls that use it as
    // plain scratch), and every launch below leaves its counters at zero.
    {
        const DeviceLayout dl = device_layout(s);
        const AttnParams sa = self_attn_params(g, r, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                                               nullptr, nullptr);
        const AttnParams ca = cross_attn_params(g, r, nullptr, nullptr, nullptr, nullptr, n_text);
        const int n1 = attention_bf16_plan(sa, dl).counters, n2 = attention_bf16_plan(ca, dl).counters;
        gp.zero2 = (int*)attn_ws;
        gp.n_zero2 = n1 > n2 ? n1 : n2;
    }
    // proj_in, and beside it in the same launch the first chunk's text K/V
    // (independent of the band).  When the band's tokens fill whole 64-token
    // tiles, proj_in applies the GroupNorm itself while staging x (from the
    // statistics launch's records), else a separate apply writes it to t16.
    {
        const bool gn_in_gemm = N % 64 == 0 && C % 64 == 0 && C <= GEMM_GN_MAXC;
        GemmParams pin = gemm(t16, C, false, mw.proj_in_w, mw.proj_in_b, rows, C, C, hid, C, true);
        if (gn_in_gemm) {
            PCPP_CHECK(launch_group_norm_stats(gp, s));
            pin.a = x;
            pin.a_mode = 1;
            pin.gn.stats = gp.stats;
            pin.gn.chunks = gp.chunks;
            pin.gn.G = gp.G;
            pin.gn.B = gp.B;
            pin.gn.eps = gp.eps;
            pin.gn.bands = gp.bands;
            pin.gn.n_bands = gp.n_bands;
            pin.gn.band = gp.band;
            pin.gn.own_out = gp.own_out;
            pin.gn_gamma = gp.gamma;
            pin.gn_beta = gp.beta;
            pin.gn_N = N;
        } else {
            PCPP_CHECK(launch_group_norm(gp, s));
        }
        PCPP_CHECK(L.kv_grouped && depth > 0 ? gemm_pair_s(pin, text_kv(0)) : gemm_s(pin));
    }

    LayerNormParams lp;
    lp.x = hid;
    lp.y = t16;
    lp.rows = rows;
    lp.C = C;
    lp.eps = 1e-5f;
    // The last FF-out also writes the stream rounded to bf16 (into t16, free
    // by then), the operand proj_out reads.
    const bool copy16 = C % 64 == 0 && F % 64 == 0;

    for (int j = 0; j < depth; ++j) {
        const pcpp_basic_block_weights_t& w = blocks[j];
        __bf16* k16 = k_out && k_out[j] ? (__bf16*)k_out[j] : (__bf16*)(ws + L.k16);
        __bf16* v16 = v_out && v_out[j] ? (__bf16*)v_out[j] : (__bf16*)(ws + L.v16);
        const void* ku = r.up > 0 ? k_up[j] : nullptr;
        const void* vu = r.up > 0 ? v_up[j] : nullptr;
        const void* kd = r.dn > 0 ? k_dn[j] : nullptr;
        const void* vd = r.dn > 0 ? v_dn[j] : nullptr;

        // Text K/V of this block's chunk (the first chunk's came with proj_in).
        const int slot = j % L.kv_slots;
        if (L.kv_grouped && slot == 0 && j > 0) PCPP_CHECK(gemm_s(text_kv(j)));
        __bf16* k2 = kv2 + 2 * slot * kv_elems;
        __bf16* v2 = k2 + kv_elems;

        // Self-attention: Q, K, V of the band; K and V are the band's export.
        lp.gamma = (const __bf16*)w.ln1_gamma;
        lp.beta = (const __bf16*)w.ln1_beta;
        PCPP_CHECK(launch_layer_norm(lp, s));
        {
            GemmParams qkv = gemm(t16, C, false, w.attn1_qkv_w, nullptr, rows, 3 * C, C, q16, C, false);
            qkv.out[1] = k16;
            qkv.out[2] = v16;
            qkv.seg = C;
            PCPP_CHECK(gemm_s(qkv));
        }
        {
            AttnParams ap = self_attn_params(g, r, q16, a16, k16, v16, ku, vu, kd, vd, nullptr);
            PCPP_CHECK(launch_attention_bf16(ap, attn_ws, L.attn_ws_bytes, s));
        }
        {
            GemmParams o = gemm(a16, C, false, w.attn1_out_w, w.attn1_out_b, rows, C, C, hid, C, true);
            o.resid = hid;
            o.ldr = C;
            o.resid_f32 = 1;
            PCPP_CHECK(gemm_s(o));
        }

        // Cross-attention to the text features.
        lp.gamma = (const __bf16*)w.ln2_gamma;
        lp.beta = (const __bf16*)w.ln2_beta;
        PCPP_CHECK(launch_layer_norm(lp, s));
        if (!L.kv_grouped) {
            GemmParams kv = gemm(text, text_dim, false, w.attn2_kv_w, nullptr, B * T, 2 * C, text_dim, k2, C, false);
            kv.out[1] = v2;
            kv.seg = C;
            PCPP_CHECK(gemm_s(kv));
        }
        // Q of the cross-attention; with at most GEMM_XA_MAXT text tokens and
        // whole 64-token tiles, the Q product's workgroups go on to the
        // attention itself (one head per tile), else it runs separately.
        if (T <= GEMM_XA_MAXT && N % 64 == 0) {
            GemmParams xq = gemm(t16, C, false, w.attn2_q_w, nullptr, rows, C, C, a16, C, false);
            xq.a_mode = 2;
            xq.xa_k = k2;
            xq.xa_v = v2;
            xq.xa_T = T;
            xq.xa_N = N;
            xq.xa_ldkv = C;
            PCPP_CHECK(gemm_s(xq));
        } else {
            PCPP_CHECK(gemm_s(gemm(t16, C, false, w.attn2_q_w, nullptr, rows, C, C, q16, C, false)));
            AttnParams ap = cross_attn_params(g, r, q16, a16, k2, v2, T);
            PCPP_CHECK(launch_attention_bf16(ap, attn_ws, L.attn_ws_bytes, s));
        }
        {
            GemmParams o = gemm(a16, C, false, w.attn2_out_w, w.attn2_out_b, rows, C, C, hid, C, true);
            o.resid = hid;
            o.ldr = C;
            o.resid_f32 = 1;
            PCPP_CHECK(gemm_s(o));
        }

        // GEGLU feed-forward.
        lp.gamma = (const __bf16*)w.ln3_gamma;
        lp.beta = (const __bf16*)w.ln3_beta;
        PCPP_CHECK(launch_layer_norm(lp, s));
        {
            GemmParams ff = gemm(t16, C, false, w.ff1_w, w.ff1_b, rows, F, C, u16, F, false);
            ff.geglu = 1;
            ff.F = F;
            PCPP_CHECK(gemm_s(ff));
        }
        {
            GemmParams o = gemm(u16, F, false, w.ff2_w, w.ff2_b, rows, C, F, hid, C, true);
            o.resid = hid;
            o.ldr = C;
            o.resid_f32 = 1;
            if (copy16 && j == depth - 1) o.out_bf16 = t16;
            PCPP_CHECK(gemm_s(o));
        }
    }

    // proj_out plus the module input.
    {
        GemmParams o = copy16 ? gemm(t16, C, false, mw.proj_out_w, mw.proj_out_b, rows, C, C, y, C, false)
                              : gemm(hid, C, true, mw.proj_out_w, mw.proj_out_b, rows, C, C, y, C, false);
        o.resid = x;
        o.ldr = C;
        o.resid_f32 = 0;
        PCPP_CHECK(gemm_s(o));
    }
#undef PCPP_CHECK
    return PCPP_OK;
}

int run_block(const pcpp_geom_t* g, const pcpp_block_weights_t* w, const void* x, const void* text,
              int32_t n_text, int32_t text_dim, const void* k_up, const void* v_up, const void* k_dn,
              const void* v_dn, const float* gn_bands, float* gn_own, void* y, void* k_fresh_out,
              void* v_fresh_out, void* workspace, size_t ws_bytes, void* stream) {
    if (w == nullptr) return PCPP_EINVAL;
    const pcpp_basic_block_weights_t b = basic_of(w);
    const void* ku[1] = {k_up};
    const void* vu[1] = {v_up};
    const void* kd[1] = {k_dn};
    const void* vd[1] = {v_dn};
    void* ko[1] = {k_fresh_out};
    void* vo[1] = {v_fresh_out};
    return run_module(g, module_of(w), &b, 1, x, text, n_text, text_dim, ku, vu, kd, vd, gn_bands, gn_own, y, ko, vo,
                      workspace, ws_bytes, stream);
}

}  // namespace

PCPP_EXPORT size_t pcpp_transformer_block_workspace_size(const pcpp_geom_t* g, const pcpp_block_weights_t* w,
                                                         int32_t n_text, int32_t text_dim) {
    Geo r;
    if (w == nullptr || validate_block(g, w->ff_inner, w->gn_groups, n_text, text_dim, &r) != PCPP_OK) return 0;
    return layout(g, r, w->ff_inner, w->gn_groups, n_text, text_dim, 1).total;
}

PCPP_EXPORT int pcpp_transformer_block(const pcpp_geom_t* g, const pcpp_block_weights_t* w, const void* x,
                                       const void* text, int32_t n_text, int32_t text_dim, const void* k_up,
                                       const void* v_up, const void* k_dn, const void* v_dn, void* y,
                                       void* k_fresh_out, void* v_fresh_out, void* workspace, size_t ws_bytes,
                                       void* stream) {
    return run_block(g, w, x, text, n_text, text_dim, k_up, v_up, k_dn, v_dn, nullptr, nullptr, y, k_fresh_out,
                     v_fresh_out, workspace, ws_bytes, stream);
}

PCPP_EXPORT int pcpp_transformer_block_sync_gn(const pcpp_geom_t* g, const pcpp_block_weights_t* w, const void* x,
                                               const void* text, int32_t n_text, int32_t text_dim,
                                               const void* k_up, const void* v_up, const void* k_dn,
                                               const void* v_dn, const float* gn_bands, float* gn_own, void* y,
                                               void* k_fresh_out, void* v_fresh_out, void* workspace,
                                               size_t ws_bytes, void* stream) {
    if (gn_bands != nullptr && ((uintptr_t)gn_bands & 3u) != 0) return PCPP_EINVAL;
    if (gn_own != nullptr && ((uintptr_t)gn_own & 3u) != 0) return PCPP_EINVAL;
    return run_block(g, w, x, text, n_text, text_dim, k_up, v_up, k_dn, v_dn, gn_bands, gn_own, y, k_fresh_out,
                     v_fresh_out, workspace, ws_bytes, stream);
}

PCPP_EXPORT size_t pcpp_transformer_module_workspace_size(const pcpp_geom_t* g, const pcpp_module_weights_t* w,
                                                          int32_t n_text, int32_t text_dim) {
    Geo r;
    if (w == nullptr || validate_block(g, w->ff_inner, w->gn_groups, n_text, text_dim, &r) != PCPP_OK) return 0;
    if (w->depth < 1 || w->depth > 64) return 0;
    return layout(g, r, w->ff_inner, w->gn_groups, n_text, text_dim, w->depth).total;
}

PCPP_EXPORT int pcpp_transformer_module(const pcpp_geom_t* g, const pcpp_module_weights_t* w, const void* x,
                                        const void* text, int32_t n_text, int32_t text_dim,
                                        const void* const* k_up, const void* const* v_up, const void* const* k_dn,
                                        const void* const* v_dn, const float* gn_bands, float* gn_own, void* y,
                                        void* const* k_fresh_out, void* const* v_fresh_out, void* workspace,
                                        size_t ws_bytes, void* stream) {
    if (w == nullptr) return PCPP_EINVAL;
    if (gn_bands != nullptr && ((uintptr_t)gn_bands & 3u) != 0) return PCPP_EINVAL;
    if (gn_own != nullptr && ((uintptr_t)gn_own & 3u) != 0) return PCPP_EINVAL;
    const ModuleW mw{w->gn_gamma, w->gn_beta, w->proj_in_w, w->proj_in_b, w->proj_out_w, w->proj_out_b, w->ff_inner,
                     w->gn_groups};
    return run_module(g, mw, w->blocks, w->depth, x, text, n_text, text_dim, k_up, v_up, k_dn, v_dn, gn_bands, gn_own,
                      y, k_fresh_out, v_fresh_out, workspace, ws_bytes, stream);
}
