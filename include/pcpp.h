/*
 * pcpp.h - C ABI of the PCPP per-patch hot path on AMD Instinct MI355X (gfx950).
 *
 * Partially Conditioned Patch Parallelism (arXiv 2412.02962) splits the
 * H x W latent feature map into n horizontal bands of h = H/n rows (Sec. 3.1)
 * and runs each band on its own device.  In every self-attention layer the
 * band's queries attend to its own fresh keys/values plus the stale keys and
 * values (previous diffusion step) of only the boundary rows of its two
 * neighbours: the lower p*h rows of the band above and the upper p*h rows of
 * the band below (Eq. 1, Sec. 3.3, Fig. 3).  This library computes one
 * device's share of that work for one band; the neighbours' stale tensors are
 * inputs supplied by the caller.
 *
 * Conventions shared by every entry point
 *   - Tensors are row-major and contiguous.  Token tensors are [B, N, C] with
 *     C = heads * head_dim; head a owns channels [a*head_dim, (a+1)*head_dim).
 *     Tokens of a band are ordered row by row (token = row * W + col).
 *   - Tensor pointers are DEVICE pointers owned by the caller.  The library
 *     never frees, retains or writes through an input pointer.  Its only
 *     state between calls is a per-device cache of the device's compute-unit
 *     count (read once, then constant).
 *   - Neighbour buffers hold the WHOLE neighbouring band, [B, h*W, C], as
 *     received from that neighbour; only its boundary rows are read.  A
 *     missing neighbour (top or bottom band) or a zero row count allows NULL.
 *   - `stream` is a hipStream_t passed as void* (NULL = default stream).
 *     Compute entry points are asynchronous: they validate, enqueue kernels
 *     and return.  The caller must not modify inputs, and must not read
 *     outputs, before the stream has passed the call.
 *   - Return value: PCPP_OK (0) or a negative PCPP_E* code.  Every argument
 *     is validated before anything is enqueued; on an error nothing is
 *     launched and no output is touched.  No exception crosses the ABI.
 *   - Element types: PCPP_DTYPE_BF16 (bfloat16 storage, float32
 *     accumulation) or PCPP_DTYPE_F32 (float32 throughout).
 *   - Work split across workgroups.  Some launches (the bf16 attention's key
 *     ranges, the split-K GEMMs inside the block, module, ResNet and
 *     convolution calls) split one tile's work over several workgroups and
 *     merge the pieces through one XCD's L2 cache.  That relies on the gfx950
 *     dispatcher dealing the workgroups of a launch round-robin over the
 *     device's XCDs of 32 compute units (workgroup w on XCD w % n_xcd).  The
 *     library splits only when the device's compute units are whole XCDs and
 *     the stream has no CU mask (hipExtStreamGetCUMask reports every compute
 *     unit); otherwise the same calls run unsplit, with the same results up
 *     to the order of float32 additions.  Do not run these calls on a device
 *     partitioned or masked in any way the CU mask does not show.
 */
#ifndef PCPP_H
#define PCPP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PCPP_VERSION 1

/* Status codes. */
#define PCPP_OK          0
#define PCPP_EINVAL     -1   /* bad geometry, p outside [0,1] or NaN, NULL where data is needed */
#define PCPP_ENOTSUP    -2   /* head_dim or dtype the kernels do not implement */
#define PCPP_EWORKSPACE -3   /* workspace missing or smaller than *_workspace_size() */
#define PCPP_EHIP       -4   /* a HIP runtime call or kernel launch failed */

/* Element types. */
#define PCPP_DTYPE_F32  0
#define PCPP_DTYPE_BF16 1

/*
 * Geometry of one self-attention layer on one band (Sec. 3.1).
 *   H, W       token grid of this layer (H rows, W columns), H % n_patches == 0
 *   n_patches  number of bands n >= 1; n = 1 is full-image attention, the
 *              synchronous warm-up steps of the method (Sec. 3.2)
 *   patch_idx  0-based band index i in [0, n); band 0 is the top band
 *              (the paper numbers bands from 1)
 *   partial    p in [0, 1]: fraction of a neighbour's height used as context;
 *              rows taken r = min(h, floor(p*h + 1e-9))
 *   heads, head_dim  multi-head layout, C = heads * head_dim
 *   batch      B >= 1 independent images (one classifier-free-guidance branch
 *              per image)
 *   step       diffusion step t >= 0; validated and otherwise unused: the
 *              result is a function of the inputs and geometry only
 *   dtype      PCPP_DTYPE_BF16 or PCPP_DTYPE_F32
 */
typedef struct pcpp_geom {
    int32_t H;
    int32_t W;
    int32_t n_patches;
    int32_t patch_idx;
    double  partial;
    int32_t heads;
    int32_t head_dim;
    int32_t batch;
    int32_t step;
    int32_t dtype;
    int32_t reserved;   /* must be 0 */
} pcpp_geom_t;

/* Library version (PCPP_VERSION). */
int pcpp_version(void);

/* Static description of a status code; never NULL. */
const char* pcpp_strerror(int status);

/*
 * Eq. 1 context geometry (host only, no GPU work).
 * Outputs (any may be NULL): h = H/n; up = rows taken from band i-1 (0 for
 * the top band); dn = rows taken from band i+1 (0 for the bottom band);
 * n_kv = (up + h + dn) * W keys per image.
 * Errors: PCPP_EINVAL for NULL g, n < 1, H % n != 0, i outside [0,n),
 * p outside [0,1] or NaN, W < 1, batch < 1, step < 0, or a non-zero
 * reserved field.
 */
int pcpp_context_rows(const pcpp_geom_t* g, int32_t* h, int32_t* up,
                      int32_t* dn, int32_t* n_kv);

/*
 * Key/value context assembly (Eq. 1, Fig. 3).
 *   k_fresh, v_fresh  [B, h*W, C] this band's keys/values of the current step
 *   k_up, v_up        [B, h*W, C] stale band i-1 (its last `up` rows are read)
 *   k_dn, v_dn        [B, h*W, C] stale band i+1 (its first `dn` rows are read)
 *   idx_out           [n_kv] int32, device: global token ids row*W + col of
 *                     the context in ascending order (rows i*h-up ..
 *                     (i+1)*h+dn-1, every column); may be NULL
 *   k_ctx, v_ctx      [B, n_kv, C] device outputs in that token order, or
 *                     both NULL to build the index set only
 * Element type from g->dtype; all tensors share it.  Neighbour pointers may
 * be NULL when the matching row count is 0.  Outputs must not overlap inputs.
 */
int pcpp_gather_context(const pcpp_geom_t* g,
                        const void* k_fresh, const void* v_fresh,
                        const void* k_up, const void* v_up,
                        const void* k_dn, const void* v_dn,
                        int32_t* idx_out, void* k_ctx, void* v_ctx,
                        void* stream);

/*
 * Bytes of device workspace pcpp_partial_attention needs for geometry g on
 * the current device (bf16 path: per-query-block work counters plus float32
 * partial outputs and row statistics of query blocks whose keys are split
 * across workgroups; 0 for the f32 path).  Returns 0 for an invalid g.
 *
 * Workspace contract: the buffer must be zero-filled before its first use
 * (e.g. hipMemset once after allocation).  Every call leaves its counters
 * zero again, and the counters sit at the same offset for every geometry
 * (the float32 partials after them need no clearing), so the same buffer (of
 * the largest size needed) serves any number of later calls of any geometry
 * on that device, graph replays included, without clearing.
 * Calls that share one workspace must be ordered on one stream.
 */
size_t pcpp_partial_attention_workspace_size(const pcpp_geom_t* g);

/*
 * Partially conditioned self-attention of band i (Sec. 3.3, Fig. 3).
 * Per image and head a: S = Q_a K_ctx,a^T / sqrt(head_dim) over the n_kv
 * context keys (stale rows above, fresh band, stale rows below), row
 * softmax, O_a = softmax(S) V_ctx,a.  No mask, no bias.
 *   q                 [B, h*W, C] queries of this band (never exchanged)
 *   k_fresh, v_fresh  [B, h*W, C]
 *   k_up, v_up, k_dn, v_dn  whole stale neighbour bands as above
 *   out               [B, h*W, C], same dtype as the inputs
 *   workspace         device scratch of ws_bytes >= the workspace size
 *                     (may be NULL when that size is 0), zero-filled before
 *                     its first use (see the workspace contract above)
 * Supported: head_dim == 64 for both dtypes.  bf16 runs on the MFMA path
 * (float32 accumulation and softmax, probabilities rounded to bf16 as the
 * operand of the P*V product); f32 runs a float32 path.
 */
int pcpp_partial_attention(const pcpp_geom_t* g, const void* q,
                           const void* k_fresh, const void* v_fresh,
                           const void* k_up, const void* v_up,
                           const void* k_dn, const void* v_dn,
                           void* out, void* workspace, size_t ws_bytes,
                           void* stream);

/*
 * Launch plan of the bf16 partially conditioned attention (host only, no GPU
 * work; for diagnostics and tests).  cus > 0: a device of `cus` compute
 * units of which `cus_enabled` may run the launch (a stream's CU mask);
 * cus == 0: the current device and the CU mask of `stream` (PCPP_EHIP if
 * the device cannot be queried).  Outputs (any may be NULL): queries per
 * block (a block is one workgroup's share of one image and head), pieces
 * per block (key ranges merged through one XCD's L2; 1 = unsplit) and the
 * launch's workgroups.  PCPP_ENOTSUP unless bf16 with head_dim 64.
 */
int pcpp_partial_attention_plan(const pcpp_geom_t* g, int32_t cus, int32_t cus_enabled,
                                void* stream, int32_t* block_queries,
                                int32_t* pieces, int32_t* workgroups);

/*
 * pcpp_partial_attention for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same computation and arguments without the workspace.
 * The library keeps, on each GPU it runs on, one device array of
 * PCPP_NOALLOC_SCRATCH_BYTES for this entry point's workspace, held until
 * the process ends; the first call on a device looks up its address and
 * clears it (a fill kernel on `stream`).  Nothing is allocated by any call.
 *   - Geometries whose workspace (pcpp_partial_attention_workspace_size)
 *     exceeds PCPP_NOALLOC_SCRATCH_BYTES fail with PCPP_EWORKSPACE before
 *     anything is launched; use pcpp_partial_attention with a caller
 *     workspace for them.
 *   - Every call on one GPU shares that GPU's array: calls that overlap on
 *     one GPU (different streams, different host threads) race and must be
 *     ordered by the caller.  Calls in one stream, graph replays included,
 *     are fine: each leaves the array ready for the next.
 * Other arguments, requirements and errors as pcpp_partial_attention.
 */
#define PCPP_NOALLOC_SCRATCH_BYTES (32u * 1024u * 1024u)
int pcpp_partial_attention_noalloc(const pcpp_geom_t* g, const void* q,
                                   const void* k_fresh, const void* v_fresh,
                                   const void* k_up, const void* v_up,
                                   const void* k_dn, const void* v_dn,
                                   void* out, void* stream);

/*
 * Multi-hop partially conditioned attention: p may exceed 1, the context
 * reaching past the immediate neighbours (Sec. 6 hypothesises that many
 * bands need it), up to the whole image at p = n - 1.  The band attends to
 * the up = min(r, i*h) rows directly above it and the dn = min(r, (n-1-i)*h)
 * rows directly below it, r = floor(p*h + 1e-9), stale, plus its own fresh
 * rows; for p <= 1 this is pcpp_partial_attention's context.  The stale rows
 * come compact instead of as whole neighbour bands:
 *   k_above, v_above  [B, up*W, C]: image rows i*h-up .. i*h-1, in order
 *                     (from bands i-1, i-2, ...; NULL when up = 0)
 *   k_below, v_below  [B, dn*W, C]: image rows (i+1)*h .. (i+1)*h+dn-1
 * p must lie in [0, max(1, n-1)] (PCPP_EINVAL otherwise).  Other arguments,
 * the workspace contract and the numerics as pcpp_partial_attention; the
 * workspace size comes from the function below.
 */
size_t pcpp_partial_attention_multihop_workspace_size(const pcpp_geom_t* g);
int pcpp_partial_attention_multihop(const pcpp_geom_t* g, const void* q,
                                    const void* k_fresh, const void* v_fresh,
                                    const void* k_above, const void* v_above,
                                    const void* k_below, const void* v_below,
                                    void* out, void* workspace, size_t ws_bytes,
                                    void* stream);

/*
 * Weights of one SDXL-shaped transformer block (device pointers, bf16,
 * nn.Linear layout [out, in]).  C = heads * head_dim, F = ff_inner,
 * T = text_dim.
 */
typedef struct pcpp_block_weights {
    const void* gn_gamma;      /* [C] GroupNorm scale (eps 1e-6)            */
    const void* gn_beta;       /* [C]                                        */
    const void* proj_in_w;     /* [C, C]                                     */
    const void* proj_in_b;     /* [C]                                        */
    const void* ln1_gamma;     /* [C] LayerNorm before self-attn (eps 1e-5)  */
    const void* ln1_beta;      /* [C]                                        */
    const void* attn1_qkv_w;   /* [3C, C] rows: W_q, then W_k, then W_v       */
    const void* attn1_out_w;   /* [C, C]                                     */
    const void* attn1_out_b;   /* [C]                                        */
    const void* ln2_gamma;     /* [C] LayerNorm before cross-attn            */
    const void* ln2_beta;      /* [C]                                        */
    const void* attn2_q_w;     /* [C, C]                                     */
    const void* attn2_kv_w;    /* [2C, T] rows: W_k, then W_v (text side)    */
    const void* attn2_out_w;   /* [C, C]                                     */
    const void* attn2_out_b;   /* [C]                                        */
    const void* ln3_gamma;     /* [C] LayerNorm before the feed-forward      */
    const void* ln3_beta;      /* [C]                                        */
    const void* ff1_w;         /* [2F, C] rows [0,F) value, [F,2F) gate      */
    const void* ff1_b;         /* [2F]                                       */
    const void* ff2_w;         /* [C, F]                                     */
    const void* ff2_b;         /* [C]                                        */
    const void* proj_out_w;    /* [C, C]                                     */
    const void* proj_out_b;    /* [C]                                        */
    int32_t ff_inner;          /* F >= 1, multiple of 64                     */
    int32_t gn_groups;         /* groups dividing C                          */
} pcpp_block_weights_t;

/* Bytes of device workspace pcpp_transformer_block needs (0 if g invalid).
 * The workspace needs no clearing: each call clears the work counters its
 * launches use before the first of them, so the buffer may hold anything on
 * entry (another call's scratch, say). */
size_t pcpp_transformer_block_workspace_size(const pcpp_geom_t* g,
                                             const pcpp_block_weights_t* w,
                                             int32_t n_text, int32_t text_dim);

/*
 * One SDXL-shaped transformer block on band i, bf16 storage with float32
 * accumulation (the method applies to the self-attention only, Sec. 3.3;
 * GroupNorm here uses the band's own statistics):
 *   t  = GroupNorm(x)                       (gn_groups groups, eps 1e-6)
 *   h  = t proj_in^T + b
 *   n1 = LayerNorm(h);  q,k,v = n1 W_q^T, n1 W_k^T, n1 W_v^T
 *   h += PartialAttention(q, k, v, k_up, v_up, k_dn, v_dn) W_o^T + b
 *   n2 = LayerNorm(h);  h += Attention(n2 W_q2^T, text W_k2^T, text W_v2^T) W_o2^T + b
 *   n3 = LayerNorm(h);  [a, g] = n3 ff1^T + b;  h += (a * GELU(g)) ff2^T + b
 *   y  = h proj_out^T + b + x
 *   x            [B, h*W, C] bf16 band tokens
 *   text         [B, n_text, text_dim] bf16 conditioning features
 *   k_up .. v_dn stale neighbour keys/values as in pcpp_partial_attention
 *   y            [B, h*W, C] bf16 output
 *   k_fresh_out, v_fresh_out  [B, h*W, C] bf16: this band's keys/values of
 *                the step, what the neighbours read as stale context at the
 *                next step (Sec. 3.2); either may be NULL
 *   workspace    device scratch, ws_bytes >= the workspace size
 * Requires dtype PCPP_DTYPE_BF16 and head_dim 64 (PCPP_ENOTSUP otherwise),
 * C <= 2048 and gn_groups <= 256 (PCPP_ENOTSUP), text_dim >= 32 with text_dim % 32 == 0,
 * n_text >= 1, ff_inner % 64 == 0, C % gn_groups == 0 (PCPP_EINVAL).  All
 * pointers, weights included, must be 16-byte aligned (PCPP_EINVAL).
 * The workspace needs no clearing (see pcpp_transformer_block_workspace_size).
 */
int pcpp_transformer_block(const pcpp_geom_t* g, const pcpp_block_weights_t* w,
                           const void* x, const void* text, int32_t n_text,
                           int32_t text_dim,
                           const void* k_up, const void* v_up,
                           const void* k_dn, const void* v_dn,
                           void* y, void* k_fresh_out, void* v_fresh_out,
                           void* workspace, size_t ws_bytes, void* stream);

/*
 * pcpp_transformer_block with synchronized GroupNorm (Sec. 3.3 keeps the
 * GroupNorm of DistriFusion, whose statistics cover the whole image and are
 * exchanged among all devices).  Arguments as pcpp_transformer_block, plus:
 *   gn_bands  [n_patches][B][gn_groups][3] float32: (count, mean, M2) of
 *             every band's GroupNorm input (M2 = sum of squared deviations
 *             from that band's mean), as all-gathered from the previous
 *             step; entry patch_idx is not read (this band's own statistics
 *             of this step take its place).  The bands are merged in band
 *             order.  NULL: band-local statistics (pcpp_transformer_block).
 *   gn_own    [B][gn_groups][3] float32 output: this band's own statistics
 *             of this step, what the other bands read at the next one; may
 *             be NULL.
 * Both need 4-byte alignment (PCPP_EINVAL otherwise).
 */
int pcpp_transformer_block_sync_gn(const pcpp_geom_t* g,
                                   const pcpp_block_weights_t* w,
                                   const void* x, const void* text,
                                   int32_t n_text, int32_t text_dim,
                                   const void* k_up, const void* v_up,
                                   const void* k_dn, const void* v_dn,
                                   const float* gn_bands, float* gn_own,
                                   void* y, void* k_fresh_out,
                                   void* v_fresh_out, void* workspace,
                                   size_t ws_bytes, void* stream);

/*
 * SDXL's transformer module of depth d (2 at the first transformer level, 10
 * at the second) on band i: GroupNorm -> proj_in -> d basic blocks ->
 * proj_out + the module input.  Each basic block is pcpp_transformer_block's
 * body (LayerNorm, Q/K/V, partially conditioned self-attention over the
 * band and the stale neighbour rows, out-proj + residual, LayerNorm,
 * cross-attention to the text, out-proj + residual, LayerNorm, GEGLU
 * feed-forward + residual) with its own weights and its own stale K/V: every
 * self-attention layer exchanges its own K and V (Sec. 3.2, 3.3).  Depth 1
 * is exactly pcpp_transformer_block.
 */
typedef struct {
    const void* ln1_gamma;   const void* ln1_beta;      /* [C]                 */
    const void* attn1_qkv_w;                            /* [3C, C] W_q, W_k, W_v */
    const void* attn1_out_w; const void* attn1_out_b;   /* [C, C], [C]         */
    const void* ln2_gamma;   const void* ln2_beta;      /* [C]                 */
    const void* attn2_q_w;                              /* [C, C]              */
    const void* attn2_kv_w;                             /* [2C, T] W_k, W_v    */
    const void* attn2_out_w; const void* attn2_out_b;   /* [C, C], [C]         */
    const void* ln3_gamma;   const void* ln3_beta;      /* [C]                 */
    const void* ff1_w;       const void* ff1_b;         /* [2F, C], [2F]       */
    const void* ff2_w;       const void* ff2_b;         /* [C, F], [C]         */
} pcpp_basic_block_weights_t;

typedef struct {
    const void* gn_gamma;    const void* gn_beta;       /* [C] (eps 1e-6)      */
    const void* proj_in_w;   const void* proj_in_b;     /* [C, C], [C]         */
    const void* proj_out_w;  const void* proj_out_b;    /* [C, C], [C]         */
    const pcpp_basic_block_weights_t* blocks;           /* host array [depth]  */
    int32_t depth;                                      /* 1 .. 64             */
    int32_t ff_inner;                                   /* F, multiple of 64   */
    int32_t gn_groups;                                  /* dividing C          */
} pcpp_module_weights_t;

/* Bytes of device workspace (0 if invalid); no clearing needed, as for
 * pcpp_transformer_block_workspace_size.  It grows with the depth up to 16
 * basic blocks: the text K/V of up to 16 blocks come from one product. */
size_t pcpp_transformer_module_workspace_size(const pcpp_geom_t* g,
                                              const pcpp_module_weights_t* w,
                                              int32_t n_text, int32_t text_dim);

/*
 * k_up, v_up, k_dn, v_dn: host arrays of depth device pointers, entry j the
 * stale neighbour K/V of basic block j as in pcpp_partial_attention (the
 * arrays may be NULL where the band has no such neighbour or r = 0).
 * k_fresh_out, v_fresh_out: NULL, or host arrays of depth device pointers
 * (entries may be NULL) receiving basic block j's own K and V [B, h*W, C].
 * gn_bands / gn_own: NULL, or the synchronized GroupNorm's statistics as in
 * pcpp_transformer_block_sync_gn.  Other arguments, requirements and errors
 * as pcpp_transformer_block.  Asynchronous on `stream`.
 */
int pcpp_transformer_module(const pcpp_geom_t* g, const pcpp_module_weights_t* w,
                            const void* x, const void* text, int32_t n_text,
                            int32_t text_dim,
                            const void* const* k_up, const void* const* v_up,
                            const void* const* k_dn, const void* const* v_dn,
                            const float* gn_bands, float* gn_own, void* y,
                            void* const* k_fresh_out, void* const* v_fresh_out,
                            void* workspace, size_t ws_bytes, void* stream);

/*
 * p-aware boundary messages of the neighbour exchange (Sec. 3.2 with Eq. 1).
 * At the next step band i-1 reads the first r rows of band i's fresh keys
 * and values (its context below) and band i+1 reads the last r rows (its
 * context above), r = min(h, floor(p*h + 1e-9)).  Sending only those rows
 * instead of the whole band is the p-aware form of the exchange; these
 * calls build and place the messages on one device (the transfer between
 * devices is the caller's).
 *
 * Message layout: [B][2][r*W][C] - per image, the r key rows, then the r
 * value rows, each row W tokens of C elements, dtype of g.
 */

/* Bytes of one message for geometry g: B * 2 * r * W * C * element size
 * (0 for an invalid geometry, and when r = 0 or n = 1). */
size_t pcpp_boundary_bytes(const pcpp_geom_t* g);

/*
 * Builds band i's messages from its fresh keys/values [B, h*W, C]:
 *   send_up  for band i-1: rows 0 .. r-1 of this band (needed when i > 0
 *            and r > 0, else ignored and may be NULL)
 *   send_dn  for band i+1: rows h-r .. h-1 (needed when i < n-1 and r > 0)
 * Messages must not overlap the inputs or each other (PCPP_EINVAL).  No
 * alignment is required.  Asynchronous on `stream`.
 */
int pcpp_pack_boundary(const pcpp_geom_t* g, const void* k_fresh,
                       const void* v_fresh, void* send_up, void* send_dn,
                       void* stream);

/*
 * Places the messages band i received into its stale buffers [B, h*W, C],
 * at the rows pcpp_partial_attention reads from them:
 *   recv_up (built by band i-1 as its send_dn) -> the last r rows of k_up
 *            and v_up (needed when i > 0 and r > 0)
 *   recv_dn (built by band i+1 as its send_up) -> the first r rows of k_dn
 *            and v_dn (needed when i < n-1 and r > 0)
 * The other rows of the stale buffers are left untouched; the attention
 * never reads them.  Buffers must not overlap (PCPP_EINVAL).  Asynchronous.
 */
int pcpp_unpack_boundary(const pcpp_geom_t* g, const void* recv_up,
                         const void* recv_dn, void* k_up, void* v_up,
                         void* k_dn, void* v_dn, void* stream);

/*
 * Messages of the exchange with multi-hop context (p > 1, the context
 * beyond the immediate neighbours that Sec. 6 suggests for many bands; the
 * stale blocks are the compact ones pcpp_partial_attention_multihop reads).
 * With r = floor(p*h + 1e-9), bands i and j exchange
 *   rows(i, j) = clamp(r - (|i - j| - 1) * h, 0, h)
 * rows in each direction: band j above band i reads band i's first rows,
 * band j below reads its last rows.  For |i - j| = 1 and p <= 1 these are
 * the messages of pcpp_pack_boundary.  Same message layout as above:
 * [B][2][rows*W][C].  The geometry g is band i's; p may go up to
 * max(1, n - 1).  `peer` is j, any band index; j = i and bands out of reach
 * give rows = 0.
 */

/* Bytes of the message between bands g.patch_idx and peer, either
 * direction (0 when none, or for invalid arguments). */
size_t pcpp_multihop_message_bytes(const pcpp_geom_t* g, int32_t peer);

/*
 * Builds band i's message for band `peer` from its fresh keys/values
 * [B, h*W, C].  Nothing to do (PCPP_OK, pointers may be NULL) when rows =
 * 0.  The message must not overlap the inputs (PCPP_EINVAL); peer out of
 * range is PCPP_EINVAL.  Asynchronous on `stream`.
 */
int pcpp_pack_multihop(const pcpp_geom_t* g, int32_t peer,
                       const void* k_fresh, const void* v_fresh, void* send,
                       void* stream);

/*
 * Places the message band i received from band `peer` (built there by
 * pcpp_pack_multihop with peer = i) into band i's compact stale blocks, at
 * the image rows it holds:
 *   peer < i: k_above/v_above [B, up*W, C] (image rows i*h-up .. i*h-1)
 *             receive band peer's last rows; the below pair may be NULL
 *   peer > i: k_below/v_below [B, dn*W, C] (rows (i+1)*h .. (i+1)*h+dn-1)
 *             receive band peer's first rows; the above pair may be NULL
 * Other rows are left untouched.  Calling it for every other band fills
 * both blocks completely.  Buffers must not overlap (PCPP_EINVAL).
 * Asynchronous on `stream`.
 */
int pcpp_unpack_multihop(const pcpp_geom_t* g, int32_t peer,
                         const void* recv, void* k_above, void* v_above,
                         void* k_below, void* v_below, void* stream);

/*
 * SDXL-shaped ResNet block on one row band: the U-Net's convolution layers
 * (Sec. 3.3 keeps their exchange of boundary pixels: a band's 3x3
 * convolution reads its neighbours' edge rows of the convolution input as
 * exchanged at the previous step).
 *   a1 = SiLU(GroupNorm(x));           h1 = conv3x3(a1) + conv1_b + tb
 *   tb = SiLU(temb) temb_w^T + temb_b  (per image, added to every token)
 *   a2 = SiLU(GroupNorm(h1));          y  = conv3x3(a2) + conv2_b + s
 *   s  = x (c_in == c_out), else x skip_w^T + skip_b (a 1x1 convolution)
 * The convolutions pad with zeros at the image's edges (left, right, and
 * above band 0 / below band n-1) and read the neighbours' edge rows
 * elsewhere.  bf16 storage, float32 accumulation; a1, h1 and a2 are stored
 * in bf16, s in float32.
 */
typedef struct {
    int32_t H, W;          /* the layer's token grid                         */
    int32_t n_patches;     /* n, H % n == 0                                  */
    int32_t patch_idx;     /* band i, 0-based                                */
    int32_t c_in, c_out;   /* channels, multiples of 64, <= 2560             */
    int32_t temb_dim;      /* time-embedding width T, multiple of 8          */
    int32_t groups;        /* GroupNorm groups, dividing c_in and c_out, <= 256 */
    int32_t batch;         /* images B (the guidance branches), <= 65535     */
    float eps;             /* GroupNorm epsilon (SDXL: 1e-5)                 */
    int32_t reserved;      /* must be 0                                      */
} pcpp_resnet_geom_t;

/* Device pointers, bf16, 16-byte aligned.  3x3 kernels are
 * [c_out][3][3][c_in_of_that_conv] (tap-major, channel-minor: element
 * (o, ky, kx, c) at ((o * 3 + ky) * 3 + kx) * C + c), linears [out][in]. */
typedef struct {
    const void* gn1_gamma; const void* gn1_beta;   /* [c_in]                 */
    const void* conv1_w;   const void* conv1_b;    /* [c_out][3][3][c_in], [c_out] */
    const void* temb_w;    const void* temb_b;     /* [c_out][T], [c_out]    */
    const void* gn2_gamma; const void* gn2_beta;   /* [c_out]                */
    const void* conv2_w;   const void* conv2_b;    /* [c_out][3][3][c_out], [c_out] */
    const void* skip_w;    const void* skip_b;     /* [c_out][c_in], [c_out]; used (and
                                                      required) only when c_in != c_out */
} pcpp_resnet_weights_t;

/* Bytes of device workspace pcpp_resnet_block needs (0 if g is invalid).
 * The workspace needs no clearing; nothing in it survives a call. */
size_t pcpp_resnet_block_workspace_size(const pcpp_resnet_geom_t* g);

/*
 *   x            [B, h*W, c_in] bf16 band tokens (h = H / n)
 *   temb         [B, T] bf16 time embedding of the step
 *   edges1_up    the band above's edges1_out of the previous step
 *                [B, 2, W, c_in] (its row 1, the band's last row, is read);
 *                needed when i > 0, else ignored
 *   edges1_dn    the band below's edges1_out (its row 0 is read); needed
 *                when i < n-1
 *   edges2_up/dn the same for the second convolution's input, [B, 2, W, c_out]
 *   gn1_bands,   NULL: GroupNorm statistics over the band's own tokens.
 *   gn2_bands    Else the synchronized GroupNorm (Sec. 3.3) as in
 *                pcpp_transformer_block_sync_gn: [n][B][groups] x (count,
 *                mean, M2) float32 of every band, entry i replaced by this
 *                band's own; 4-byte aligned
 *   gn1_own,     NULL, or [B][groups] x (count, mean, M2) float32 of this
 *   gn2_own      band's two GroupNorm inputs, for the others' next step
 *   y            [B, h*W, c_out] bf16 output
 *   edges1_out,  NULL, or this band's first and last rows of a1 / a2,
 *   edges2_out   [B, 2, W, c] bf16: what its neighbours read at the next step;
 *                they must not overlap each other or the edges inputs
 * Errors: PCPP_EINVAL (geometry, NULL or misaligned pointers, 16-byte
 * alignment for the bf16 tensors), PCPP_ENOTSUP (channels not multiples of
 * 64 or above 2560, groups above 256), PCPP_EWORKSPACE.  Asynchronous.
 */
int pcpp_resnet_block(const pcpp_resnet_geom_t* g, const pcpp_resnet_weights_t* w,
                      const void* x, const void* temb,
                      const void* edges1_up, const void* edges1_dn,
                      const void* edges2_up, const void* edges2_dn,
                      const float* gn1_bands, float* gn1_own,
                      const float* gn2_bands, float* gn2_own,
                      void* y, void* edges1_out, void* edges2_out,
                      void* workspace, size_t ws_bytes, void* stream);

/*
 * The U-Net's 3x3 convolutions on one row band (Sec. 3.3 keeps the exchange
 * of boundary pixels for convolutions): the row directly above the band and
 * the row directly below it come from the neighbours (their last / first
 * row of the convolution input, as exchanged), zeros at the image's edges
 * and at the left and right.  Weights [c_out][3][3][c_in] bf16 (element
 * (o, ky, kx, c) at ((o * 3 + ky) * 3 + kx) * c_in + c), bias [c_out] or
 * NULL; bf16 storage, float32 accumulation.
 *   PCPP_CONV_SAME  stride 1: y [B, h*W, c_out]
 *   PCPP_CONV_DOWN  stride 2, padding 1 (SDXL's downsampler): output (y, x)
 *                   reads input rows 2y-1 .. 2y+1 of the band, so only the
 *                   row above is needed; h and W even; y [B, (h/2)*(W/2), c_out]
 *   PCPP_CONV_UP    nearest 2x upsampling, then stride 1 (SDXL's upsampler):
 *                   the neighbour rows are upsampled the same way;
 *                   y [B, (2h)*(2W), c_out]
 */
#define PCPP_CONV_SAME 0
#define PCPP_CONV_DOWN 1
#define PCPP_CONV_UP   2

typedef struct {
    int32_t H, W;          /* the input's token grid                         */
    int32_t n_patches;     /* n, H % n == 0                                  */
    int32_t patch_idx;     /* band i, 0-based                                */
    int32_t c_in, c_out;   /* multiples of 64                                */
    int32_t batch;         /* images B, <= 65535                             */
    int32_t mode;          /* PCPP_CONV_SAME, PCPP_CONV_DOWN or PCPP_CONV_UP */
    int32_t reserved;      /* must be 0                                      */
} pcpp_conv_geom_t;

/* Bytes of device workspace pcpp_conv3x3 needs (0 if g is invalid).  The
 * workspace needs no clearing; nothing in it survives a call. */
size_t pcpp_conv3x3_workspace_size(const pcpp_conv_geom_t* g);

/*
 *   x       [B, h*W, c_in] bf16 band tokens (h = H / n)
 *   row_up  [B, W, c_in] the row above the band (the band above's last row);
 *           needed when i > 0, else ignored
 *   row_dn  [B, W, c_in] the row below (the band below's first row); needed
 *           when i < n-1 for SAME and UP, ignored for DOWN
 *   w, bias, y as above; all pointers 16-byte aligned, y must not overlap
 *           the inputs.
 * Errors: PCPP_EINVAL (geometry, NULL or misaligned pointers), PCPP_ENOTSUP
 * (channels not multiples of 64), PCPP_EWORKSPACE.  Asynchronous on `stream`.
 */
int pcpp_conv3x3(const pcpp_conv_geom_t* g, const void* x, const void* row_up,
                 const void* row_dn, const void* w, const void* bias, void* y,
                 void* workspace, size_t ws_bytes, void* stream);

/*
 * pcpp_conv3x3 that also exports the band's first and last input rows (Sec.
 * 3.2: what the neighbours read as row_dn and row_up at the next step):
 *   first_out, last_out  [B, W, c_in] (either may be NULL), 16-byte aligned,
 *                        not overlapping the inputs, y or each other
 *                        (PCPP_EINVAL).  UP exports the rows before upsampling.
 * Otherwise the same as pcpp_conv3x3 (which is this call without exports).
 */
int pcpp_conv3x3_export(const pcpp_conv_geom_t* g, const void* x,
                        const void* row_up, const void* row_dn, const void* w,
                        const void* bias, void* y, void* first_out,
                        void* last_out, void* workspace, size_t ws_bytes,
                        void* stream);

/*
 * [rows, ca] and [rows, cb] bf16 side by side into out [rows, ca + cb]: the
 * U-Net up path's concatenation of a level's state with its skip connection
 * (the ResNet that follows takes ca + cb channels).  b = NULL fills the cb
 * channels with zeros (the padding of the 4 latent channels to the 64 the
 * convolution takes).  ca, cb multiples of 8; pointers 16-byte aligned; out
 * must not overlap a or b (PCPP_EINVAL).  Asynchronous on `stream`.
 */
int pcpp_concat_channels(int64_t rows, const void* a, int32_t ca, const void* b,
                         int32_t cb, void* out, void* stream);

/*
 * GroupNorm over each image's tokens, affine, then SiLU if silu = 1: the
 * U-Net's output head before conv_out (SDXL: 32 groups, eps 1e-5).
 * bands = NULL: statistics of x itself.  Else the synchronized GroupNorm
 * (Sec. 3.3): bands [n_bands][batch][groups] x (count, mean, M2) float32 of
 * every band, entry `band` replaced by x's own, merged in band order.
 * own_out: NULL, or [batch][groups] x (count, mean, M2) of x.  x, y [batch,
 * tokens, channels] bf16 (y may not overlap x), gamma/beta [channels];
 * channels % 8 == 0, <= 2560, groups <= 256 dividing channels (PCPP_ENOTSUP
 * otherwise).  The workspace needs no clearing.  Asynchronous on `stream`.
 */
/*
 * LayerNorm over the channel axis of float32 rows, affine, bf16 output: the
 * normalization in front of each of the transformer block's three branches
 * (SDXL: eps 1e-5; the block runs it internally), here on its own.  x [rows,
 * channels] float32, y [rows, channels] bf16 (y may not overlap x),
 * gamma/beta [channels] bf16; 1 <= rows <= 2^24; channels % 4 == 0 and
 * <= 2048 (PCPP_ENOTSUP otherwise); eps > 0; pointers 16-byte aligned
 * (PCPP_EINVAL).  Asynchronous on `stream`.
 */
int pcpp_layer_norm(int64_t rows, int32_t channels, float eps, const float* x,
                    const void* gamma, const void* beta, void* y,
                    void* stream);

size_t pcpp_group_norm_workspace_size(int32_t batch, int32_t tokens,
                                      int32_t channels, int32_t groups);
int pcpp_group_norm(int32_t batch, int32_t tokens, int32_t channels,
                    int32_t groups, float eps, int32_t silu, const void* x,
                    const void* gamma, const void* beta, const float* bands,
                    int32_t n_bands, int32_t band, float* own_out, void* y,
                    void* workspace, size_t ws_bytes, void* stream);

/*
 * The update of a band's latent at the end of a step (Sec. 3.1): the two
 * guidance branches' noise predictions are combined by classifier-free
 * guidance (Eq. 2), e = eps_u + s (eps_c - eps_u), and then
 *   PCPP_STEP_DDPM: Eq. 3 and Eq. 4,
 *     x_{t-1} = (x_t - (1 - alpha_t) / sqrt(1 - alphabar_t) e) / sqrt(alpha_t)
 *               + sigma_t z          (z may be NULL: no noise term)
 *   PCPP_STEP_DDIM: the deterministic DDIM update (the paper's sampler,
 *     Sec. 4): x_{t-1} = sqrt(alphabar_prev) x0 + sqrt(1 - alphabar_prev) e
 *     with x0 = (x_t - sqrt(1 - alphabar_t) e) / sqrt(alphabar_t); z must be NULL.
 * The two coefficients of x_t and e are computed on the host in double
 * precision, the update in float32 on the device.
 */
#define PCPP_STEP_DDPM 0
#define PCPP_STEP_DDIM 1

typedef struct {
    float guidance;       /* s (the paper uses 5), finite                  */
    float alpha_t;        /* DDPM: (0, 1]                                   */
    float alphabar_t;     /* DDPM: (0, 1); DDIM: (0, 1]                     */
    float sigma_t;        /* DDPM: scale of z                               */
    float alphabar_prev;  /* DDIM: (0, 1], the level stepped to             */
    int32_t mode;         /* PCPP_STEP_DDPM or PCPP_STEP_DDIM               */
    int32_t reserved;     /* must be 0                                      */
} pcpp_step_params_t;

/*
 * x_t, eps_uncond, eps_cond, z, x_prev: n float32 values each (any layout,
 * the same for all), device pointers; x_prev may be x_t (in place), no
 * other overlap.  No alignment is required.  PCPP_EINVAL for invalid
 * parameters or NULL pointers (n > 0).  Asynchronous on `stream`.
 */
int pcpp_guided_step(const pcpp_step_params_t* sp, int64_t n, const float* x_t,
                     const float* eps_uncond, const float* eps_cond,
                     const float* z, float* x_prev, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* PCPP_H */
