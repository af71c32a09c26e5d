// Partially conditioned self-attention, bf16 storage, on gfx950 MFMA.
//
// Computes, per image and head, softmax(Q K_ctx^T / sqrt(64)) V_ctx where
// the key/value context is the band's fresh tokens plus the stale boundary
// rows of its neighbours (Sec. 3.3 and Eq. 1 of arXiv 2412.02962).  The three
// key/value sources are read in place (no assembled copy): every key row of a
// 32-key tile picks its source from its token index.
//
// Work decomposition.  A unit is one 32-key tile of one 64-query block of one
// (image, head).  The query blocks are dealt out to the XCDs in contiguous
// ranges (consecutive blocks share a head, hence keys, in that XCD's L2);
// inside an XCD the units of its blocks, in (block, tile) order, are cut into
// equal contiguous ranges, one per workgroup, two workgroups per compute
// unit.  Workgroup w runs on XCD w % n_xcd (the hardware deals workgroups out
// round-robin), so every workgroup that shares a block shares an L2: a block
// split between workgroups is merged through that L2 with ordinary stores and
// one counter per split block (the last contributor to arrive merges and
// resets the counter to zero), without any cache-wide writeback.
//
// Inside a workgroup: 4 wavefronts, one per SIMD, split the tiles of the
// current block; each streams its own tiles through a private LDS ring (two K
// and two V slots, filled with direct global->LDS loads) and synchronises
// with nobody until the block's tiles are done, so the two workgroups on a
// compute unit interleave MFMA and softmax work freely.  The wavefronts'
// partial results are then merged through LDS.
//
// Per 32-key tile and wavefront (64 queries = two 32-query column blocks):
//   S^T = K Q^T      8 MFMA 32x32x16; K from LDS, Q^T in registers.  The
//                    transposed product leaves each lane with one query and
//                    16 of the tile's keys: a row max needs one exchange
//                    with the partner lane (lane ^ 32), the row sum none.
//   online softmax   in log2 units, p = exp2(s*log2(e)/8 - m) against the
//                    running max m; the tile max is only taken (and m
//                    raised, O and l rescaled) when a lane's probabilities
//                    of the tile sum to 2^20 or more, so p < 2^20.
//   O^T += V^T P^T   8 MFMA 32x32x16; P^T is the B operand taken straight
//                    from the S^T accumulators (inside each 16-key step the
//                    key order is permuted the same way on both operands);
//                    V^T comes from the row-major V tile through the
//                    transposing LDS read ds_read_b64_tr_b16.
// Tile x-1's P V MFMAs run while the softmax of tile x is computed.
// Row sums accumulate the bf16 probabilities with v_dot2 against (1, 1), so
// numerator and denominator see the same rounded weights.

#include <math.h>

#include "common.h"
#include "kernels.h"

namespace pcpp {

namespace {

constexpr int D = 64;
constexpr int TILE = 32;                   // keys per tile
constexpr int QB = 64;                     // queries per block
constexpr int NW = 4;                      // wavefronts per workgroup
constexpr int NTHREADS = 64 * NW;
constexpr int WG_PER_CU = 2;
constexpr int TILE_BYTES = TILE * D * 2;   // 4 KB of K or of V
constexpr int LOADS_PER_TILE = TILE_BYTES / 1024;  // 1 KB direct-to-LDS loads
constexpr int OSTR = 68;                   // merge buffer row stride (floats)
constexpr int RING_BYTES = NW * TILE_BYTES > QB * OSTR * 4 ? NW * TILE_BYTES : QB * OSTR * 4;
constexpr float P_LIMIT = 1048576.0f;      // 2^20: bound on a lane's probability sum per tile
constexpr int PIECE_SLOTS = 2;             // partial-result slots per workgroup
constexpr int MIN_TILES_PER_WAVE = 4;
constexpr int CUS_PER_XCD = 32;            // gfx950

static_assert(WG_PER_CU * (4 * RING_BYTES + NW * QB * 2 * 4 + 16) <= 160 * 1024,
              "two workgroups share a compute unit's LDS");

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef const __attribute__((address_space(1))) void* gptr_t;
typedef __attribute__((address_space(3))) void* lptr_t;

// LDS swizzles: 16-byte chunk c of tile row r is stored at slot c ^ mask(r).
// K rows are read 16 bytes per lane by 16 consecutive rows at one chunk; V
// rows by four rows x 32 bytes per 16 lanes (transposing read).
__device__ __forceinline__ int k_mask(int r) { return (r >> 1) & 7; }
__device__ __forceinline__ int v_mask(int r) { return ((r >> 1) & 3) << 1; }

struct Sched {
    int32_t n_xcd;      // XCDs; workgroup w runs on XCD w % n_xcd
    int32_t per_xcd;    // workgroups per XCD
    int32_t n_tiles;    // key tiles per query block
    int32_t nqb;        // query blocks per (image, head)
    int64_t n_blocks;   // query blocks in total
    int32_t whole;      // 1: ranges hold whole blocks only (no merging across workgroups)
    int* xcc_of;        // [grid]: XCC id + 1 each workgroup ran on (diagnostic)
    int* counters;      // [grid]: zero at launch, left zero
    float* part_o;      // [grid * PIECE_SLOTS][QB][D]
    float* part_ml;     // [grid * PIECE_SLOTS][QB][2]
};

__device__ __forceinline__ int64_t pick(int j, int end0, int end1, int64_t a0, int64_t a1, int64_t a2) {
    const int64_t a12 = j < end1 ? a1 : a2;
    return j < end0 ? a0 : a12;
}

// Transposing LDS reads of one V^T operand (rows p and p + 8 rows), in
// inline assembly: the compiler sees no address for them, so it does not
// order them after the direct-to-LDS loads still in flight into other ring
// slots.  Their results are complete only after lds_wait().
__device__ __forceinline__ void lds_read_tr2(const char* p, u32x2& lo, u32x2& hi) {
    const uint32_t a = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const char*)p;
    asm volatile("ds_read_b64_tr_b16 %0, %2\n\tds_read_b64_tr_b16 %1, %2 offset:1024"
                 : "=&v"(lo), "=&v"(hi)
                 : "v"(a));
}
// Waits for every outstanding LDS read; the operands tie the wait to the
// registers the reads wrote.
__device__ __forceinline__ void lds_wait(u32x2 (&v)[8]) {
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4]), "+v"(v[5]), "+v"(v[6]), "+v"(v[7]));
}
// The four 16-byte K reads of one score product (chunks c0, c0+2, c0+4,
// c0+6 of a row, each at its swizzled slot), in inline assembly for the
// same reason, followed by their wait.
__device__ __forceinline__ void lds_read_k4(const char* row, int c0, int mask, u32x4 (&k)[4]) {
    const uint32_t a = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const char*)row;
    const uint32_t a0 = a + (((c0 + 0) ^ mask) << 4), a1 = a + (((c0 + 2) ^ mask) << 4);
    const uint32_t a2 = a + (((c0 + 4) ^ mask) << 4), a3 = a + (((c0 + 6) ^ mask) << 4);
    asm volatile(
        "ds_read_b128 %0, %4\n\tds_read_b128 %1, %5\n\tds_read_b128 %2, %6\n\tds_read_b128 %3, %7\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(k[0]), "=&v"(k[1]), "=&v"(k[2]), "=&v"(k[3])
        : "v"(a0), "v"(a1), "v"(a2), "v"(a3));
}

// Value of lanes l and l ^ 32 combined, without an LDS round trip.
__device__ __forceinline__ float max_xor32(float v) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_xor32(float v) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Workgroup of XCD-local index j owns units [T*j/J, T*(j+1)/J) of its XCD's
// T units (or, with whole blocks, the blocks [B*j/J, B*(j+1)/J)).
__device__ __forceinline__ int64_t range_start(int64_t T, int64_t nblk, int n_tiles, int j, int J, bool whole) {
    return whole ? nblk * j / J * n_tiles : T * j / J;
}
// Workgroup whose range holds unit u (ranges may be empty when J > T).
__device__ __forceinline__ int owner_of(int64_t u, int64_t T, int J) { return (int)(((u + 1) * J - 1) / T); }

__global__ __launch_bounds__(NTHREADS, WG_PER_CU) void attn_bf16_kernel(AttnParams p, Sched sc) {
    // Separate arrays per ring slot: with distinct objects the compiler can
    // tell a direct-to-LDS load into one slot from reads of another and does
    // not make those reads wait for the loads.  Wavefront w uses bytes
    // [w*4K, (w+1)*4K) of each; after a block the four arrays are the four
    // wavefronts' merge buffers.
    __shared__ __attribute__((aligned(16))) char kring0[RING_BYTES];
    __shared__ __attribute__((aligned(16))) char kring1[RING_BYTES];
    __shared__ __attribute__((aligned(16))) char vring0[RING_BYTES];
    __shared__ __attribute__((aligned(16))) char vring1[RING_BYTES];
    __shared__ __attribute__((aligned(16))) float ml_lds[NW * QB * 2];  // (m, l) per wavefront and query
    __shared__ int flag_lds;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int col = lane & 31;
    const int half = lane >> 5;
    const int C = p.C;
    const int kv_end = p.kv.n_kv;
    const float sl2 = p.scale_log2;
    const bf16x2 ones = {(bf16)1.0f, (bf16)1.0f};
    const int n_tiles = sc.n_tiles;

    const int x = blockIdx.x % sc.n_xcd;
    const int j = blockIdx.x / sc.n_xcd;
    const int J = sc.per_xcd;
    if (tid == 0) sc.xcc_of[blockIdx.x] = (__builtin_amdgcn_s_getreg(0xf814) & 15) + 1;  // HW_REG_XCC_ID

    const int64_t bx0 = sc.n_blocks * x / sc.n_xcd;
    const int64_t nblk = sc.n_blocks * (x + 1) / sc.n_xcd - bx0;
    const int64_t T = nblk * n_tiles;
    const bool whole = sc.whole != 0;
    const int64_t s_j = range_start(T, nblk, n_tiles, j, J, whole);
    const int64_t e_j = range_start(T, nblk, n_tiles, j + 1, J, whole);

    // transposing-read lane geometry inside a V tile
    const int jj = lane & 15;
    const int tr_row = 4 * half + (jj >> 2);
    const int tr_e = 16 * ((lane >> 4) & 1) + 4 * (jj & 3);
    const int wbase = wave * TILE_BYTES;

    // Lane offsets (bytes) of the direct-to-LDS loads inside a tile: lane l
    // loads row 8i + (l >> 3), chunk (l & 7) ^ mask(row).  The K mask of
    // row 8i + r is k_mask(r) ^ 4 for odd i; the V mask does not depend on i.
    const int ld_r = lane >> 3, ld_pos = lane & 7;
    const uint32_t lane_off_k0 = ld_r * C * 2 + ((ld_pos ^ k_mask(ld_r)) << 4);
    const uint32_t lane_off_k1 = ld_r * C * 2 + ((ld_pos ^ k_mask(ld_r) ^ 4) << 4);
    const uint32_t lane_off_v = ld_r * C * 2 + ((ld_pos ^ v_mask(ld_r)) << 4);

    // lane geometry of the merge: query ql of the block, dims [d0, d0 + 16)
    const int ql = 16 * wave + (lane >> 2);
    const int d0 = 16 * (lane & 3);

    for (int64_t u = s_j; u < e_j;) {
        const int64_t bl = u / n_tiles;  // block, XCD-local
        const int t0 = (int)(u - bl * n_tiles);
        const int64_t bend = (bl + 1) * n_tiles;
        const int t1 = (int)((e_j < bend ? e_j : bend) - bl * n_tiles);
        const bool first_seg = u == s_j;
        u = bl * n_tiles + t1;
        const int64_t blk = bx0 + bl;
        const int qb = (int)(blk % sc.nqb);
        const int64_t bh = blk / sc.nqb;
        const int head = (int)(bh % p.heads);
        const int b = (int)(bh / p.heads);
        const int head_off = head * D;

        // this wavefront's tiles [w0, w0 + n)
        const int nseg = t1 - t0;
        const int w0 = t0 + nseg * wave / NW;
        const int n = t0 + nseg * (wave + 1) / NW - w0;

        // Row bases (bytes), pre-offset so that key row j of a segment is base + j*C*2.
        const int64_t o0 = (int64_t)b * p.kv.bstride[0] + head_off;
        const int64_t o1 = (int64_t)b * p.kv.bstride[1] - (int64_t)p.kv.end0 * C + head_off;
        const int64_t o2 = (int64_t)b * p.kv.bstride[2] - (int64_t)p.kv.end1 * C + head_off;
        const int64_t ka0 = (int64_t)(uintptr_t)p.kv.k[0] + o0 * 2;
        const int64_t ka1 = (int64_t)(uintptr_t)p.kv.k[1] + o1 * 2;
        const int64_t ka2 = (int64_t)(uintptr_t)p.kv.k[2] + o2 * 2;
        const int64_t va0 = (int64_t)(uintptr_t)p.kv.v[0] + o0 * 2;
        const int64_t va1 = (int64_t)(uintptr_t)p.kv.v[1] + o1 * 2;
        const int64_t va2 = (int64_t)(uintptr_t)p.kv.v[2] + o2 * 2;

        // Stage tile t (32 rows x 128 bytes) into dst: four 1 KB loads of
        // eight rows each; lane l fills LDS chunk l & 7 of its row with the
        // global chunk that the swizzle puts there.  A tile inside one key
        // source takes a scalar base and the fixed lane offsets; a tile that
        // straddles two sources or the end picks the source row by row.
        auto issue_tile = [&](int t_in, char* dst, bool is_v) {
            const int t = __builtin_amdgcn_readfirstlane(t_in);
            const int j0 = t * TILE, j1 = j0 + TILE;
            const bool one_src = j1 <= kv_end && (j1 <= p.kv.end0 || j0 >= p.kv.end0) &&
                                 (j1 <= p.kv.end1 || j0 >= p.kv.end1);
            if (one_src) {
                const int64_t base = (is_v ? pick(j0, p.kv.end0, p.kv.end1, va0, va1, va2)
                                           : pick(j0, p.kv.end0, p.kv.end1, ka0, ka1, ka2)) +
                                     (int64_t)j0 * C * 2;
#pragma unroll
                for (int i = 0; i < LOADS_PER_TILE; ++i) {
                    const uint32_t off = is_v ? lane_off_v : (i & 1) ? lane_off_k1 : lane_off_k0;
                    const char* g = (const char*)(uintptr_t)(base + (int64_t)i * 8 * C * 2) + off;
                    __builtin_amdgcn_global_load_lds((gptr_t)g, (lptr_t)(dst + wbase + i * 1024), 16, 0, 0);
                }
                return;
            }
            const int rr = lane >> 3;
            const int pos = lane & 7;
#pragma unroll
            for (int i = 0; i < LOADS_PER_TILE; ++i) {
                const int row = 8 * i + rr;
                const int c = pos ^ (is_v ? v_mask(row) : k_mask(row));
                int jk = t * TILE + row;
                jk = jk < kv_end ? jk : kv_end - 1;
                const int64_t base = is_v ? pick(jk, p.kv.end0, p.kv.end1, va0, va1, va2)
                                          : pick(jk, p.kv.end0, p.kv.end1, ka0, ka1, ka2);
                const int64_t addr = base + (int64_t)jk * C * 2 + c * 16;
                __builtin_amdgcn_global_load_lds((gptr_t)(uintptr_t)addr, (lptr_t)(dst + wbase + i * 1024), 16, 0, 0);
            }
        };

        // Q^T operands of the block's 64 queries.
        const int q_base = qb * QB;
        bf16x8 qop[2][4];
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) {
            const int qrow = min(q_base + 32 * cb + col, p.nq - 1);
            const bf16* qp = (const bf16*)p.q + (int64_t)b * p.q_bstride + (int64_t)qrow * C + head_off + 8 * half;
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) qop[cb][kk] = *(const bf16x8*)(qp + 16 * kk);
        }

        f32x16 o[2][2];
        float m_run[2], l_run[2];
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) {
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int r = 0; r < 16; ++r) o[cb][mb][r] = 0.f;
            m_run[cb] = -INFINITY;
            l_run[cb] = 0.f;
        }

        // Raw scores of tile t for the 64 queries (two 32-query column
        // blocks), masked past the last key.
        auto qk = [&](int t, const char* kring, f32x16* sc2, bool may_mask) {
            u32x4 kr[4];
            lds_read_k4(kring + wbase + col * 128, half, k_mask(col), kr);
            bf16x8 kop[4];
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) kop[kk] = __builtin_bit_cast(bf16x8, kr[kk]);
#pragma unroll
            for (int cb = 0; cb < 2; ++cb)
#pragma unroll
                for (int rr = 0; rr < 16; ++rr) sc2[cb][rr] = 0.f;
#pragma unroll
            for (int kk = 0; kk < 4; ++kk)
#pragma unroll
                for (int cb = 0; cb < 2; ++cb) sc2[cb] = mfma32x32x16(kop[kk], qop[cb][kk], sc2[cb]);
            if (may_mask) {
#pragma unroll
                for (int cb = 0; cb < 2; ++cb)
#pragma unroll
                    for (int rr = 0; rr < 16; ++rr) {
                        const int jk = t * TILE + 8 * (rr >> 2) + 4 * half + (rr & 3);
                        if (jk >= kv_end) sc2[cb][rr] = -INFINITY;
                    }
            }
        };

        // Online softmax.  Probabilities are taken against the running max,
        // p = exp2(s*log2(e)/8 - m), and summed per lane in the bf16 values
        // the P V product uses.  Only when a lane's 16 probabilities of the
        // tile sum to 2^20 or more (or to inf / NaN: the first tile, where m
        // is -inf) is the tile's max taken, m raised to it, O and l rescaled
        // and the probabilities recomputed.  So p < 2^20 always, and the max
        // reduction is off the common path.
        auto tile_probs = [&](const f32x16* sc2, int cb, bf16x8 (*pb)[2], float& lt) {
            const float mneg = -m_run[cb];
#pragma unroll
            for (int rr = 0; rr < 16; ++rr)
                pb[cb][rr >> 3][rr & 7] = f32_to_bf16(fast_exp2(fmaf(sc2[cb][rr], sl2, mneg)));
            float s0 = 0.f, s1 = 0.f;
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                bf16x2 p0 = {pb[cb][0][2 * w], pb[cb][0][2 * w + 1]};
                bf16x2 p1 = {pb[cb][1][2 * w], pb[cb][1][2 * w + 1]};
                s0 = __builtin_amdgcn_fdot2_f32_bf16(p0, ones, s0, false);
                s1 = __builtin_amdgcn_fdot2_f32_bf16(p1, ones, s1, false);
            }
            lt = s0 + s1;
        };
        auto probs = [&](const f32x16* sc2, bf16x8 (*pb)[2]) {
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) {
                float lt;
                tile_probs(sc2, cb, pb, lt);
                if (__any(!(lt < P_LIMIT))) {
                    float m4[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        m4[i] = fmaxf(fmaxf(sc2[cb][4 * i], sc2[cb][4 * i + 1]), fmaxf(sc2[cb][4 * i + 2], sc2[cb][4 * i + 3]));
                    const float mx = max_xor32(fmaxf(fmaxf(m4[0], m4[1]), fmaxf(m4[2], m4[3]))) * sl2;
                    const float m_new = fmaxf(m_run[cb], mx);
                    const float alpha = fast_exp2(m_run[cb] - m_new);
                    m_run[cb] = m_new;
                    l_run[cb] *= alpha;
#pragma unroll
                    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                        for (int rr = 0; rr < 16; ++rr) o[cb][mb][rr] *= alpha;
                    tile_probs(sc2, cb, pb, lt);
                }
                l_run[cb] += lt;
            }
        };

        // O^T += V^T P^T for the tile in vring.
        auto pv = [&](const char* vring, bf16x8 (*pb)[2]) {
            const char* vt = vring + wbase;
            u32x2 vr[8];
#pragma unroll
            for (int st = 0; st < 2; ++st) {
                const int row = 16 * st + tr_row;
#pragma unroll
                for (int mb = 0; mb < 2; ++mb) {
                    const int e = 32 * mb + tr_e;
                    const char* vp = vt + row * 128 + (((e >> 3) ^ v_mask(row)) << 4) + ((e & 7) << 1);
                    lds_read_tr2(vp, vr[4 * st + 2 * mb], vr[4 * st + 2 * mb + 1]);
                }
            }
            lds_wait(vr);
#pragma unroll
            for (int st = 0; st < 2; ++st)
#pragma unroll
                for (int mb = 0; mb < 2; ++mb) {
                    const u32x2 lo = vr[4 * st + 2 * mb], hi = vr[4 * st + 2 * mb + 1];
                    const u32x4 v4 = {lo[0], lo[1], hi[0], hi[1]};
                    const bf16x8 vop = __builtin_bit_cast(bf16x8, v4);
#pragma unroll
                    for (int cb = 0; cb < 2; ++cb) o[cb][mb] = mfma32x32x16(vop, pb[cb][st], o[cb][mb]);
                }
        };

        // Software pipeline over the wavefront's n tiles.  Round x computes
        // the scores of tile x and then tile x-1's P V product (MFMA), while
        // tile x's softmax (VALU) overlaps the latter; only tile x-1's bf16
        // probabilities carry over.  K(x+1) is loaded from the start of round
        // x into the K slot tile x-1 used, V(x+1) from the end of round x into
        // the V slot tile x-1 used; round x therefore only waits for K(x)
        // (and everything before it), with V(x) in flight.
        auto round_step = [&](int xr, const char* kcur, char* knext, char* vprev, bf16x8 (*pb_prev)[2],
                              bf16x8 (*pb_cur)[2]) {
            if (xr < n) {
                __builtin_amdgcn_s_waitcnt(0xF70 | LOADS_PER_TILE);  // vmcnt(4): K(x) has landed
                if (xr + 1 < n) issue_tile(w0 + xr + 1, knext, false);
            } else {
                __builtin_amdgcn_s_waitcnt(0xF70);  // vmcnt(0): V(n-1) has landed
            }
            const int t = w0 + xr;
            f32x16 s_cur[2];
            if (xr < n) qk(t, kcur, s_cur, t * TILE + TILE > kv_end);
            if (xr >= 1) pv(vprev, pb_prev);
            if (xr < n) probs(s_cur, pb_cur);
            if (xr + 1 < n) issue_tile(w0 + xr + 1, vprev, true);
        };
        if (n > 0) {
            bf16x8 pb0[2][2], pb1[2][2];
            issue_tile(w0, kring0, false);
            issue_tile(w0, vring0, true);
            for (int xr = 0; xr <= n; xr += 2) {
                round_step(xr, kring0, kring1, vring1, pb1, pb0);
                if (xr + 1 <= n) round_step(xr + 1, kring1, kring0, vring0, pb0, pb1);
            }
        }

        // ---- merge the wavefronts' partial results through LDS ----
        float l_tot[2];
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) l_tot[cb] = sum_xor32(l_run[cb]);
        if (half == 0) {
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) {
                float* ml = ml_lds + (wave * QB + 32 * cb + col) * 2;
                ml[0] = m_run[cb];
                ml[1] = l_tot[cb];
            }
        }
        __syncthreads();  // every wavefront is done with its ring; (m, l) are visible
        // merged max and sum of query q of the block over the wavefronts
        auto block_ml = [&](int q, float& M, float& L) {
            M = -INFINITY;
#pragma unroll
            for (int k = 0; k < NW; ++k) {
                const float* ml = ml_lds + (k * QB + q) * 2;
                if (ml[1] > 0.f) M = fmaxf(M, ml[0]);
            }
            L = 0.f;
#pragma unroll
            for (int k = 0; k < NW; ++k) {
                const float* ml = ml_lds + (k * QB + q) * 2;
                if (ml[1] > 0.f) L += ml[1] * fast_exp2(ml[0] - M);
            }
        };
        {
            char* mybuf = wave == 0 ? kring0 : wave == 1 ? kring1 : wave == 2 ? vring0 : vring1;
#pragma unroll
            for (int cb = 0; cb < 2; ++cb) {
                float M, L;
                block_ml(32 * cb + col, M, L);
                const float w_own = l_tot[cb] > 0.f ? fast_exp2(m_run[cb] - M) * __builtin_amdgcn_rcpf(L) : 0.f;
#pragma unroll
                for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                    for (int c4 = 0; c4 < 4; ++c4) {
                        float* dst = (float*)mybuf + (32 * cb + col) * OSTR + 32 * mb + 8 * c4 + 4 * half;
                        const f32x4 v = {o[cb][mb][4 * c4] * w_own, o[cb][mb][4 * c4 + 1] * w_own,
                                         o[cb][mb][4 * c4 + 2] * w_own, o[cb][mb][4 * c4 + 3] * w_own};
                        *(f32x4*)dst = v;
                    }
            }
        }
        __syncthreads();
        // normalised output of the workgroup's piece for (ql, [d0, d0+16))
        float acc[16];
        {
            const int off = ql * OSTR + d0;
            const float* b0 = (const float*)kring0 + off;
            const float* b1 = (const float*)kring1 + off;
            const float* b2 = (const float*)vring0 + off;
            const float* b3 = (const float*)vring1 + off;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const f32x4 v = *(const f32x4*)(b0 + 4 * i) + *(const f32x4*)(b1 + 4 * i) +
                                *(const f32x4*)(b2 + 4 * i) + *(const f32x4*)(b3 + 4 * i);
#pragma unroll
                for (int e = 0; e < 4; ++e) acc[4 * i + e] = v[e];
            }
        }
        float M_own, L_own;
        block_ml(ql, M_own, L_own);
        const int q_out = q_base + ql;
        bf16* out_row = (bf16*)p.out + (int64_t)b * p.q_bstride + (int64_t)q_out * C + head_off + d0;
        auto store_out = [&](const float* a, float scale) {
            if (q_out >= p.nq) return;
            bf16x8 v0, v1;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                v0[e] = f32_to_bf16(a[e] * scale);
                v1[e] = f32_to_bf16(a[8 + e] * scale);
            }
            *(bf16x8*)out_row = v0;
            *(bf16x8*)(out_row + 8) = v1;
        };

        if (t0 == 0 && t1 == n_tiles) {
            store_out(acc, 1.0f);
        } else {
            // A piece of a block that other workgroups of this XCD share.
            const int64_t slot = (int64_t)(x * J + j) * PIECE_SLOTS + (first_seg ? 0 : 1);
            float* po = sc.part_o + (slot * QB + ql) * D + d0;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const f32x4 v = {acc[4 * i], acc[4 * i + 1], acc[4 * i + 2], acc[4 * i + 3]};
                *(f32x4*)(po + 4 * i) = v;
            }
            if ((lane & 3) == 0) {
                float* pml = sc.part_ml + (slot * QB + ql) * 2;
                pml[0] = M_own;
                pml[1] = L_own;
            }
            __builtin_amdgcn_s_waitcnt(0xF70);  // vmcnt(0): this thread's stores reached the L2
            __syncthreads();
            const int64_t blk_u0 = bl * n_tiles;
            const int jf = owner_of(blk_u0, T, J);
            const int jl = owner_of(blk_u0 + n_tiles - 1, T, J);
            if (tid == 0) {
                // Count tiles: the contribution that completes the block's
                // n_tiles merges.  The counter lives at the index of the
                // block's first workgroup, unique among split blocks.
                int* counter = sc.counters + x * J + jf;
                const int prev = __hip_atomic_fetch_add(counter, t1 - t0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
                const int last = prev + (t1 - t0) == n_tiles;
                if (last) __hip_atomic_store(counter, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
                flag_lds = last;
            }
            __syncthreads();
            if (flag_lds) {
                // Every piece, this workgroup's own included, is read back
                // from the workspace and summed in workgroup order, so the
                // result does not depend on which contributor arrived last.
                float Mx = -INFINITY;
                for (int jo = jf; jo <= jl; ++jo) {
                    const int64_t so = range_start(T, nblk, n_tiles, jo, J, false);
                    if (so == range_start(T, nblk, n_tiles, jo + 1, J, false)) continue;
                    const int64_t sl = (int64_t)(x * J + jo) * PIECE_SLOTS + (so >= blk_u0 ? 0 : 1);
                    Mx = fmaxf(Mx, sc.part_ml[(sl * QB + ql) * 2]);
                }
                float wsum = 0.f;
                float res[16];
#pragma unroll
                for (int e = 0; e < 16; ++e) res[e] = 0.f;
                for (int jo = jf; jo <= jl; ++jo) {
                    const int64_t so = range_start(T, nblk, n_tiles, jo, J, false);
                    if (so == range_start(T, nblk, n_tiles, jo + 1, J, false)) continue;
                    const int64_t sl = (int64_t)(x * J + jo) * PIECE_SLOTS + (so >= blk_u0 ? 0 : 1);
                    const float* pml = sc.part_ml + (sl * QB + ql) * 2;
                    const float wk = pml[1] * fast_exp2(pml[0] - Mx);
                    wsum += wk;
                    const float* pk = sc.part_o + (sl * QB + ql) * D + d0;
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const f32x4 v = *(const f32x4*)(pk + 4 * i);
#pragma unroll
                        for (int e = 0; e < 4; ++e) res[4 * i + e] += wk * v[e];
                    }
                }
                store_out(res, 1.0f / wsum);
            }
        }
        __syncthreads();  // merge buffers and (m, l) are free for the next block
    }
}

struct Plan {
    int32_t n_xcd, per_xcd, grid, max_grid, n_tiles, nqb, whole;
    int64_t n_blocks;
    size_t off_xcc, off_counters, off_o, off_ml, ws_bytes;
};

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

int device_cus() {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 256;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
        return 256;
    return cus;
}

// Two workgroups per compute unit.  The workspace layout depends only on the
// compute unit count: [XCC record: max_grid ints][counters: max_grid ints]
// [partial outputs: max_grid x 2 slots][partial row statistics: same].
Plan make_plan(const AttnParams& p) {
    Plan pl;
    const int cus = device_cus();
    pl.max_grid = WG_PER_CU * cus;
    pl.n_tiles = (p.kv.n_kv + TILE - 1) / TILE;
    pl.nqb = (p.nq + QB - 1) / QB;
    pl.n_blocks = (int64_t)p.batch * p.heads * pl.nqb;
    // Merging across workgroups needs the XCD layout of a gfx950 device
    // (32 compute units per XCD); otherwise every range holds whole blocks.
    const bool xcd_known = cus % CUS_PER_XCD == 0;
    pl.n_xcd = xcd_known ? cus / CUS_PER_XCD : 1;
    pl.whole = xcd_known ? 0 : 1;
    const int64_t blk_per_xcd = (pl.n_blocks + pl.n_xcd - 1) / pl.n_xcd;
    int64_t per = pl.max_grid / pl.n_xcd;
    if (pl.whole) {
        if (per > blk_per_xcd) per = blk_per_xcd;
    } else {
        const int64_t need = (blk_per_xcd * pl.n_tiles + NW * MIN_TILES_PER_WAVE - 1) / (NW * MIN_TILES_PER_WAVE);
        if (per > need) per = need;
    }
    if (per < 1) per = 1;
    pl.per_xcd = (int32_t)per;
    pl.grid = pl.n_xcd * pl.per_xcd;
    size_t off = 0;
    pl.off_xcc = off;
    off += align256((size_t)pl.max_grid * sizeof(int));
    pl.off_counters = off;
    off += align256((size_t)pl.max_grid * sizeof(int));
    pl.off_o = off;
    off += align256((size_t)pl.max_grid * PIECE_SLOTS * QB * D * sizeof(float));
    pl.off_ml = off;
    off += align256((size_t)pl.max_grid * PIECE_SLOTS * QB * 2 * sizeof(float));
    pl.ws_bytes = off;
    return pl;
}

}  // namespace

size_t attention_bf16_ws_bytes(const AttnParams& p) { return make_plan(p).ws_bytes; }

hipError_t launch_attention_bf16(const AttnParams& p, void* ws, size_t ws_bytes, hipStream_t stream) {
    const Plan pl = make_plan(p);
    if (ws == nullptr || ws_bytes < pl.ws_bytes) return hipErrorInvalidValue;
    // unit positions times workgroup counts stay far inside int64
    if ((double)pl.n_blocks * pl.n_tiles * (pl.per_xcd + 1) > 4.0e18) return hipErrorInvalidValue;
    Sched sc;
    sc.n_xcd = pl.n_xcd;
    sc.per_xcd = pl.per_xcd;
    sc.n_tiles = pl.n_tiles;
    sc.nqb = pl.nqb;
    sc.n_blocks = pl.n_blocks;
    sc.whole = pl.whole;
    sc.xcc_of = (int*)((char*)ws + pl.off_xcc);
    sc.counters = (int*)((char*)ws + pl.off_counters);
    sc.part_o = (float*)((char*)ws + pl.off_o);
    sc.part_ml = (float*)((char*)ws + pl.off_ml);
    attn_bf16_kernel<<<pl.grid, NTHREADS, 0, stream>>>(p, sc);
    return hipGetLastError();
}

}  // namespace pcpp
