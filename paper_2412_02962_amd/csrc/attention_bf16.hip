// Partially conditioned self-attention, bf16 storage, on gfx950 MFMA.
//
// Computes, per image and head, softmax(Q K_ctx^T / sqrt(64)) V_ctx where
// the key/value context is the band's fresh tokens plus the stale boundary
// rows of its neighbours (Sec. 3.3 and Eq. 1 of arXiv 2412.02962).  The three
// key/value sources are read in place (no assembled copy): a 64-key tile that
// lies inside one source is fetched from that source's base; a tile that
// straddles two sources (or the end) picks the source row by row.
//
// Work decomposition.  A block is 128 queries of one (image, head); its key
// tiles are cut into k equal pieces and a workgroup computes one piece of one
// block.  Two workgroups share a compute unit (two wavefronts per SIMD, from
// different workgroups, so that their tile barriers are independent), so a
// launch runs in waves of twice as many workgroups as there are compute
// units; k is chosen by a cost estimate (waves x (tiles per piece + a fixed
// cost per piece)): at the 2048 px level-1 shape k = 3 (480 workgroups, one
// wave); larger shapes take several waves of smaller pieces instead of a
// ragged last wave of whole blocks.  The blocks are dealt out to the XCDs in
// contiguous ranges and all pieces of a block run on one XCD: workgroup w
// runs on XCD w % n_xcd (the hardware deals workgroups out round-robin), so
// the pieces of a block are merged through that XCD's L2 with ordinary
// stores and one counter per block (the last piece to arrive merges and
// resets the counter to zero).  Pieces of the blocks of one head start on
// the same key tiles, so their tiles are fetched from HBM once and then hit
// in the L2.
//
// Inside a workgroup the four wavefronts (one per SIMD) own 32 queries each
// and walk the same key tiles, staged once per workgroup in LDS by direct
// global->LDS loads into four K and four V slots (tile t+3's keys and tile
// t+2's values load while tile t is computed; one barrier per tile).  Tiles
// that lie inside one key source (the usual case) are addressed with scalar
// arithmetic only: a wave-uniform 64-bit base and the per-lane offsets of
// the load's saddr form.

// Software pipeline over 32-key half-tiles h.  Step h holds S(h) (scores of
// half h) and P(h-1) (bf16 probabilities of half h-1) in registers and
// interleaves, one matrix product at a time, the VALU softmax of S(h) with
// the 8 MFMA 32x32x16 of O^T += V(h-1)^T P(h-1)^T and S(h+1)^T = K(h+1) Q^T;
// the LDS operands of step h+1 are read during step h.
//   S^T = K Q^T      K from LDS, Q^T in registers.  The transposed product
//                    leaves each lane with one query and 16 keys of the
//                    half: a row max needs one exchange with the partner
//                    lane (lane ^ 32), the row sum none.
//   online softmax   in log2 units, p = exp2(s*log2(e)/8 - m) against the
//                    running max m; the half's max is only taken (and m
//                    raised, O and l rescaled) when a lane's probabilities
//                    of the half sum to 2^20 or more, so p < 2^20.
//   O^T += V^T P^T   P^T is the B operand taken straight from the S^T
//                    accumulators (inside each 16-key step the key order is
//                    permuted the same way on both operands); V^T comes from
//                    the row-major V tile through the transposing LDS read
//                    ds_read_b64_tr_b16.
// Row sums accumulate the bf16 probabilities with v_dot2 against (1, 1), so
// numerator and denominator see the same rounded weights.

#include <math.h>

#include "common.h"
#include "kernels.h"

namespace pcpp {

namespace {

constexpr int D = 64;
constexpr int KT = 64;                      // keys per tile
constexpr int QW = 32;                      // queries per wavefront
constexpr int NW = 4;                       // wavefronts per workgroup (one per SIMD)
constexpr int QB = QW * NW;                 // queries per block
constexpr int NTHREADS = 64 * NW;
constexpr int WG_PER_CU = 8 / NW;           // two workgroups per compute unit: two wavefronts per SIMD
constexpr int TILE_BYTES = KT * D * 2;      // 8 KB of K or of V
constexpr int SLOTS = 4;                    // LDS slots for K tiles, and for V tiles
constexpr int V_REGION = SLOTS * TILE_BYTES;
constexpr float P_LIMIT = 1048576.0f;       // 2^20: bound on a lane's probability sum per half-tile
constexpr int MIN_TILES_PER_PIECE = 3;

constexpr int PIECES = TILE_BYTES / 1024 / NW;  // 1 KB pieces of a tile each wavefront stages
static_assert(WG_PER_CU * 2 * V_REGION + 64 <= 160 * 1024, "the workgroups of a compute unit share its LDS");
static_assert(PIECES >= 1 && PIECES * NW * 1024 == TILE_BYTES, "the wavefronts stage whole 1 KB pieces of a tile");

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef const __attribute__((address_space(1))) void* gptr_t;
typedef __attribute__((address_space(3))) void* lptr_t;

// 16 bytes per lane from global memory straight into LDS: lane l's bytes land
// at lds + 16 l (lds is the wave-uniform LDS byte address).  Written as inline
// assembly so that the compiler does not track the LDS write: its own tracking
// of such writes covers at most a few LDS buffers and otherwise waits for every
// staging load in flight before any LDS read.  The kernel orders these writes
// before the reads itself, with vmcnt waits and barriers.  Loads complete in
// order, so the compiler's own vmcnt waits for register loads stay safe: they
// only become more conservative.
__device__ __forceinline__ void dma16(const void* g, const char* lds) {
    const uint32_t a = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lptr_t)lds);
    asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "{m0}"(a) : "memory");
}

// The same with a wave-uniform 64-bit base in SGPRs and a 32-bit per-lane
// byte offset (the load's saddr form): no per-lane address arithmetic.
// lds is the wave-uniform LDS byte address.
__device__ __forceinline__ void dma16_s(uint64_t base, uint32_t voff, uint32_t lds) {
    asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(base), "{m0}"(lds) : "memory");
}

// A wave-uniform value known to the compiler as such (kept in SGPRs).
__device__ __forceinline__ uint64_t uniform64(uint64_t x) {
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(x >> 32));
    return ((uint64_t)hi << 32) | lo;
}

// LDS swizzles: 16-byte chunk c of tile row r is stored at slot c ^ mask(r).
// K rows are read 16 bytes per lane by 32 consecutive rows at one chunk; V
// rows by four rows x 32 bytes per 16 lanes (transposing read).  Both masks
// repeat every 16 rows, so a half-tile (32 rows) offset keeps them.
__device__ __forceinline__ int k_mask(int r) { return (r >> 1) & 7; }
__device__ __forceinline__ int v_mask(int r) { return ((r >> 1) & 3) << 1; }

struct Sched {
    int32_t n_xcd;      // XCDs; workgroup w runs on XCD w % n_xcd
    int32_t bpx;        // blocks per XCD (the last XCD may hold fewer)
    int32_t k;          // pieces per block
    int32_t n_tiles;    // key tiles per block
    int32_t nqb;        // blocks per (image, head)
    int32_t n_blocks;   // blocks in total
    int* counters;      // [n_blocks]: zero at launch, left zero (split launches only)
    float* part_o;      // [grid][QB * D] partial outputs of pieces
    float* part_ml;     // [grid][QB][2] their row statistics
};

__device__ __forceinline__ int64_t pick(int j, int end0, int end1, int64_t a0, int64_t a1, int64_t a2) {
    const int64_t a12 = j < end1 ? a1 : a2;
    return j < end0 ? a0 : a12;
}

// LDS operands of one pipeline step: K of a half-tile (four 16-byte chunks
// per lane) and V^T of a half-tile (32-dim block mb, 16-key step st).
struct Operands {
    bf16x8 k[4];
    bf16x8 v[2][2];  // [mb][st]
};

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// Two transposing reads (rows p and p + 8 of a V tile) form one V^T operand.
__device__ __forceinline__ bf16x8 read_vt(const char* p) {
    const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)p);
    const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p + 1024));
    const short __attribute__((ext_vector_type(8))) w = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_bit_cast(bf16x8, w);
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

#define SCHED_FENCE() __builtin_amdgcn_sched_barrier(0)

__global__ __launch_bounds__(NTHREADS, WG_PER_CU) void attn_bf16_kernel(AttnParams p, Sched sc) {
    // Three K and three V slots, each its own object: a direct-to-LDS load
    // in flight into one slot is then known not to touch the others, and the
    // compiler orders LDS reads of the other slots freely.
    __shared__ __attribute__((aligned(16))) char ks0[TILE_BYTES];
    __shared__ __attribute__((aligned(16))) char ks1[TILE_BYTES];
    __shared__ __attribute__((aligned(16))) char ks2[TILE_BYTES];
    __shared__ __attribute__((aligned(16))) char ks3[TILE_BYTES];
    __shared__ __attribute__((aligned(16))) char vs0[TILE_BYTES];
    __shared__ __attribute__((aligned(16))) char vs1[TILE_BYTES];
    __shared__ __attribute__((aligned(16))) char vs2[TILE_BYTES];
    __shared__ __attribute__((aligned(16))) char vs3[TILE_BYTES];
    __shared__ int flag_lds;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
    const int col = lane & 31;
    const int half = lane >> 5;
    const int C = p.C;
    const int kv_end = p.kv.n_kv;
    const int end0 = p.kv.end0, end1 = p.kv.end1;
    const float sl2 = p.scale_log2;
    // (1, 1) in a register the compiler cannot see through: the row-sum dots
    // then take it as an operand, and the first dot of a half can take the
    // inline constant 0 as its addend instead of a register cleared by a move.
    bf16x2 ones = {(bf16)1.0f, (bf16)1.0f};
    {
        uint32_t ou = __builtin_bit_cast(uint32_t, ones);
        asm volatile("" : "+v"(ou));
        ones = __builtin_bit_cast(bf16x2, ou);
    }
    const int n_tiles = sc.n_tiles;

    const int x = blockIdx.x % sc.n_xcd;
    const int j = blockIdx.x / sc.n_xcd;
    const int bl = j / sc.k;            // block, XCD-local
    const int piece = j - bl * sc.k;
    const int blk = x * sc.bpx + bl;
    if (bl >= sc.bpx || blk >= sc.n_blocks) return;  // idle slot of the last XCD (uniform)
    const int t0 = (int)((int64_t)n_tiles * piece / sc.k);
    const int t1 = (int)((int64_t)n_tiles * (piece + 1) / sc.k);

    // Staging geometry: wavefront w fills the 1 KB pieces 2w and 2w+1 of a
    // tile (rows 8*piece .. +8); lane l fills LDS slot l & 7 of row
    // 8*piece + (l >> 3) with the global chunk the swizzle puts there.
    int ld_row[PIECES];
    uint32_t ld_koff[PIECES], ld_voff[PIECES];
#pragma unroll
    for (int i = 0; i < PIECES; ++i) {
        const int r = 8 * (PIECES * wave + i) + (lane >> 3);
        ld_row[i] = r;
        ld_koff[i] = (uint32_t)(r * C * 2 + (((lane & 7) ^ k_mask(r)) << 4));
        ld_voff[i] = (uint32_t)(r * C * 2 + (((lane & 7) ^ v_mask(r)) << 4));
    }

    // K operand reads (within a half-tile of a K slot): row col, chunks
    // 2*kk + half at their swizzled slots.
    int k_rel[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) k_rel[kk] = col * 128 + (((2 * kk + half) ^ k_mask(col)) << 4);
    // Transposing V reads (within a half-tile of a V slot), per 32-dim block
    // mb and 16-key step st.
    int v_rel[2];
    {
        const int jj = lane & 15;
        const int tr_row = 4 * half + (jj >> 2);
        const int tr_e = 16 * ((lane >> 4) & 1) + 4 * (jj & 3);
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) {
            const int e = 32 * mb + tr_e;
            v_rel[mb] = tr_row * 128 + (((e >> 3) ^ v_mask(tr_row)) << 4) + ((e & 7) << 1);
        }
    }
    // Operands of key half kb of the tile in slot kt, and of value half vb
    // of the tile in slot vt.
    auto read_step = [&](const char* kt, int kb, const char* vt, int vb, Operands& o) {
        const char* kh = kt + kb * (TILE_BYTES / 2);
        const char* vh = vt + vb * (TILE_BYTES / 2);
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) o.k[kk] = *(const bf16x8*)(kh + k_rel[kk]);
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int st = 0; st < 2; ++st) o.v[mb][st] = read_vt(vh + v_rel[mb] + st * 2048);
    };

    {
        const int qb = blk % sc.nqb;
        const int bh = blk / sc.nqb;
        const int head = bh % p.heads;
        const int b = bh / p.heads;
        const int head_off = head * D;

        // Source bases (bytes), pre-offset so that key row j of a segment is base + j*C*2.
        const int64_t o0 = (int64_t)b * p.kv.bstride[0] + head_off;
        const int64_t o1 = (int64_t)b * p.kv.bstride[1] - (int64_t)end0 * C + head_off;
        const int64_t o2 = (int64_t)b * p.kv.bstride[2] - (int64_t)end1 * C + head_off;
        const int64_t ka0 = (int64_t)(uintptr_t)p.kv.k[0] + o0 * 2;
        const int64_t ka1 = (int64_t)(uintptr_t)p.kv.k[1] + o1 * 2;
        const int64_t ka2 = (int64_t)(uintptr_t)p.kv.k[2] + o2 * 2;
        const int64_t va0 = (int64_t)(uintptr_t)p.kv.v[0] + o0 * 2;
        const int64_t va1 = (int64_t)(uintptr_t)p.kv.v[1] + o1 * 2;
        const int64_t va2 = (int64_t)(uintptr_t)p.kv.v[2] + o2 * 2;

        // Sources whose boundaries fall on tile boundaries (the usual case:
        // W * rows a multiple of 64) take every tile from one source, picked
        // by comparing the tile index with two precomputed tile numbers and
        // addressed with scalar arithmetic only.
        const bool aligned = end0 % KT == 0 && end1 % KT == 0 && kv_end % KT == 0;
        const int tb0 = end0 / KT, tb1 = end1 / KT;
        const uint32_t tile_g = (uint32_t)(KT * C * 2);  // bytes between consecutive tiles of a source (C <= 2^20 / 64)
        const uint64_t sk0 = uniform64((uint64_t)ka0), sk1 = uniform64((uint64_t)ka1), sk2 = uniform64((uint64_t)ka2);
        const uint64_t sv0 = uniform64((uint64_t)va0), sv1 = uniform64((uint64_t)va1), sv2 = uniform64((uint64_t)va2);
        // LDS byte addresses of the slots' parts this wavefront stages.
        auto lds_of = [&](const char* slot) {
            return (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lptr_t)slot) +
                   (uint32_t)(PIECES * wave * 1024);
        };

        // Stage tile t of K (is_v = false) or V into the slot at dst.
        auto issue = [&](int t_in, char* slot, bool is_v) {
            const int t = __builtin_amdgcn_readfirstlane(t_in);
            char* dst = slot + PIECES * wave * 1024;
            const uint32_t* off = is_v ? ld_voff : ld_koff;
            if (aligned) {
                const uint64_t a0 = is_v ? sv0 : sk0, a1 = is_v ? sv1 : sk1, a2 = is_v ? sv2 : sk2;
                const uint64_t src = t < tb0 ? a0 : (t < tb1 ? a1 : a2);
                const uint64_t base = src + (uint64_t)(uint32_t)t * tile_g;
                const uint32_t lds = lds_of(slot);
#pragma unroll
                for (int i = 0; i < PIECES; ++i) dma16_s(base, off[i], lds + i * 1024);
                return;
            }
            const int j0 = t * KT, j1 = j0 + KT;
            const bool one_src = j1 <= kv_end && (j1 <= end0 || j0 >= end0) && (j1 <= end1 || j0 >= end1);
            if (one_src) {
                const int64_t base = (is_v ? pick(j0, end0, end1, va0, va1, va2) : pick(j0, end0, end1, ka0, ka1, ka2)) +
                                     (int64_t)j0 * C * 2;
#pragma unroll
                for (int i = 0; i < PIECES; ++i)
                    dma16((const char*)(uintptr_t)base + off[i], dst + i * 1024);
                return;
            }
#pragma unroll
            for (int i = 0; i < PIECES; ++i) {
                int jk = j0 + ld_row[i];
                jk = jk < kv_end ? jk : kv_end - 1;
                const int64_t base = (is_v ? pick(jk, end0, end1, va0, va1, va2) : pick(jk, end0, end1, ka0, ka1, ka2)) +
                                     ((int64_t)jk - ld_row[i]) * C * 2;
                dma16((const char*)(uintptr_t)base + off[i], dst + i * 1024);
            }
        };

        // Prologue: K of tiles t0 and t0+1 and V of tile t0, then Q^T.
        issue(t0, ks0, false);
        issue(t0, vs0, true);
        if (t0 + 1 < t1) issue(t0 + 1, ks1, false);
        // Q^T operands of the wavefront's 32 queries.
        const int q_base = qb * QB + QW * wave;
        bf16x8 qop[4];
        {
            const int qrow = min(q_base + col, p.nq - 1);
            const bf16* qp = (const bf16*)p.q + (int64_t)b * p.q_bstride + (int64_t)qrow * C + head_off + 8 * half;
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) qop[kk] = *(const bf16x8*)(qp + 16 * kk);
        }

        f32x16 o[2];
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int r = 0; r < 16; ++r) o[mb][r] = 0.f;
        // Running max (log2 units) and the lane's share of the row sum.
        float m_run = -INFINITY, l_run = 0.f;

        // Mask the scores of half-tile h past the last key.
        auto mask_half = [&](int h, f32x16& sv) {
            if ((h >> 1) * KT + KT > kv_end) {
                // (hidden from the compiler, which otherwise computes the
                // lane's key offset before the branch, in every half-tile)
                int hl = 4 * half;
                asm volatile("" : "+v"(hl));
#pragma unroll
                for (int rr = 0; rr < 16; ++rr) {
                    const int jk = (h >> 1) * KT + 32 * (h & 1) + 8 * (rr >> 2) + hl + (rr & 3);
                    if (jk >= kv_end) sv[rr] = -INFINITY;
                }
            }
        };

        __builtin_amdgcn_s_waitcnt(0xF70);  // vmcnt(0): this thread's staging loads and Q have landed
        __builtin_amdgcn_s_barrier();
        // K of tile t0+2 and V of tile t0+1 load during the first period.
        if (t0 + 2 < t1) issue(t0 + 2, ks2, false);
        if (t0 + 1 < t1) issue(t0 + 1, vs1, true);

        // S(2 t0) from key half 0 of tile t0; operands of step 2 t0: key half
        // 1 of tile t0 and, standing in for the absent half 2 t0 - 1, value
        // half 0 of tile t0 (multiplied by all-zero probabilities).
        f32x16 s_a, s_b;
        Operands op_a, op_b;
        {
            Operands o0;
            read_step(ks0, 0, vs0, 0, o0);
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) s_a = mfma32x32x16(o0.k[kk], qop[kk], kk == 0 ? f32x16{} : s_a);
            mask_half(2 * t0, s_a);
        }
        read_step(ks0, 1, vs0, 0, op_a);
        bf16x8 p_a[2], p_b[2];
#pragma unroll
        for (int st = 0; st < 2; ++st)
#pragma unroll
            for (int e = 0; e < 8; ++e) p_b[st][e] = (bf16)0.0f;

        // One pipeline step h: softmax of s_cur -> p_cur, interleaved with
        // O^T += V(h-1)^T p_prev^T and s_nxt = K(h+1) Q^T from op_cur; the
        // operands of step h+1 are read into op_nxt first.
        auto step = [&](int h, f32x16& s_cur, f32x16& s_nxt, bf16x8 (&p_prev)[2], bf16x8 (&p_cur)[2],
                        Operands& op_cur, Operands& op_nxt, const char* nk, int nk_half, const char* nv, int nv_half) {
            SCHED_FENCE();
            float acc0 = 0.f;
            float mneg = -m_run;
            // probabilities of elements 2i, 2i+1 and their bf16 sum (one chain
            // of dots in pair order)
            auto pair = [&](int i) {
                const float e0 = fast_exp2(fmaf(s_cur[2 * i], sl2, mneg));
                const float e1 = fast_exp2(fmaf(s_cur[2 * i + 1], sl2, mneg));
                const bf16x2 pk = {f32_to_bf16(e0), f32_to_bf16(e1)};
                p_cur[i >> 2][2 * (i & 3)] = pk[0];
                p_cur[i >> 2][2 * (i & 3) + 1] = pk[1];
                if (i == 0) {
                    // the first pair starts the chain with the inline constant 0 as addend
                    asm("v_dot2_f32_bf16 %0, %1, %2, 0"
                        : "=v"(acc0)
                        : "v"(__builtin_bit_cast(uint32_t, pk)), "v"(__builtin_bit_cast(uint32_t, ones)));
                } else {
                    acc0 = __builtin_amdgcn_fdot2_f32_bf16(pk, ones, acc0, false);
                }
            };
            SCHED_FENCE();
            pair(0);
            pair(1);
            SCHED_FENCE();
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int st = i >> 2, mb = (i >> 1) & 1;
                if ((i & 1) == 0) {
                    o[mb] = mfma32x32x16(op_cur.v[mb][st], p_prev[st], o[mb]);
                } else {
                    const int kk = i >> 1;
                    s_nxt = mfma32x32x16(op_cur.k[kk], qop[kk], kk == 0 ? f32x16{} : s_nxt);
                }
                SCHED_FENCE();
                // The operand that product i of the next step uses, read a
                // whole step ahead; one or two LDS reads per product keep
                // the LDS queue from filling up.
                if ((i & 1) == 0) {
                    const int nst = i >> 2, nmb = (i >> 1) & 1;
                    op_nxt.v[nmb][nst] = read_vt(nv + nv_half * (TILE_BYTES / 2) + v_rel[nmb] + nst * 2048);
                } else {
                    const int nkk = i >> 1;
                    op_nxt.k[nkk] = *(const bf16x8*)(nk + nk_half * (TILE_BYTES / 2) + k_rel[nkk]);
                }
                if (i < 6) pair(i + 2);
                SCHED_FENCE();
            }
            float lt = acc0;
            if (__any(!(lt < P_LIMIT))) {
                // Only when a lane's 16 probabilities of the half sum to 2^20
                // or more (or to inf / NaN: the first half, where m is -inf)
                // is the half's max taken, m raised to it, O and l rescaled
                // and the probabilities recomputed.
                float m4[4];
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    m4[i] = fmaxf(fmaxf(s_cur[4 * i], s_cur[4 * i + 1]), fmaxf(s_cur[4 * i + 2], s_cur[4 * i + 3]));
                const float mx = max_xor32(fmaxf(fmaxf(m4[0], m4[1]), fmaxf(m4[2], m4[3]))) * sl2;
                const float m_new = fmaxf(m_run, mx);
                const float alpha = fast_exp2(m_run - m_new);
                m_run = m_new;
                mneg = -m_new;
                l_run *= alpha;
#pragma unroll
                for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                    for (int rr = 0; rr < 16; ++rr) o[mb][rr] *= alpha;
#pragma unroll
                for (int i = 0; i < 8; ++i) pair(i);
                lt = acc0;
            }
            l_run += lt;
            mask_half(h + 1, s_nxt);
        };

        // Period of tile pt: its two halves.  Slots: K(pt) in kc, K(pt+1) in
        // kn, V(pt) in vc; K(pt+3) and V(pt+2) are staged into kl and vl, so
        // every tile has two periods to arrive.
        auto period = [&](int pt, char* kc, char* kn, char* kl, char* vc, char* vl) {
            // Two wavefronts (one of each workgroup on the compute unit)
            // share each SIMD; issue favours the older one at equal
            // priority.  Raising the priority for the first half-tile and
            // dropping it for the second lets the one behind catch up.
            __builtin_amdgcn_s_setprio(1);
            if (pt > t0) {
                // The previous period staged K(pt+2) (if it exists) and
                // V(pt+1) (if it exists), PIECES loads per thread each; the
                // loads before them, K(pt+1) and V(pt) among them, must land.
                if (pt + 2 < t1)
                    __builtin_amdgcn_s_waitcnt(0xF70 | (2 * PIECES));
                else if (pt + 1 < t1)
                    __builtin_amdgcn_s_waitcnt(0xF70 | PIECES);
                else
                    __builtin_amdgcn_s_waitcnt(0xF70);
                // Everyone's loads have landed and nobody reads the slots of
                // K(pt-1) and V(pt-2) any more.  A bare barrier: a fence would
                // also wait for the loads still in flight.
                __builtin_amdgcn_s_barrier();
            }
            if (pt + 3 < t1) issue(pt + 3, kl, false);
            if (pt + 2 < t1) issue(pt + 2, vl, true);
            // Keys of tile pt+1.  Past the end the slot holds stale bytes that
            // no load is writing; their products are never used.  (A select
            // between slots here would hide from the compiler which slot is
            // read, and it would then wait for every staging load in flight.)
            step(2 * pt, s_a, s_b, p_b, p_a, op_a, op_b, kn, 0, vc, 0);
            __builtin_amdgcn_s_setprio(0);
            step(2 * pt + 1, s_b, s_a, p_a, p_b, op_b, op_a, kn, 1, vc, 1);
        };
        for (int pt = t0; pt < t1; pt += 4) {
            period(pt, ks0, ks1, ks3, vs0, vs2);
            if (pt + 1 < t1) period(pt + 1, ks1, ks2, ks0, vs1, vs3);
            if (pt + 2 < t1) period(pt + 2, ks2, ks3, ks1, vs2, vs0);
            if (pt + 3 < t1) period(pt + 3, ks3, ks0, ks2, vs3, vs1);
        }
        // Drain: O^T += V(2 t1 - 1)^T P(2 t1 - 1)^T, operands in op_a.
#pragma unroll
        for (int st = 0; st < 2; ++st)
#pragma unroll
            for (int mb = 0; mb < 2; ++mb) o[mb] = mfma32x32x16(op_a.v[mb][st], p_b[st], o[mb]);

        // ---- block epilogue ----
        const float l_tot = sum_xor32(l_run);
        const int q_out = q_base + col;
        bf16* out_row = (bf16*)p.out + (int64_t)b * p.q_bstride + (int64_t)min(q_out, p.nq - 1) * C + head_off + 4 * half;
        // Lane (col, half) holds dims 32*mb + 8*g + 4*half + {0..3} of query col in o[mb][4g..4g+3].
        auto store_out = [&](const f32x16 (&a)[2], float scale) {
            if (q_out >= p.nq) return;
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    bf16x4 v;
#pragma unroll
                    for (int e = 0; e < 4; ++e) v[e] = f32_to_bf16(a[mb][4 * g + e] * scale);
                    *(bf16x4*)(out_row + 32 * mb + 8 * g) = v;
                }
        };

        if (sc.k == 1) {
            store_out(o, l_tot > 0.f ? 1.0f / l_tot : 0.f);
            return;
        }
        // A piece of a block whose other pieces run on this XCD: store the
        // unnormalised O^T accumulators and (m, l), lane-major, then count.
        {
            float* po = sc.part_o + (int64_t)blockIdx.x * (QB * D) + wave * (QW * D) + lane * 4;
#pragma unroll
            for (int c = 0; c < 8; ++c) {
                const int mb = c >> 2, g = c & 3;
                const f32x4 v = {o[mb][4 * g], o[mb][4 * g + 1], o[mb][4 * g + 2], o[mb][4 * g + 3]};
                *(f32x4*)(po + c * 256) = v;
            }
            if (half == 0) {
                float* pml = sc.part_ml + ((int64_t)blockIdx.x * QB + QW * wave + col) * 2;
                pml[0] = m_run;
                pml[1] = l_tot;
            }
        }
        __builtin_amdgcn_s_waitcnt(0xF70);  // vmcnt(0): this thread's stores reached the L2
        __syncthreads();
        if (tid == 0) {
            int* counter = sc.counters + blk;
            const int prev = __hip_atomic_fetch_add(counter, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            const int last = prev == sc.k - 1;
            if (last) __hip_atomic_store(counter, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            flag_lds = last;
        }
        __syncthreads();
        if (!flag_lds) return;
        // Last piece: combine all k pieces in piece order (this one from
        // registers, the others from the workspace) with a running max, one
        // code path for every piece, so the result does not depend on which
        // piece arrived last.  The next piece's loads are issued before the
        // current one is combined.
        float M = -INFINITY, L = 0.f;
        f32x16 res[2];
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int r = 0; r < 16; ++r) res[mb][r] = 0.f;
        auto load_piece = [&](int pi, f32x16 (&pc)[2], float& mk, float& lk) {
            const int w = (bl * sc.k + pi) * sc.n_xcd + x;
            if (w == (int)blockIdx.x) {
                pc[0] = o[0];
                pc[1] = o[1];
                mk = m_run;
                lk = l_tot;
                return;
            }
            const float* pml = sc.part_ml + ((int64_t)w * QB + QW * wave + col) * 2;
            mk = pml[0];
            lk = pml[1];
            const float* pk = sc.part_o + (int64_t)w * (QB * D) + wave * (QW * D) + lane * 4;
#pragma unroll
            for (int c = 0; c < 8; ++c) {
                const f32x4 v = *(const f32x4*)(pk + c * 256);
#pragma unroll
                for (int e = 0; e < 4; ++e) pc[c >> 2][4 * (c & 3) + e] = v[e];
            }
        };
        f32x16 pc_a[2], pc_b[2];
        float m_a, l_a, m_b, l_b;
        auto combine = [&](const f32x16 (&pc)[2], float mk, float lk) {
            const float Mn = fmaxf(M, mk);
            const float a = fast_exp2(M - Mn);
            const float w = fast_exp2(mk - Mn);
            L = __builtin_fmaf(lk, w, L * a);
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int r = 0; r < 16; ++r) res[mb][r] = __builtin_fmaf(pc[mb][r], w, res[mb][r] * a);
            M = Mn;
        };
        load_piece(0, pc_a, m_a, l_a);
        for (int pi = 0; pi < sc.k; pi += 2) {
            if (pi + 1 < sc.k) load_piece(pi + 1, pc_b, m_b, l_b);
            combine(pc_a, m_a, l_a);
            if (pi + 1 < sc.k) {
                if (pi + 2 < sc.k) load_piece(pi + 2, pc_a, m_a, l_a);
                combine(pc_b, m_b, l_b);
            }
        }
        store_out(res, L > 0.f ? 1.0f / L : 0.f);
    }
}

struct Plan {
    int32_t n_xcd, bpx, k, grid, n_tiles, nqb, n_blocks;
    size_t off_counters, off_o, off_ml, ws_bytes;
    bool fits;
};

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Pieces per block, from a cost estimate; the k with the smallest estimate
// wins (the smallest such k on ties).  A launch of W workgroups runs in
// ceil(W / max_grid) waves (max_grid = two workgroups per compute unit).
//   Shapes whose whole blocks fit one wave (the 2048 px level-1 and level-2
//   bands): in hundredths of the time a tile takes when two workgroups share
//   a compute unit (1.09 us at level 1), a workgroup that has its compute
//   unit to itself (W <= compute units) runs a tile in 0.64 of that time, a
//   split costs about 2.6 tile times per wave (partial stores, counter,
//   merge), and a launch with compute units holding two workgroups about
//   1.8 more (measured on the level-2 bands at batch 1 and 2: 10 to 12 tiles,
//   80 or 160 blocks).
//   Larger shapes: waves x (tiles per piece + 4), in tile times; they take
//   several waves of smaller pieces rather than a ragged last wave of whole
//   blocks.
constexpr int64_t TILE_COST_SHARED = 100;
constexpr int64_t TILE_COST_ALONE = 64;
constexpr int64_t PIECE_COST = 257;
constexpr int64_t SHARED_CU_COST = 183;
constexpr int64_t PIECE_COST_TILES = 4;
constexpr int64_t MAX_SPLIT_BLOCKS = 65536;  // work counters kept at a fixed place

int64_t pick_k(int64_t slots, int64_t cus, int64_t n_tiles) {
    const int64_t max_grid = (int64_t)WG_PER_CU * cus;
    const int64_t k_max = n_tiles / MIN_TILES_PER_PIECE;
    const bool one_wave = slots <= max_grid;
    int64_t best_k = 1, best = -1;
    for (int64_t k = 1; k == 1 || (k <= k_max && k <= 64); ++k) {
        const int64_t w = slots * k;
        const int64_t waves = (w + max_grid - 1) / max_grid;
        const int64_t tiles = (n_tiles + k - 1) / k;
        int64_t cost;
        if (one_wave) {
            const bool alone = w <= cus;
            cost = waves * (tiles * (alone ? TILE_COST_ALONE : TILE_COST_SHARED) + (k > 1 ? PIECE_COST : 0)) +
                   (alone ? 0 : SHARED_CU_COST);
        } else {
            cost = waves * (tiles + PIECE_COST_TILES);
        }
        if (best < 0 || cost < best) {
            best = cost;
            best_k = k;
        }
    }
    return best_k;
}

// Workspace layout, independent of the geometry where it matters: [work
// counters: MAX_SPLIT_BLOCKS ints, always at offset 0, left zero by every
// call][partial outputs: one per workgroup][partial row statistics: same].
// The partial regions grow with the grid of a split launch; their contents
// need no clearing.  Pieces are merged only where the device layout says
// that workgroup w runs on XCD w % n_xcd; otherwise every workgroup
// computes whole blocks.
Plan make_plan(const AttnParams& p, const DeviceLayout& d) {
    Plan pl;
    pl.n_tiles = (p.kv.n_kv + KT - 1) / KT;
    pl.nqb = (p.nq + QB - 1) / QB;
    const int64_t n_blocks = (int64_t)p.batch * p.heads * pl.nqb;
    pl.n_blocks = (int32_t)(n_blocks < INT32_MAX ? n_blocks : INT32_MAX);
    pl.n_xcd = d.xcd_merge ? d.n_xcd : 1;
    const int64_t bpx = (n_blocks + pl.n_xcd - 1) / pl.n_xcd;
    int64_t k = 1;
    if (d.xcd_merge && n_blocks <= MAX_SPLIT_BLOCKS) k = pick_k(pl.n_xcd * bpx, d.cus, pl.n_tiles);
    pl.k = (int32_t)k;
    pl.bpx = (int32_t)(bpx < INT32_MAX ? bpx : INT32_MAX);
    const int64_t grid = (int64_t)pl.n_xcd * bpx * k;
    pl.grid = (int32_t)(grid < INT32_MAX ? grid : INT32_MAX);
    pl.fits = grid < INT32_MAX && n_blocks < INT32_MAX / 2;
    const size_t pieces = k > 1 ? (size_t)grid : 0;
    size_t off = 0;
    pl.off_counters = off;
    off += align256((size_t)MAX_SPLIT_BLOCKS * sizeof(int));
    pl.off_o = off;
    off += align256(pieces * QB * D * sizeof(float));
    pl.off_ml = off;
    off += align256(pieces * QB * 2 * sizeof(float));
    pl.ws_bytes = off;
    return pl;
}

}  // namespace

size_t attention_bf16_ws_bytes(const AttnParams& p) { return make_plan(p, device_layout_unmasked()).ws_bytes; }

size_t attention_bf16_counter_bytes() { return align256((size_t)MAX_SPLIT_BLOCKS * sizeof(int)); }

AttnPlanInfo attention_bf16_plan(const AttnParams& p, const DeviceLayout& d) {
    const Plan pl = make_plan(p, d);
    return AttnPlanInfo{QB, pl.k, pl.grid, pl.k > 1 ? pl.n_blocks : 0};
}

hipError_t launch_attention_bf16(const AttnParams& p, void* ws, size_t ws_bytes, hipStream_t stream) {
    const Plan pl = make_plan(p, device_layout(stream));
    if (ws == nullptr || ws_bytes < pl.ws_bytes) return hipErrorInvalidValue;
    if (!pl.fits) return hipErrorInvalidValue;
    Sched sc;
    sc.n_xcd = pl.n_xcd;
    sc.bpx = pl.bpx;
    sc.k = pl.k;
    sc.n_tiles = pl.n_tiles;
    sc.nqb = pl.nqb;
    sc.n_blocks = pl.n_blocks;
    sc.counters = (int*)((char*)ws + pl.off_counters);
    sc.part_o = (float*)((char*)ws + pl.off_o);
    sc.part_ml = (float*)((char*)ws + pl.off_ml);
    attn_bf16_kernel<<<pl.grid, NTHREADS, 0, stream>>>(p, sc);
    return hipGetLastError();
}

}  // namespace pcpp
