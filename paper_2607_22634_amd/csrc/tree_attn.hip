// Stage 3: tree-masked verification attention (one target layer).
//
// Every query row (node n, query head h) attends to the cached prefix of its
// sequence and to the tree nodes on its root path.  Rows are packed per KV
// head: row rho = n * G + (h - g * G), so one workgroup serves the G query
// heads that share KV head g and streams each K/V tile through LDS once for
// all of them.  The key sequence of sequence b is virtual: positions
// 0 .. ctx_b-1 read the packed cache, positions ctx_b .. ctx_b+n_nodes-1
// read the tree K/V and are masked by the ancestor bitmask.
//
// bf16 path (matrix cores, v_mfma_f32_32x32x16_bf16).  A workgroup is eight
// waves (two per SIMD), each owning 32 query rows.  Scores are computed
// transposed, S^T = K Q^T: a lane then holds one query row and 16 of the 32
// keys of a block, the row max needs one cross-half swap, and the bf16
// probabilities are already in the B-operand layout of O^T = V^T P^T.  K and
// V sit in LDS row-major (rows padded so that the b128 K reads and the
// transposed ds_read_b64_tr_b16 V reads are free of bank conflicts).  Three
// 64-key LDS buffers rotate: tile t is consumed, tile t+1 is resident (the
// last block of a tile already scores the first block of the next), tile t+2
// waits in registers; one barrier per tile.  Inside a wave the scores of
// block i+1 are issued ahead of the softmax and P V of block i, so the matrix
// cores can run while the vector ALUs work.  The running reference maximum
// only moves when a block exceeds it by a margin, which keeps the 64-register
// accumulator rescale off the common path.  The context is split across
// workgroups when the batch alone cannot fill the chip; each split leaves,
// per query row, its (reference, sum) pair and its output divided by its own
// sum (bf16), which a second kernel merges.
#include <math.h>

#include <type_traits>

#include "common.hpp"

namespace presto {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef short short4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float floatx2 __attribute__((ext_vector_type(2)));

// Two fp32 -> two bf16 (round to nearest even) in one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((floatx2){lo, hi}, bf16x2));
}

constexpr int kKeyTile = 64;      // keys per LDS tile: two 32-key blocks per barrier
constexpr int kBlocksPerTile = kKeyTile / 32;
constexpr int kRing = 4;          // LDS tile buffers: tile t consumed, t+1 resident, t+2 and t+3 in flight
constexpr int kMaxAncWords = 16;  // ancestor words per node: n_max <= 1024
constexpr int kRowsPerWave = 32;  // one 32-row MFMA block per wave
// Workgroups are 8 waves, two per SIMD, so that one wave's vector work runs
// while the other's MFMAs occupy the matrix core.
constexpr int kAttnWaves = 8;
constexpr int kAttnRows = kAttnWaves * kRowsPerWave;  // query rows per workgroup
constexpr float kLog2e = 1.4426950408889634f;

struct AttnArgs {
    const uint16_t* q;
    const uint16_t* kc;
    const uint16_t* vc;
    const int32_t* ctx_off;
    int32_t ctx_slots;  // 0: ctx_off is [batch + 1] offsets; 1: (start, len) pairs
    const uint16_t* kt;
    const uint16_t* vt;
    const uint64_t* anc;
    const int32_t* n_nodes;
    uint16_t* out;
    // split partials when splits > 1: the normalised output as bf16
    // [b, g, split, rho < G n_max, D] (a workgroup's rows are contiguous, so
    // its writes fill whole cache lines) and (m, l) fp32 [b, g, rho, split]
    uint16_t* part_o;
    float2* part_ml;
    int32_t batch, n_max, hq, hkv, G, W;
    int32_t row_tiles, rows_per_tile, splits, split_len;  // rows_per_tile: a multiple of 32, <= 256
    int32_t n_tasks, n_blocks;
    int32_t compact;  // tasks dealt over the (sequence, split) pairs that hold keys
    float scale_log2;  // scale * log2(e)
};

// Cache rows of sequence b: start c0 and length ctx, from packed offsets
// [batch + 1] or from (start, len) pairs [batch, 2].
struct CtxSpan {
    int c0, ctx;
};
__device__ __forceinline__ CtxSpan ctx_span(const int32_t* off, int b, int slots) {
    if (slots) return {off[2 * b], off[2 * b + 1]};
    return {off[b], off[b + 1] - off[b]};
}

__device__ __forceinline__ int clamp_nodes(int nn, int n_max) {
    return nn < 1 ? 1 : (nn > n_max ? n_max : nn);
}

// Blocks are dealt to the 8 XCDs round-robin; renumber them so that
// consecutive logical tasks (the row tiles of one KV range) share an XCD
// and its L2.
__device__ __forceinline__ int xcd_task(int bid, int n_blocks) {
    const int per = n_blocks >> 3;
    return (bid & 7) * per + (bid >> 3);
}

// LDS layout of the bf16 kernel (bytes).  A K tile is 64 key rows of D
// bf16 (D*2 bytes, no padding) with the 16-byte chunks of row r permuted by
// chunk ^ (r mod 16); a V tile likewise with chunk ^ 4(r mod 4).  The two
// permutations make the fragment reads free of bank conflicts (sixteen
// consecutive K rows read one chunk each: sixteen different chunks; the
// transposed V reads of four consecutive rows cover four disjoint 64-byte
// chunk groups), and since the global-to-LDS loads write 64 consecutive
// 16-byte chunks per instruction, the permutation is applied by choosing
// which global chunk each lane fetches.  K tiles of the ring sit in the
// first 64 KB and V tiles in the second, so that every fragment read is a
// per-lane base register plus an immediate offset.
// Global-to-LDS load of 16 bytes per lane (global_load_lds_dwordx4): lane
// l's bytes land at LDS address lds + 16 l (lds wave-uniform, in m0).  The
// instruction is issued from inline assembly so that the compiler does not
// guard every later LDS read with a wait for all outstanding loads; the
// kernel waits for each tile itself (vmcnt) before the barrier that
// publishes it.
__device__ __forceinline__ void lds_load16(const void* gptr, uint32_t lds) {
    asm volatile("global_load_lds_dwordx4 %0, off" ::"v"(gptr), "{m0}"(lds) : "memory");
}
// the same with a wave-uniform base and a per-lane 32-bit byte offset (the
// base and the LDS address are read from the first lane, so that they are
// scalar operands whatever registers the caller computed them in)
__device__ __forceinline__ void lds_load16(const void* base, uint32_t off, uint32_t lds) {
    const uint64_t b = (uint64_t)(uintptr_t)base;
    // readfirstlane returns a signed int: both halves go through uint32_t so
    // that the low half is zero-extended, not sign-extended, into the pointer
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)b);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
    const uint64_t sb = ((uint64_t)hi << 32) | (uint64_t)lo;
    const uint32_t m0v = (uint32_t)__builtin_amdgcn_readfirstlane(lds);
    asm volatile("global_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(sb), "{m0}"(m0v) : "memory");
}

template <int D>
struct AttnLds {
    static constexpr int kTile = kKeyTile * D * 2;           // bytes of one K (or V) tile
    static constexpr int kV = kRing * kTile;                 // start of the V tiles
};

template <int D>
__global__ __launch_bounds__(kAttnWaves * kWave) void tree_attn_bf16_kernel(AttnArgs a) {
    constexpr int KS = D / 16;                 // S^T contraction steps over the head dimension
    constexpr int DB = D / 32;                 // 32-wide blocks of the output head dimension
    constexpr int CH = D / 8;                  // 16-byte chunks per K/V row
    constexpr int NT = kAttnWaves * kWave;
    constexpr int ROWS = kAttnRows;
    // global-to-LDS loads per thread per tile, K and V each: 64 rows x CH
    // chunks, 64 chunks per instruction
    constexpr int LPT = kKeyTile * CH / 64 / kAttnWaves;
    constexpr int ROWS_PER_LOAD = 64 / CH;     // key rows covered by one load instruction
    static_assert(LPT >= 1 && LPT * kAttnWaves * 64 == kKeyTile * CH, "tile loads must divide evenly");
    static_assert(AttnLds<D>::kV + kRing * AttnLds<D>::kTile <= 65536 * 2, "ring must fit 128 KB");
    __shared__ __align__(16) char s_kv[2 * kRing * AttnLds<D>::kTile];
    // ancestor rows of this workgroup's nodes: at most ROWS nodes (G = 1)
    // of at most kMaxAncWords words; with the ring this is 160 KB at D = 128
    __shared__ uint64_t s_anc[ROWS * kMaxAncWords];

    int task, split, g, b;
    if (a.compact) {
        // task = ((pair * hkv) + g) * row_tiles + rt, pair = the index of
        // (sequence b, split) among the splits the sequences actually have,
        // in sequence order.  Every wave counts the pairs itself, then deals
        // the tasks over the XCDs as in the dense case, but over the tasks
        // that exist (the grid is an upper bound).
        const int lane0 = lane_id();
        auto splits_of = [&](int bb) {
            if (bb >= a.batch) return 0;
            const int kb = ctx_span(a.ctx_off, bb, a.ctx_slots).ctx + clamp_nodes(a.n_nodes[bb], a.n_max);
            return (kb + a.split_len - 1) / a.split_len;
        };
        int pairs = 0;
        for (int b0 = 0; b0 < a.batch; b0 += kWave) {
            const int incl = wave_prefix_sum_i32(splits_of(b0 + lane0));
            pairs += __builtin_amdgcn_readlane(incl, kWave - 1);
        }
        const int n_tasks = pairs * a.hkv * a.row_tiles;
        const int n_blocks = (n_tasks + 7) / 8 * 8;
        if ((int)blockIdx.x >= n_blocks) return;
        task = xcd_task(blockIdx.x, n_blocks);
        if (task >= n_tasks) return;
        g = (task / a.row_tiles) % a.hkv;
        const int item = task / a.row_tiles / a.hkv;
        b = -1;
        split = 0;
        int base = 0;
        for (int b0 = 0; b0 < a.batch; b0 += kWave) {
            const int ns = splits_of(b0 + lane0);
            const int incl = wave_prefix_sum_i32(ns);
            const uint64_t hit = __ballot(ns > 0 && item >= base + incl - ns && item < base + incl);
            if (hit) {
                const int l = __ffsll((unsigned long long)hit) - 1;
                b = b0 + l;
                // last split first (see below)
                split = __builtin_amdgcn_readlane(incl, l) - 1 - (item - base);
                break;
            }
            base += __builtin_amdgcn_readlane(incl, kWave - 1);
        }
        if (b < 0) return;
    } else {
        task = xcd_task(blockIdx.x, a.n_blocks);
        if (task >= a.n_tasks) return;
        // task = ((b * splits + split') * hkv + g) * row_tiles + rt with the
        // splits in reverse (split' = 0 is the last split): the XCDs start
        // their workgroups a few microseconds apart in XCD order, and the
        // last split, which holds the tree keys and their masks and so runs
        // longest, then lands on the XCDs that start first.
        g = (task / a.row_tiles) % a.hkv;
        split = a.splits - 1 - (task / a.row_tiles / a.hkv) % a.splits;
        b = task / a.row_tiles / a.hkv / a.splits;
    }
    const int rt = task % a.row_tiles;

    const CtxSpan cs = ctx_span(a.ctx_off, b, a.ctx_slots);
    const int c0 = cs.c0, ctx = cs.ctx;
    const int nn = clamp_nodes(a.n_nodes[b], a.n_max);
    const int keys = ctx + nn;
    const int k_begin = split * a.split_len;
    if (k_begin >= keys) return;  // nothing of this sequence in this split
    const int k_end = min(keys, k_begin + a.split_len);
    const int ntiles = (k_end - k_begin + kKeyTile - 1) / kKeyTile;
    const int nblocks = (k_end - k_begin + 31) / 32;
    const int live_rows = a.G * nn;
    const int all_rows = a.G * a.n_max;
    const int mask_from = min(ctx, k_end);  // keys at or beyond need a mask

    const int tid = threadIdx.x;
    const int wave = tid / kWave, lane = lane_id();
    const int l32 = lane & 31, h = lane >> 5;
    // Row blocks: wave w takes block w, except that when fewer than
    // kAttnWaves blocks hold live rows (A of them), the last one is shared by
    // waves A-1 .. kAttnWaves-1, each taking every nshare-th key block, and
    // their states are combined at the end: a 4-row tail block then costs a
    // SIMD a fraction of a full one.
    const int RT = a.rows_per_tile;
    const int tile_live = min(max(live_rows - rt * RT, 0), RT);
    const int A = (tile_live + kRowsPerWave - 1) / kRowsPerWave;
    const int nshare = (A >= 1 && A < kAttnWaves) ? kAttnWaves - A + 1 : 1;
    const bool shared = nshare > 1 && wave >= A - 1;
    const int sidx = shared ? wave - (A - 1) : 0;
    const int row0 = rt * RT + (shared ? A - 1 : wave) * kRowsPerWave;  // first query row of this wave
    const bool active = row0 < live_rows;
    const int rho = row0 + l32;  // this lane's query row
    const int qn = rho / a.G, qh = rho - qn * a.G;
    const int node = min(qn, a.n_max - 1);
    const float c = a.scale_log2;

    // Q fragments, B operand of S^T = K Q^T: lane holds row l32,
    // d = ks*16 + h*8 .. +8, pre-scaled by scale*log2(e) (rounded once to
    // bf16), so that the scores come out in log2 units.
    bf16x8 qf[KS];
    {
        const uint16_t* qp = a.q + (((int64_t)b * a.n_max + qn) * a.hq + g * a.G + qh) * D;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            uint4 u = make_uint4(0, 0, 0, 0);
            if (rho < all_rows) u = *reinterpret_cast<const uint4*>(qp + ks * 16 + h * 8);
            const uint32_t w[4] = {u.x, u.y, u.z, u.w};
            uint32_t r[4];
#pragma unroll
            for (int j = 0; j < 4; ++j)
                r[j] = pack_bf16x2(__uint_as_float(w[j] << 16) * c, __uint_as_float(w[j] & 0xffff0000u) * c);
            qf[ks] = __builtin_bit_cast(bf16x8, make_uint4(r[0], r[1], r[2], r[3]));
        }
    }
    // ancestor bitmask rows of the nodes this workgroup serves, when the
    // split reaches the tree keys (masks then read LDS, not global memory)
    const int n_first = (rt * RT) / a.G;
    if (k_end > ctx) {
        const int n_last = min((rt * RT + RT - 1) / a.G, a.n_max - 1);
        const int words = (n_last - n_first + 1) * a.W;
        const uint64_t* src = a.anc + ((int64_t)b * a.n_max + n_first) * a.W;
        for (int w = tid; w < words; w += NT) s_anc[w] = src[w];
    }

    // ---- K/V tiles: global -> LDS directly (global_load_lds_dwordx4), a
    // ring of kRing tiles.  Load instruction j of this wave covers key rows
    // ROWS_PER_LOAD * (wave * LPT + j) .. of the tile; lane l writes chunk
    // l % CH of row l / CH and so fetches the global chunk that the row's
    // permutation puts there.  The byte offsets of those chunks within a
    // tile that lies wholly in the cache are fixed for the whole loop.
    uint32_t goff_k[LPT], goff_v[LPT];
    int lrow[LPT], lck[LPT], lcv[LPT];
#pragma unroll
    for (int j = 0; j < LPT; ++j) {
        const int r = ROWS_PER_LOAD * (wave * LPT + j) + lane / CH;
        const int pc = lane % CH;
        lrow[j] = r;
        lck[j] = pc ^ (r & (CH - 1) & 15);
        lcv[j] = pc ^ ((4 * (r & 3)) & (CH - 1));
        goff_k[j] = (uint32_t)((r * a.hkv * D + lck[j] * 8) * 2);
        goff_v[j] = (uint32_t)((r * a.hkv * D + lcv[j] * 8) * 2);
    }
    const int fast_end = min(ctx, k_end);
    const int64_t tree_row0 = (int64_t)b * a.n_max;
    // all loads of the tile starting at key t0 into ring buffer `buf`
    const uint32_t lds_kv = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)s_kv;
    // the four base pointers as scalars: a per-lane choice between them is
    // then a register select, not a load from the argument block
    auto scalar_ptr = [](const uint16_t* ptr) {
        const uint64_t v = (uint64_t)(uintptr_t)ptr;
        const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
        const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
        return (const uint16_t*)(uintptr_t)(((uint64_t)hi << 32) | lo);
    };
    const uint16_t* const kc_s = scalar_ptr(a.kc);
    const uint16_t* const vc_s = scalar_ptr(a.vc);
    const uint16_t* const kt_s = scalar_ptr(a.kt);
    const uint16_t* const vt_s = scalar_ptr(a.vt);
    auto load_tile = [&](int t0, int buf) {
        const uint32_t kdst = lds_kv + buf * AttnLds<D>::kTile + wave * LPT * 1024;
        const uint32_t vdst = kdst + AttnLds<D>::kV;
        if (t0 + kKeyTile <= fast_end) {
            const int64_t row = ((int64_t)(c0 + t0) * a.hkv + g) * D;
            const uint16_t* kb = a.kc + row;
            const uint16_t* vb = a.vc + row;
#pragma unroll
            for (int j = 0; j < LPT; ++j) {
                lds_load16(kb, goff_k[j], kdst + j * 1024);
                lds_load16(vb, goff_v[j], vdst + j * 1024);
            }
        } else {
            // keys below ctx from the cache, the others from the tree K/V;
            // rows past k_end repeat the last key (their scores are masked)
#pragma unroll
            for (int j = 0; j < LPT; ++j) {
                const int kk = min(t0 + lrow[j], k_end - 1);
                const bool in_ctx = kk < ctx;
                const int64_t base = in_ctx ? ((int64_t)(c0 + kk) * a.hkv + g) * D
                                            : ((tree_row0 + (kk - ctx)) * a.hkv + g) * D;
                const uint16_t* kp = (in_ctx ? kc_s : kt_s) + base + lck[j] * 8;
                const uint16_t* vp = (in_ctx ? vc_s : vt_s) + base + lcv[j] * 8;
                lds_load16(kp, kdst + j * 1024);
                lds_load16(vp, vdst + j * 1024);
            }
        }
    };
    // vmcnt(n) with the other counters left alone (gfx9 encoding)
#define PRESTO_WAIT_VM(n) __builtin_amdgcn_s_waitcnt(((n) & 15) | (((n) >> 4) << 14) | 0x0f70)

    floatx16 o[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int i = 0; i < 16; ++i) o[db][i] = 0.f;

    // per-lane LDS byte addresses of the fragment reads (ring buffer 0,
    // block 0); buffer, block and step offsets are immediates
    constexpr uint32_t lds0 = 0;  // offsets from s_kv
    uint32_t kaddr[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
        kaddr[ks] = lds0 + l32 * (D * 2) + ((((2 * ks + h) ^ (l32 & 15)) & (CH - 1)) * 16);
    const int vr = 4 * h + ((lane & 15) >> 2);                  // row within an 8-row group
    const int vc = ((lane >> 4) & 1) * 2 + ((lane & 3) >> 1);   // chunk within a 4-chunk group
    uint32_t vaddr[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db)
        vaddr[db] = lds0 + AttnLds<D>::kV + vr * (D * 2) + (((4 * (db ^ (vr & 3))) + vc) & (CH - 1)) * 16 +
                    (lane & 1) * 8;

    auto row_max = [&](const floatx16& S) {
        float mx = S[0];
#pragma unroll
        for (int e = 1; e < 16; ++e) mx = fmaxf(mx, S[e]);
        const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx),
                                                         false, false);
        return fmaxf(mx, __uint_as_float(h == 0 ? sw[1] : sw[0]));
    };
    // Visibility of the block's 32 keys for this lane's row as one 32-bit
    // mask (bit t: key j0 + t): context keys, then the row's ancestor bits
    // from tree index j0 - ctx on, cut at the split's end; each element then
    // costs one bit test and one select.
    auto apply_mask = [&](floatx16& S, int j0) {
        const int s0 = j0 - ctx;  // tree index of the block's first key (< 0: it starts in the context)
        uint32_t anc = 0u;
        if (j0 + 32 > ctx) {
            const uint64_t* arow = &s_anc[(node - n_first) * a.W];
            if (s0 >= 0) {
                const int w = s0 >> 6, sh = s0 & 63;
                const uint64_t lo = arow[w];
                const uint64_t hi = w + 1 < a.W ? arow[w + 1] : 0ull;
                anc = (uint32_t)(sh == 0 ? lo : (lo >> sh) | (hi << (64 - sh)));
            } else {
                anc = (uint32_t)(arow[0] << (-s0));  // -s0 in 1 .. 31
            }
        }
        const int nctx = ctx - j0, nend = k_end - j0;
        const uint32_t ctx_mask = nctx >= 32 ? ~0u : (nctx <= 0 ? 0u : (1u << nctx) - 1u);
        const uint32_t end_mask = nend >= 32 ? ~0u : (nend <= 0 ? 0u : (1u << nend) - 1u);
        const uint32_t vis = ((ctx_mask | anc) & end_mask) >> (4 * h);
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const int t = 8 * (e >> 2) + (e & 3);  // element e is key j0 + 8(e/4) + 4h + e%4
            S[e] = ((vis >> t) & 1u) ? S[e] : -INFINITY;
        }
    };

    // ---- Key loop, pipelined over three key blocks so that the matrix
    // cores always have two independent chains and the vector ALUs work in
    // their shadow.  Step i issues, interleaved,
    //   * the P V MFMAs of block i (probabilities from step i-1),
    //   * the score MFMAs of block i+2 (its tile is resident),
    //   * the exponentials of block i+1 (scores from step i-1).
    // Every score chain starts from -m, so the MFMAs deliver x = s*c - m and
    // a probability costs one v_exp.  m is a lazy reference: no per-block
    // maximum is taken; a row whose block sum exceeds 2^8 (some x above
    // about 3) or that has no mass yet takes an exact step (block maximum,
    // rescale of o and l), which is rare.
    constexpr int EPK = 16 / KS;  // exponentials per score MFMA
    static_assert(EPK * KS == 16 && EPK % 2 == 0 && KS == 2 * DB, "head_dim 64 or 128");
    const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
    float m = 0.f, l_run = 0.f;  // lazy reference (log2 units) and row sum
    floatx16 negm;
#pragma unroll
    for (int e = 0; e < 16; ++e) negm[e] = 0.f;
    typedef __attribute__((address_space(3))) short4_t* lds_s4;
    // scores of block blk of ring buffer buf (compile-time) into Sx
    auto qk = [&](auto bufc, int blk, floatx16& Sx) {
        constexpr int buf = decltype(bufc)::value;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const uint4 u = *reinterpret_cast<const uint4*>(s_kv + kaddr[ks] + buf * AttnLds<D>::kTile +
                                                             blk * 32 * D * 2);
            Sx = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, u), qf[ks],
                                                         ks == 0 ? negm : Sx, 0, 0, 0);
        }
    };
    auto exps = [&](const floatx16& Sx, uint32_t (&Px)[8]) {
        float ls = 0.f;
#pragma unroll
        for (int e = 0; e < 16; e += 2) {
            Px[e >> 1] = pack_bf16x2(__builtin_amdgcn_exp2f(Sx[e]), __builtin_amdgcn_exp2f(Sx[e + 1]));
            ls = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, Px[e >> 1]), ones, ls, false);
        }
        return ls;
    };
    auto row_sum = [&](float v) {
        const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
        return v + __uint_as_float(h == 0 ? sw[1] : sw[0]);
    };
    // exact step for the rows that need it: move m to the block's maximum,
    // rescale the accumulated state and recompute the block's probabilities
    // (Sy: a block already scored against the old m, shifted along)
    auto exact = [&](floatx16& Sx, uint32_t (&Px)[8], float& ls, bool need, floatx16& Sy) {
        const float mx = row_max(Sx);
        const float delta = (need && mx != -INFINITY) ? mx : 0.f;
        const float alpha = l_run > 0.f ? __builtin_amdgcn_exp2f(-delta) : 0.f;
        m += delta;
        l_run *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db) o[db] *= alpha;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            Sx[e] -= delta;
            Sy[e] -= delta;
            negm[e] = -m;
        }
        ls = row_sum(exps(Sx, Px));
    };
    auto j0_of = [&](int i) { return k_begin + i * 32; };
    auto masked = [&](int i) { return j0_of(i) + 32 > mask_from; };

    floatx16 Sa = negm, Sb = negm;  // scores of blocks i+1 and i+2
    uint32_t Pp[8];                 // probabilities of block i
    // one block step: block i = 2 t + q; V of tile t in ring buffer bv, the
    // K of block i+2 (tile t+1) in ring buffer bk
    auto step = [&](auto bvc, auto bkc, int i, int q) {
        constexpr int bv = decltype(bvc)::value, bk = decltype(bkc)::value;
        const bool more = i + 1 < nblocks;
        if (more && masked(i + 1)) apply_mask(Sa, j0_of(i + 1));
        const int kblk = (i + 2) % kBlocksPerTile;
        uint32_t Pn[8];
        float ls = 0.f;
#pragma unroll
        for (int st = 0; st < 2; ++st) {
            const bf16x8 pb =
                __builtin_bit_cast(bf16x8, make_uint4(Pp[4 * st], Pp[4 * st + 1], Pp[4 * st + 2], Pp[4 * st + 3]));
#pragma unroll
            for (int db = 0; db < DB; ++db) {
                const uint32_t v0 = vaddr[db] + bv * AttnLds<D>::kTile + q * 32 * D * 2 + st * 16 * D * 2;
                const short4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4)(s_kv + v0));
                const short4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4)(s_kv + v0 + 8 * D * 2));
                const uint2 ul = __builtin_bit_cast(uint2, lo), uh = __builtin_bit_cast(uint2, hi);
                const bf16x8 va = __builtin_bit_cast(bf16x8, make_uint4(ul.x, ul.y, uh.x, uh.y));
                o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb, o[db], 0, 0, 0);
                const int ks = st * DB + db;
                const uint4 u = *reinterpret_cast<const uint4*>(s_kv + kaddr[ks] + bk * AttnLds<D>::kTile +
                                                                 kblk * 32 * D * 2);
                Sb = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, u), qf[ks],
                                                             ks == 0 ? negm : Sb, 0, 0, 0);
#pragma unroll
                for (int uu = 0; uu < EPK; uu += 2) {
                    const int e = ks * EPK + uu;
                    Pn[e >> 1] = pack_bf16x2(__builtin_amdgcn_exp2f(Sa[e]), __builtin_amdgcn_exp2f(Sa[e + 1]));
                    ls = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, Pn[e >> 1]), ones, ls, false);
                }
            }
        }
        if (more) {
            ls = row_sum(ls);
            const bool need = !(ls <= 256.f) || l_run + ls == 0.f;
            if (__ballot(need)) exact(Sa, Pn, ls, need, Sb);
            l_run += ls;
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) Pp[j] = Pn[j];
        Sa = Sb;
    };
    // P V of block q of ring buffer bv with the probabilities P
    auto pv = [&](auto bvc, int q, const uint32_t (&P)[8]) {
        constexpr int bv = decltype(bvc)::value;
#pragma unroll
        for (int st = 0; st < 2; ++st) {
            const bf16x8 pb =
                __builtin_bit_cast(bf16x8, make_uint4(P[4 * st], P[4 * st + 1], P[4 * st + 2], P[4 * st + 3]));
#pragma unroll
            for (int db = 0; db < DB; ++db) {
                const uint32_t v0 = vaddr[db] + bv * AttnLds<D>::kTile + q * 32 * D * 2 + st * 16 * D * 2;
                const short4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4)(s_kv + v0));
                const short4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4)(s_kv + v0 + 8 * D * 2));
                const uint2 ul = __builtin_bit_cast(uint2, lo), uh = __builtin_bit_cast(uint2, hi);
                const bf16x8 va = __builtin_bit_cast(bf16x8, make_uint4(ul.x, ul.y, uh.x, uh.y));
                o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb, o[db], 0, 0, 0);
            }
        }
    };
    // a shared block's wave: block i (block q of ring buffer bv) on its own,
    // scores, probabilities and P V in sequence (it takes every nshare-th
    // block only)
    auto shared_step = [&](auto bvc, int i, int q) {
        floatx16 S = negm;
        qk(bvc, q, S);
        if (masked(i)) apply_mask(S, j0_of(i));
        uint32_t P[8];
        float ls = row_sum(exps(S, P));
        const bool need = !(ls <= 256.f) || l_run + ls == 0.f;
        floatx16 none = S;
        if (__ballot(need)) exact(S, P, ls, need, none);
        l_run += ls;
        pv(bvc, q, P);
    };
    // one tile: its two block steps, then the load of tile t+3 into the
    // buffer of tile t-1 (every wave finished it before the last barrier),
    // and the wait for tile t+2 before the barrier
    auto tile = [&](auto uc, int t) {
        constexpr int u = decltype(uc)::value;
        using BV = std::integral_constant<int, u>;
        using BK = std::integral_constant<int, (u + 1) % kRing>;
        load_tile(k_begin + (t + 3) * kKeyTile, (u + 3) % kRing);
        if (active && !shared) {
            if (2 * t < nblocks) step(BV{}, BK{}, 2 * t, 0);
            if (2 * t + 1 < nblocks) step(BV{}, BK{}, 2 * t + 1, 1);
        } else if (active) {
#pragma unroll
            for (int q = 0; q < kBlocksPerTile; ++q) {
                const int i = 2 * t + q;
                if (i < nblocks && i % nshare == sidx) shared_step(BV{}, i, q);
            }
        }
        PRESTO_WAIT_VM(2 * LPT);
        __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's LDS reads are done
        __builtin_amdgcn_s_barrier();
    };

    // prologue: tiles 0..2 requested, tiles 0 and 1 awaited (and with them
    // Q and the ancestor rows, which were requested first)
    load_tile(k_begin, 0);
    load_tile(k_begin + kKeyTile, 1);
    load_tile(k_begin + 2 * kKeyTile, 2);
    PRESTO_WAIT_VM(2 * LPT);
    __syncthreads();
    using B0 = std::integral_constant<int, 0>;
    if (active && !shared) {
        floatx16 S0 = negm;
        qk(B0{}, 0, S0);
        if (masked(0)) apply_mask(S0, j0_of(0));
        float ls;
        exact(S0, Pp, ls, true, Sb);  // m from block 0; Sb not yet live
        l_run = ls;
        qk(B0{}, 1, Sa);
    }
    for (int t = 0; t < ntiles; t += kRing) {
        tile(std::integral_constant<int, 0>{}, t);
        if (t + 1 < ntiles) tile(std::integral_constant<int, 1>{}, t + 1);
        if (t + 2 < ntiles) tile(std::integral_constant<int, 2>{}, t + 2);
        if (t + 3 < ntiles) tile(std::integral_constant<int, 3>{}, t + 3);
    }
    PRESTO_WAIT_VM(0);  // no load into LDS outlives the workgroup
#undef PRESTO_WAIT_VM

    // ---- the shared block's states, combined pairwise through the (now
    // idle) tile ring: per round the waves at odd multiples of `stride` write
    // (m, l, O) and their partners fold them in
    if (nshare > 1) {
        constexpr int SLOT = kWave * (16 * DB + 2);  // floats per written state
        float* s_state = reinterpret_cast<float*>(s_kv);
        for (int stride = 1; stride < nshare; stride *= 2) {
            __syncthreads();  // every wave's loads have landed; the ring is free
            const bool writer = shared && (sidx % (2 * stride)) == stride;
            const bool reader = shared && (sidx % (2 * stride)) == 0 && sidx + stride < nshare;
            if (writer) {
                float* st = s_state + (sidx / (2 * stride)) * SLOT + lane;
                st[0] = m;
                st[kWave] = l_run;
#pragma unroll
                for (int db = 0; db < DB; ++db)
#pragma unroll
                    for (int e = 0; e < 16; ++e) st[(2 + db * 16 + e) * kWave] = o[db][e];
            }
            __syncthreads();
            if (reader) {
                const float* st = s_state + (sidx / (2 * stride)) * SLOT + lane;
                const float m2 = st[0], l2 = st[kWave];
                const float M = l_run > 0.f ? (l2 > 0.f ? fmaxf(m, m2) : m) : m2;
                const float a1 = l_run > 0.f ? __builtin_amdgcn_exp2f(m - M) : 0.f;
                const float a2 = l2 > 0.f ? __builtin_amdgcn_exp2f(m2 - M) : 0.f;
#pragma unroll
                for (int db = 0; db < DB; ++db)
#pragma unroll
                    for (int e = 0; e < 16; ++e) o[db][e] = a1 * o[db][e] + a2 * st[(2 + db * 16 + e) * kWave];
                l_run = a1 * l_run + a2 * l2;
                m = M;
            }
        }
        if (shared && sidx != 0) return;  // the combined state is wave A-1's
    }

    // ---- epilogue: lane holds row l32, d = db*32 + 8(i/4) + 4h + i%4
    if (rho >= all_rows) return;
    const float l = l_run;  // whole-row sum
    if (a.splits == 1) {
        uint16_t* op = a.out + (((int64_t)b * a.n_max + qn) * a.hq + g * a.G + qh) * D;
        const float inv = (rho < live_rows && l > 0.f) ? 1.f / l : 0.f;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                const int dd = db * 32 + 8 * q4 + 4 * h;
                *reinterpret_cast<uint2*>(op + dd) =
                    make_uint2(pack_bf16x2(o[db][4 * q4] * inv, o[db][4 * q4 + 1] * inv),
                               pack_bf16x2(o[db][4 * q4 + 2] * inv, o[db][4 * q4 + 3] * inv));
            }
    } else {
        // normalised here, so bf16 holds it to the output's own precision
        // output [b, g, split, row] (a workgroup's rows are contiguous: whole
        // lines); (m, l) [b, g, row, split] (the merge reads a row's splits
        // side by side)
        const int64_t bg = (int64_t)b * a.hkv + g;
        const int64_t pr = (bg * a.splits + split) * all_rows + rho;
        const int64_t pm = (bg * all_rows + rho) * a.splits + split;
        uint16_t* po = a.part_o + pr * D;
        const float inv = l > 0.f ? 1.f / l : 0.f;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                const int dd = db * 32 + 8 * q4 + 4 * h;
                *reinterpret_cast<uint2*>(po + dd) =
                    make_uint2(pack_bf16x2(o[db][4 * q4] * inv, o[db][4 * q4 + 1] * inv),
                               pack_bf16x2(o[db][4 * q4 + 2] * inv, o[db][4 * q4 + 3] * inv));
            }
        if (h == 0) a.part_ml[pm] = make_float2(l > 0.f ? m : -INFINITY, l);
    }
}

// Merge of the split partials: one wave per query row.  Lane s reads the
// (m, l) pair of split s (at most 64 splits) and forms its weight
// l exp2(m - M); the splits' normalised outputs are read in groups of
// kMergeUnroll.  The pairs and the first group of outputs are requested
// together with the row's node count and context length, before any of
// them is known (entries of splits the row does not have are read but
// never used), so a row with up to kMergeUnroll splits costs one memory
// round trip.
constexpr int kMergeUnroll = 8;
template <int D>
__global__ __launch_bounds__(256) void tree_attn_merge_kernel(AttnArgs a) {
    constexpr int PER = D / kWave;  // output dims per lane
    static_assert(PER == 1 || PER == 2, "head_dim 64 or 128");
    const int lane = lane_id();
    // grid: x covers the rows of one (sequence, KV head) four per block, y
    // the (sequence, KV head) pairs
    const int rows_g = a.G * a.n_max;
    const int rho = (int)blockIdx.x * (blockDim.x / kWave) + (int)threadIdx.x / kWave;
    if (rho >= rows_g) return;
    const int bg = (int)blockIdx.y;
    const int b = bg / a.hkv, g = bg - b * a.hkv;
    const int n = rho / a.G, hh = rho - n * a.G;
    // split s of this row: ((b, g) * splits + s) * rows + rho; every
    // offset within one (b, g) block of partials fits 32 bits
    const uint16_t* po = a.part_o + ((int64_t)bg * a.splits * rows_g + rho) * D + lane * PER;
    const uint32_t sstride = (uint32_t)rows_g * D;  // elements from one split to the next
    auto load_out = [&](int sp, float (&v)[PER]) {
        const uint16_t* q = po + (uint32_t)sp * sstride;
        if constexpr (PER == 1) {
            v[0] = bf16_to_f(*q);
        } else {
            const uint32_t w2 = *reinterpret_cast<const uint32_t*>(q);
            v[0] = bf16lo(w2);
            v[1] = bf16hi(w2);
        }
    };
    // everything independent is requested at once
    const int nn_raw = a.n_nodes[b];
    const CtxSpan cs = ctx_span(a.ctx_off, b, a.ctx_slots);
    float2 ml = make_float2(-INFINITY, 0.f);
    if (lane < a.splits) ml = a.part_ml[((int64_t)bg * rows_g + rho) * a.splits + lane];
    float v0[kMergeUnroll][PER];
#pragma unroll
    for (int u = 0; u < kMergeUnroll; ++u) load_out(min(u, a.splits - 1), v0[u]);

    const int nn = clamp_nodes(nn_raw, a.n_max);
    const int keys = cs.ctx + nn;
    const int nsplit = min(a.splits, (keys + a.split_len - 1) / a.split_len);
    uint16_t* op = a.out + (((int64_t)b * a.n_max + n) * a.hq + g * a.G + hh) * D + lane * PER;
    float acc[PER];
#pragma unroll
    for (int e = 0; e < PER; ++e) acc[e] = 0.f;
    if (rho < a.G * nn) {
        if (lane >= nsplit) ml = make_float2(-INFINITY, 0.f);
        const float M = wave_max_f32_dpp(ml.x);
        const float wl = ml.x == -INFINITY ? 0.f : exp2f(ml.x - M) * ml.y;  // weight of split `lane`
        const float L = wave_sum_f32_dpp(wl);
        auto add = [&](int sp, const float (&v)[PER]) {
            const float w = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wl), sp));
#pragma unroll
            for (int e = 0; e < PER; ++e) acc[e] += w * v[e];
        };
#pragma unroll
        for (int u = 0; u < kMergeUnroll; ++u)
            if (u < nsplit) add(u, v0[u]);
        for (int s0 = kMergeUnroll; s0 < nsplit; s0 += kMergeUnroll) {
            float v[kMergeUnroll][PER];
#pragma unroll
            for (int u = 0; u < kMergeUnroll; ++u) load_out(min(s0 + u, nsplit - 1), v[u]);
#pragma unroll
            for (int u = 0; u < kMergeUnroll; ++u)
                if (s0 + u < nsplit) add(s0 + u, v[u]);
        }
        const float inv = L > 0.f ? 1.f / L : 0.f;
#pragma unroll
        for (int e = 0; e < PER; ++e) acc[e] *= inv;
    }
    if constexpr (PER == 1) {
        *op = f_to_bf16(acc[0]);
    } else {
        *reinterpret_cast<uint32_t*>(op) =
            (uint32_t)f_to_bf16(acc[0]) | ((uint32_t)f_to_bf16(acc[1]) << 16);
    }
}

// fp32 path: one wave per (b, n, h) row, plain fp32 arithmetic.  Each lane
// runs an online softmax over a strided subset of keys; lanes are merged
// through LDS at the end.
template <int D>
__global__ __launch_bounds__(kWave) void tree_attn_f32_kernel(
    const float* __restrict__ q, const float* __restrict__ kc, const float* __restrict__ vc,
    const int32_t* __restrict__ ctx_off, int32_t ctx_slots, const float* __restrict__ kt,
    const float* __restrict__ vt, const uint64_t* __restrict__ anc,
    const int32_t* __restrict__ n_nodes, float* __restrict__ out, int32_t n_max, int32_t hq,
    int32_t hkv, float scale) {
    __shared__ float s_acc[kWave][D + 1];
    __shared__ float s_m[kWave], s_l[kWave];
    const int lane = lane_id();
    const int h = blockIdx.x % hq;
    const int n = (blockIdx.x / hq) % n_max;
    const int b = blockIdx.x / hq / n_max;
    const int G = hq / hkv, g = h / G, W = (n_max + 63) / 64;
    const int nn = clamp_nodes(n_nodes[b], n_max);
    float* op = out + (((int64_t)b * n_max + n) * hq + h) * D;
    if (n >= nn) {
        for (int e = lane; e < D; e += kWave) op[e] = 0.f;
        return;
    }
    const CtxSpan cs = ctx_span(ctx_off, b, ctx_slots);
    const int c0 = cs.c0, ctx = cs.ctx;
    const float* qp = q + (((int64_t)b * n_max + n) * hq + h) * D;
    const uint64_t* arow = anc + ((int64_t)b * n_max + n) * W;
    float qv[D];
#pragma unroll
    for (int e = 0; e < D; ++e) qv[e] = qp[e];
    float acc[D];
#pragma unroll
    for (int e = 0; e < D; ++e) acc[e] = 0.f;
    float m = -INFINITY, l = 0.f;
    for (int j = lane; j < ctx + nn; j += kWave) {
        const float *kp, *vp;
        if (j < ctx) {
            kp = kc + ((int64_t)(c0 + j) * hkv + g) * D;
            vp = vc + ((int64_t)(c0 + j) * hkv + g) * D;
        } else {
            const int t = j - ctx;
            if (!((arow[t >> 6] >> (t & 63)) & 1ull)) continue;
            kp = kt + (((int64_t)b * n_max + t) * hkv + g) * D;
            vp = vt + (((int64_t)b * n_max + t) * hkv + g) * D;
        }
        float dot = 0.f;
#pragma unroll
        for (int e = 0; e < D; ++e) dot += qv[e] * kp[e];
        const float sc = dot * scale;
        const float mn = fmaxf(m, sc);
        const float al = expf(m - mn), p = expf(sc - mn);
        l = l * al + p;
#pragma unroll
        for (int e = 0; e < D; ++e) acc[e] = acc[e] * al + p * vp[e];
        m = mn;
    }
    s_m[lane] = m;
    s_l[lane] = l;
#pragma unroll
    for (int e = 0; e < D; ++e) s_acc[lane][e] = acc[e];
    __syncthreads();
    float M = -INFINITY;
    for (int i = 0; i < kWave; ++i) M = fmaxf(M, s_m[i]);
    float L = 0.f;
    for (int i = 0; i < kWave; ++i) L += s_m[i] == -INFINITY ? 0.f : s_l[i] * expf(s_m[i] - M);
    for (int e = lane; e < D; e += kWave) {
        float v = 0.f;
        for (int i = 0; i < kWave; ++i)
            v += s_m[i] == -INFINITY ? 0.f : s_acc[i][e] * expf(s_m[i] - M);
        op[e] = v / L;
    }
}

}  // namespace presto

namespace presto_host {

using namespace presto;

struct AttnPlan {
    int G, rows, row_tiles, rows_per_tile, waves, rb, splits, split_len;
    bool compact;
    int64_t tasks, blocks;
};

static AttnPlan attn_plan(const presto_attn_desc* d) {
    AttnPlan p;
    p.G = d->hq / d->hkv;
    p.rows = p.G * d->n_max;
    // 256 query rows per workgroup: eight waves of one 32-row block, or four
    // waves of two (each K/V fragment read from LDS then feeds two MFMAs)
    p.waves = kAttnWaves;
    p.rows_per_tile = kAttnRows;
    p.row_tiles = (p.rows + p.rows_per_tile - 1) / p.rows_per_tile;
    // context splits: one workgroup per CU, so the time in key-block units
    // (about 0.85 us each) is (rounds of workgroups) x (key blocks per split
    // + about 3 for a workgroup's prologue) plus the merge, whose partials
    // (2 D + 8 bytes per query row and split, written and read back, about
    // 4 MB per key-block time) grow with the split count
    // With ragged contexts and the caller's total, the workgroups are dealt
    // over the (sequence, split) pairs that exist (about total/len + batch/2
    // of them) rather than batch x splits of the longest sequence.
    const int64_t per_pair = (int64_t)d->hkv * p.row_tiles;  // workgroups per (sequence, split)
    const int keys = d->max_ctx + d->n_max;                  // the longest sequence
    p.compact = d->batch > 1 && d->total_ctx > 0 && d->total_ctx < (int64_t)d->batch * d->max_ctx;
    const double total_keys = (double)d->total_ctx + (double)d->batch * d->n_max;
    const int max_splits = (keys + 127) / 128;
    double best_cost = 1e30;
    p.splits = 1;
    p.split_len = (keys + kKeyTile - 1) / kKeyTile * kKeyTile;
    for (int s = 1; s <= kWave && s <= max_splits; ++s) {  // the merge gives each split a lane
        int len = (keys + s - 1) / s;
        len = (len + kKeyTile - 1) / kKeyTile * kKeyTile;
        const int se = (keys + len - 1) / len;
        const double pairs = p.compact ? fmin((double)d->batch * se, total_keys / len + 0.5 * d->batch)
                                       : (double)d->batch * se;
        const double rounds = ceil(pairs * per_pair / 256.0);
        const double merge_bytes =
            se > 1 ? 2.0 * d->hkv * p.rows * pairs * (2.0 * d->head_dim + 8.0) : 0.0;
        const double cost = rounds * ((len + 31) / 32 + 3) + merge_bytes / 4.0e6;
        if (cost < best_cost - 1e-9) {
            best_cost = cost;
            p.splits = se;
            p.split_len = len;
        }
    }
    p.tasks = (int64_t)d->batch * p.splits * per_pair;  // in compact mode an upper bound
    p.blocks = (p.tasks + 7) / 8 * 8;
    // When the whole grid fits one round (one workgroup per CU), the tiles
    // are balanced: the same number of row tiles, each a multiple of 32 rows
    // (a 32-row block never straddles two tiles).  260 rows then make tiles
    // of 160 and 100 rows instead of 256 and 4: a workgroup of 256 rows runs
    // two waves per SIMD through every key block (about 1 us per block), one
    // of 160 rows one and a quarter (the idle waves share the fifth block's
    // keys), and the 4-row tiles, nearly idle, disappear.
    if (!p.compact && p.tasks <= 256 && p.row_tiles > 1)
        p.rows_per_tile = kRowsPerWave * ((p.rows + kRowsPerWave * p.row_tiles - 1) / (kRowsPerWave * p.row_tiles));
    return p;
}

size_t attn_workspace_bytes(const presto_attn_desc* d) {
    if (d->dt != PRESTO_DT_BF16) return 0;
    const AttnPlan p = attn_plan(d);
    if (p.splits <= 1) return 0;
    const size_t prs = (size_t)d->batch * d->hkv * p.G * d->n_max * p.splits;
    return ((prs * d->head_dim * sizeof(uint16_t) + 255) & ~(size_t)255) + prs * sizeof(float2) + 256;
}

presto_status launch_tree_attention(const presto_attn_desc* d, const void* q, const void* k_cache,
                                    const void* v_cache, const int32_t* ctx_offsets,
                                    const void* k_tree, const void* v_tree, const uint64_t* anc,
                                    const int32_t* n_nodes, void* out, void* ws,
                                    hipStream_t stream) {
    if (d->dt == PRESTO_DT_F32) {
        const unsigned grid = (unsigned)((int64_t)d->batch * d->n_max * d->hq);
#define PRESTO_F32(DD)                                                                           \
    tree_attn_f32_kernel<DD><<<grid, kWave, 0, stream>>>(                                        \
        (const float*)q, (const float*)k_cache, (const float*)v_cache, ctx_offsets,              \
        d->ctx_layout == PRESTO_CTX_SLOTS,                                                       \
        (const float*)k_tree, (const float*)v_tree, anc, n_nodes, (float*)out, d->n_max, d->hq, \
        d->hkv, d->scale)
        if (d->head_dim == 64) PRESTO_F32(64); else PRESTO_F32(128);
#undef PRESTO_F32
        return check_launch("tree_attn_f32_kernel");
    }
    const AttnPlan p = attn_plan(d);
    if (p.splits > 1 && (int64_t)d->batch * d->hkv > 65535)  // the merge's grid.y
        return set_error(PRESTO_ERR_UNSUPPORTED, "tree attention: batch x KV heads %lld above 65535",
                         (long long)d->batch * d->hkv);
    AttnArgs a;
    a.q = (const uint16_t*)q;
    a.kc = (const uint16_t*)k_cache;
    a.vc = (const uint16_t*)v_cache;
    a.ctx_off = ctx_offsets;
    a.ctx_slots = d->ctx_layout == PRESTO_CTX_SLOTS;
    a.kt = (const uint16_t*)k_tree;
    a.vt = (const uint16_t*)v_tree;
    a.anc = anc;
    a.n_nodes = n_nodes;
    a.out = (uint16_t*)out;
    {
        const size_t prs = (size_t)d->batch * d->hkv * p.G * d->n_max * p.splits;
        a.part_o = (uint16_t*)ws;
        a.part_ml = (float2*)((char*)ws + ((prs * d->head_dim * sizeof(uint16_t) + 255) & ~(size_t)255));
    }
    a.batch = d->batch;
    a.n_max = d->n_max;
    a.hq = d->hq;
    a.hkv = d->hkv;
    a.G = p.G;
    a.W = (d->n_max + 63) / 64;
    a.row_tiles = p.row_tiles;
    a.rows_per_tile = p.rows_per_tile;
    a.splits = p.splits;
    a.split_len = p.split_len;
    a.n_tasks = (int32_t)p.tasks;
    a.compact = p.compact ? 1 : 0;
    a.n_blocks = (int32_t)p.blocks;
    a.scale_log2 = d->scale * kLog2e;
    const dim3 block(p.waves * kWave), grid((unsigned)p.blocks);
    if (d->head_dim == 64)
        tree_attn_bf16_kernel<64><<<grid, block, 0, stream>>>(a);
    else
        tree_attn_bf16_kernel<128><<<grid, block, 0, stream>>>(a);
    presto_status st = check_launch("tree_attn_bf16_kernel");
    if (st != PRESTO_OK || p.splits == 1) return st;
    const dim3 mgrid((unsigned)((p.rows + 3) / 4), (unsigned)(d->batch * d->hkv));
    if (d->head_dim == 64)
        tree_attn_merge_kernel<64><<<mgrid, 256, 0, stream>>>(a);
    else
        tree_attn_merge_kernel<128><<<mgrid, 256, 0, stream>>>(a);
    return check_launch("tree_attn_merge_kernel");
}

}  // namespace presto_host
