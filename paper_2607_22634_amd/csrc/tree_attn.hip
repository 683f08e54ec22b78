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
constexpr int kBufs = 3;          // LDS tile buffers
constexpr float kSlack = 8.f;     // log2 headroom before the accumulator is rescaled
constexpr int kMaxAncWords = 16;  // ancestor words per node: n_max <= 1024
constexpr int kRowsPerWave = 32;  // one 32-row MFMA block per wave
// Workgroups are 8 waves, two per SIMD: one wave's softmax hides behind the
// other's MFMAs (with one wave per SIMD the matrix cores sit idle during it).
constexpr int kAttnWaves = 8;
// 32-row blocks per wave.  Two (four waves, each K/V fragment feeding two
// MFMAs) needs about 340 registers per lane at head_dim 128 and spills with
// the current register allocation, so one block per wave is used.
constexpr int kAttnRowBlocks = 1;
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
    int32_t row_tiles, splits, split_len;
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

// This thread's PT 16-byte pieces of one K tile and one V tile.
template <int PT>
struct TilePieces {
    uint4 k[PT], v[PT];
};

// Loads this thread's pieces of the K and V tile that starts at key t0.
// Keys below ctx come from the packed cache row c0 + j, the others from the
// tree K/V of node j - ctx; rows past k_end repeat the last key (every load
// stays in bounds; their scores are masked to -inf).
template <int D, int PT, int NT>
__device__ __forceinline__ TilePieces<PT> fetch_tile(const uint16_t* kc, const uint16_t* vc,
                                                     const uint16_t* kt, const uint16_t* vt, int tid,
                                                     int t0, int k_end, int ctx, int c0, int hkv,
                                                     int g, int64_t tree_row0) {
    const int64_t kv_stride = (int64_t)hkv * D;
    TilePieces<PT> r;
#pragma unroll
    for (int i = 0; i < PT; ++i) {
        const int p = tid + i * NT;
        const int kk = p / (D / 8), c8 = p % (D / 8);
        const int j = min(t0 + kk, k_end - 1);
        const bool in_ctx = j < ctx;
        const int64_t off = in_ctx ? (int64_t)(c0 + j) * kv_stride + (int64_t)g * D + c8 * 8
                                   : ((tree_row0 + (j - ctx)) * hkv + g) * D + c8 * 8;
        const uint16_t* kp = in_ctx ? kc : kt;
        const uint16_t* vp = in_ctx ? vc : vt;
        r.k[i] = *reinterpret_cast<const uint4*>(kp + off);
        r.v[i] = *reinterpret_cast<const uint4*>(vp + off);
    }
    return r;
}

template <int D, int NW, int RB>
__global__ __launch_bounds__(NW * kWave) void tree_attn_bf16_kernel(AttnArgs a) {
    constexpr int KS = D / 16;                 // S^T contraction steps over the head dimension
    constexpr int DB = D / 32;                 // 32-wide blocks of the output head dimension
    constexpr int KROW = D + 8;                // K row in LDS (bf16): conflict-free b128 reads
    constexpr int VROW = D + 32;               // V row in LDS: conflict-free transposed b64 reads
    constexpr int PIECES = kKeyTile * D / 8;   // 16-byte pieces of one K (or V) tile
    constexpr int NT = NW * kWave;
    constexpr int PT = PIECES / NT;            // pieces per thread
    constexpr int WROWS = RB * kRowsPerWave;   // query rows per wave (RB blocks of 32)
    constexpr int ROWS = NW * WROWS;           // query rows per workgroup
    constexpr int KBUF = kKeyTile * KROW, VBUF = kKeyTile * VROW;
    static_assert(PT * NT == PIECES, "tile pieces must divide evenly");
    __shared__ __align__(16) uint16_t sK[kBufs * KBUF];
    __shared__ __align__(16) uint16_t sV[kBufs * VBUF];
    __shared__ uint64_t s_anc[(ROWS + 1) * kMaxAncWords];  // ancestor rows of this tile's nodes

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
    const int row0 = rt * ROWS + wave * WROWS;  // first query row of this wave
    const bool active = row0 < live_rows;
    int rho[RB], qn[RB], qh[RB], node[RB];  // this lane's query row in each row block
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        rho[rb] = row0 + rb * kRowsPerWave + l32;
        qn[rb] = rho[rb] / a.G;
        qh[rb] = rho[rb] - qn[rb] * a.G;
        node[rb] = min(qn[rb], a.n_max - 1);
    }

    // Q fragments, B operand of S^T = K Q^T: lane holds row l32, d = ks*16 + h*8 .. +8.
    // Loaded before the first K/V tiles, so the waits for those tiles also
    // cover Q and nothing in the key loop waits on global loads but the stage.
    bf16x8 qf[RB][KS];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        const uint16_t* qp = a.q + (((int64_t)b * a.n_max + qn[rb]) * a.hq + g * a.G + qh[rb]) * D;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            uint4 u = make_uint4(0, 0, 0, 0);
            if (rho[rb] < all_rows) u = *reinterpret_cast<const uint4*>(qp + ks * 16 + h * 8);
            qf[rb][ks] = __builtin_bit_cast(bf16x8, u);
        }
    }

    // ---- K/V staging: global -> registers -> LDS, three buffers: while tile t
    // is consumed, tile t+1 is already in LDS (the last block of a tile scores
    // the first block of the next one) and tile t+2 is in flight.
    // A tile wholly inside the context is read at a uniform base plus a
    // per-thread 32-bit byte offset fixed for the whole loop (no per-tile
    // address arithmetic); other tiles take the general path.
    const int fast_end = min(ctx, k_end);
    uint32_t piece_off[PT];
#pragma unroll
    for (int i = 0; i < PT; ++i) {
        const int p = tid + i * NT;
        piece_off[i] = (uint32_t)(((p / (D / 8)) * a.hkv * D + (p % (D / 8)) * 8) * 2);
    }
    auto fetch = [&](int t0) {
        if (t0 + kKeyTile <= fast_end) {
            const int64_t row = ((int64_t)(c0 + t0) * a.hkv + g) * D;
            const char* kb = reinterpret_cast<const char*>(a.kc + row);
            const char* vb = reinterpret_cast<const char*>(a.vc + row);
            TilePieces<PT> r;
#pragma unroll
            for (int i = 0; i < PT; ++i) {
                r.k[i] = *reinterpret_cast<const uint4*>(kb + piece_off[i]);
                r.v[i] = *reinterpret_cast<const uint4*>(vb + piece_off[i]);
            }
            return r;
        }
        return fetch_tile<D, PT, NT>(a.kc, a.vc, a.kt, a.vt, tid, t0, k_end, ctx, c0, a.hkv, g,
                                     (int64_t)b * a.n_max);
    };
    auto stage = [&](int buf, const TilePieces<PT>& tp) {
#pragma unroll
        for (int i = 0; i < PT; ++i) {
            const int p = tid + i * NT;
            const int kk = p / (D / 8), c8 = p % (D / 8);
            *reinterpret_cast<uint4*>(&sK[buf * KBUF + kk * KROW + c8 * 8]) = tp.k[i];
            *reinterpret_cast<uint4*>(&sV[buf * VBUF + kk * VROW + c8 * 8]) = tp.v[i];
        }
    };
    // unconditional: tiles past the split only repeat the last key, and a
    // buffer staged with them is never read
    TilePieces<PT> pend = fetch(k_begin);
    {
        const TilePieces<PT> second = fetch(k_begin + kKeyTile);
        stage(0, pend);
        stage(1, second);
    }
    pend = fetch(k_begin + 2 * kKeyTile);
    // ancestor bitmask rows of the nodes this workgroup serves, when the
    // split reaches the tree keys (masks then read LDS, not global memory)
    const int n_first = (rt * ROWS) / a.G;
    if (k_end > ctx) {
        const int n_last = min((rt * ROWS + ROWS - 1) / a.G, a.n_max - 1);
        const int words = (n_last - n_first + 1) * a.W;
        const uint64_t* src = a.anc + ((int64_t)b * a.n_max + n_first) * a.W;
        for (int w = tid; w < words; w += NT) s_anc[w] = src[w];
    }
    __syncthreads();

    floatx16 o[RB][DB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int i = 0; i < 16; ++i) o[rb][db][i] = 0.f;
    // Running reference m (log2 domain, scaled) and denominator l per row.
    // m only moves when a block's maximum exceeds it by more than kSlack, so
    // most blocks skip the accumulator rescale; probabilities stay below
    // 2^kSlack.
    float m_run[RB], l_run[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        m_run[rb] = -INFINITY;
        l_run[rb] = 0.f;
    }

    const float c = a.scale_log2;
    // per-lane LDS element offsets; every fragment read adds only a constant
    const int k_lane = l32 * KROW + h * 8;
    const int v_lane = (4 * h + ((lane & 15) >> 2)) * VROW + ((lane >> 4) & 1) * 16 + 4 * (lane & 3);

    // S^T blocks of 32 keys (block i of the split) for every row block: each
    // K fragment read from LDS feeds RB MFMAs
    auto scores = [&](int i, floatx16 (&S)[RB]) {
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
            for (int e = 0; e < 16; ++e) S[rb][e] = 0.f;
        const int buf = (i / kBlocksPerTile) % kBufs, blk = i % kBlocksPerTile;
        int koff = buf * KBUF + blk * 32 * KROW + k_lane;
        asm volatile("" : "+v"(koff));  // keep the per-read constants as immediate offsets
        const uint16_t* kb = sK + koff;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const bf16x8 ka = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(kb + ks * 16));
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
                S[rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[rb][ks], S[rb], 0, 0, 0);
        }
    };
    // element e of a lane is key j0 + 8(e/4) + 4h + e%4
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
    auto apply_mask = [&](floatx16& S, int j0, int nd) {
        const int s0 = j0 - ctx;  // tree index of the block's first key (< 0: it starts in the context)
        uint32_t anc = 0u;
        if (j0 + 32 > ctx) {
            const uint64_t* arow = &s_anc[(nd - n_first) * a.W];
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
    // move m of row block rb when its block maximum mx (raw score) exceeds
    // it by more than kSlack
    auto update = [&](int rb, float mx) {
        const float mx2 = mx * c;
        const bool need = mx2 > m_run[rb] + kSlack;
        if (__ballot(need)) {
            const float mn = need ? mx2 : m_run[rb];
            const float alpha = need ? __builtin_amdgcn_exp2f(m_run[rb] - mn) : 1.f;
            m_run[rb] = mn;
            l_run[rb] *= alpha;
#pragma unroll
            for (int db = 0; db < DB; ++db) o[rb][db] *= alpha;
        }
    };

    // one 32-key block: scores of every row block (K fragments shared), then
    // the softmax and P V of each row block; with two row blocks one block's
    // softmax overlaps the other's MFMAs
    auto block_step = [&](int t, int q, int i, floatx16 (&S)[RB]) {
        const int j0 = k_begin + i * 32;
        float mx[RB];
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) mx[rb] = row_max(S[rb]);
        if (j0 + 32 > mask_from) {
#pragma unroll
            for (int rb = 0; rb < RB; ++rb) {
                apply_mask(S[rb], j0, node[rb]);
                mx[rb] = row_max(S[rb]);
            }
        }
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) update(rb, mx[rb]);
        uint32_t P[RB][8];
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
            const float m_use = m_run[rb] == -INFINITY ? 0.f : m_run[rb];
            float ls = 0.f;
#pragma unroll
            for (int e = 0; e < 16; e += 2) {
                const float p0 = __builtin_amdgcn_exp2f(fmaf(S[rb][e], c, -m_use));
                const float p1 = __builtin_amdgcn_exp2f(fmaf(S[rb][e + 1], c, -m_use));
                ls += p0 + p1;
                P[rb][e >> 1] = pack_bf16x2(p0, p1);
            }
            l_run[rb] += ls;
        }
        int voff = (t % kBufs) * VBUF + q * 32 * VROW + v_lane;
        asm volatile("" : "+v"(voff));
        const uint16_t* vb = sV + voff;
#pragma unroll
        for (int st = 0; st < 2; ++st) {
#pragma unroll
            for (int db = 0; db < DB; ++db) {
                const uint16_t* v0 = vb + st * 16 * VROW + db * 32;
                const short4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (__attribute__((address_space(3))) short4_t*)(v0));
                const short4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (__attribute__((address_space(3))) short4_t*)(v0 + 8 * VROW));
                const uint2 ul = __builtin_bit_cast(uint2, lo), uh = __builtin_bit_cast(uint2, hi);
                const bf16x8 va = __builtin_bit_cast(bf16x8, make_uint4(ul.x, ul.y, uh.x, uh.y));
#pragma unroll
                for (int rb = 0; rb < RB; ++rb) {
                    const bf16x8 pb = __builtin_bit_cast(
                        bf16x8, make_uint4(P[rb][4 * st], P[rb][4 * st + 1], P[rb][4 * st + 2], P[rb][4 * st + 3]));
                    o[rb][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb, o[rb][db], 0, 0, 0);
                }
            }
        }
    };

    if constexpr (RB == 1) {
        // one row block: the scores of block i+1 (its tile is already in LDS)
        // are issued ahead of the softmax and P V of block i
        floatx16 S_cur[1];
        if (active) scores(0, S_cur);
        for (int t = 0; t < ntiles; ++t) {
            if (active) {
#pragma unroll
                for (int q = 0; q < kBlocksPerTile; ++q) {
                    const int i = t * kBlocksPerTile + q;
                    if (i < nblocks) {
                        floatx16 S_nxt[1];
                        scores(i + 1, S_nxt);
                        block_step(t, q, i, S_cur);
                        S_cur[0] = S_nxt[0];
                    }
                }
            }
            // tile t+2 goes into the buffer of tile t-1, which every wave
            // finished before the previous barrier
            stage((t + 2) % kBufs, pend);
            pend = fetch(k_begin + (t + 3) * kKeyTile);
            __syncthreads();
        }
    } else {
        for (int t = 0; t < ntiles; ++t) {
            if (active) {
#pragma unroll
                for (int q = 0; q < kBlocksPerTile; ++q) {
                    const int i = t * kBlocksPerTile + q;
                    if (i < nblocks) {
                        floatx16 S[RB];
                        scores(i, S);
                        block_step(t, q, i, S);
                    }
                }
            }
            stage((t + 2) % kBufs, pend);
            pend = fetch(k_begin + (t + 3) * kKeyTile);
            __syncthreads();
        }
    }

    // ---- epilogue: lane holds row l32 of each row block, d = db*32 + 8(i/4) + 4h + i%4
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
        float l = l_run[rb];
        {
            const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(l), __float_as_uint(l), false,
                                                             false);
            l += __uint_as_float(h == 0 ? sw[1] : sw[0]);
        }
        if (rho[rb] >= all_rows) continue;
        if (a.splits == 1) {
            uint16_t* op = a.out + (((int64_t)b * a.n_max + qn[rb]) * a.hq + g * a.G + qh[rb]) * D;
            const float inv = (rho[rb] < live_rows && l > 0.f) ? 1.f / l : 0.f;
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
                for (int q4 = 0; q4 < 4; ++q4) {
                    const int dd = db * 32 + 8 * q4 + 4 * h;
                    *reinterpret_cast<uint2*>(op + dd) =
                        make_uint2(pack_bf16x2(o[rb][db][4 * q4] * inv, o[rb][db][4 * q4 + 1] * inv),
                                   pack_bf16x2(o[rb][db][4 * q4 + 2] * inv, o[rb][db][4 * q4 + 3] * inv));
                }
        } else {
            // normalised here, so bf16 holds it to the output's own precision
            // output [b, g, split, row] (a workgroup's rows are contiguous: whole
            // lines); (m, l) [b, g, row, split] (the merge reads a row's splits
            // side by side)
            const int64_t bg = (int64_t)b * a.hkv + g;
            const int64_t pr = (bg * a.splits + split) * all_rows + rho[rb];
            const int64_t pm = (bg * all_rows + rho[rb]) * a.splits + split;
            uint16_t* po = a.part_o + pr * D;
            const float inv = l > 0.f ? 1.f / l : 0.f;
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
                for (int q4 = 0; q4 < 4; ++q4) {
                    const int dd = db * 32 + 8 * q4 + 4 * h;
                    *reinterpret_cast<uint2*>(po + dd) =
                        make_uint2(pack_bf16x2(o[rb][db][4 * q4] * inv, o[rb][db][4 * q4 + 1] * inv),
                                   pack_bf16x2(o[rb][db][4 * q4 + 2] * inv, o[rb][db][4 * q4 + 3] * inv));
                }
            if (h == 0) a.part_ml[pm] = make_float2(m_run[rb], l);
        }
    }
}

// Merge of the split partials: one wave per query row.  Lane s reads the
// (m, l) pair of split s (at most 64 splits) and forms its weight
// l exp2(m - M); the splits' normalised outputs are then read in groups of
// kMergeUnroll with every load of a group issued before the first is used,
// so a row costs two memory round trips rather than one per split.
constexpr int kMergeUnroll = 8;
template <int D>
__global__ __launch_bounds__(256) void tree_attn_merge_kernel(AttnArgs a) {
    constexpr int PER = D / kWave;  // output dims per lane
    const int lane = lane_id();
    const int64_t r = (int64_t)blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
    const int64_t rows = (int64_t)a.batch * a.hkv * a.G * a.n_max;
    if (r >= rows) return;
    const int rho = (int)(r % (a.G * a.n_max));
    const int g = (int)((r / (a.G * a.n_max)) % a.hkv);
    const int b = (int)(r / ((int64_t)a.G * a.n_max * a.hkv));
    const int n = rho / a.G, hh = rho - n * a.G;
    const int nn = clamp_nodes(a.n_nodes[b], a.n_max);
    uint16_t* op = a.out + (((int64_t)b * a.n_max + n) * a.hq + g * a.G + hh) * D + lane * PER;
    float acc[PER];
#pragma unroll
    for (int e = 0; e < PER; ++e) acc[e] = 0.f;
    if (rho < a.G * nn) {
        const int keys = ctx_span(a.ctx_off, b, a.ctx_slots).ctx + nn;
        const int nsplit = min(a.splits, (keys + a.split_len - 1) / a.split_len);
        // split s of this row: ((b, g) * splits + s) * rows + rho
        const int64_t rows_g = (int64_t)a.G * a.n_max;
        const int64_t pr = ((int64_t)b * a.hkv + g) * a.splits * rows_g + rho;
        const uint16_t* po = a.part_o + pr * D + lane * PER;
        float2 ml = make_float2(-INFINITY, 0.f);
        if (lane < nsplit) ml = a.part_ml[(((int64_t)b * a.hkv + g) * rows_g + rho) * a.splits + lane];
        const float M = wave_max_f32_dpp(ml.x);
        const float wl = ml.x == -INFINITY ? 0.f : exp2f(ml.x - M) * ml.y;  // weight of split `lane`
        const float L = wave_sum_f32_dpp(wl);
        for (int s0 = 0; s0 < nsplit; s0 += kMergeUnroll) {
            float v[kMergeUnroll][PER];
#pragma unroll
            for (int u = 0; u < kMergeUnroll; ++u) {
                const int s = min(s0 + u, nsplit - 1);
                if constexpr (PER == 1) {
                    v[u][0] = bf16_to_f(po[s * rows_g * D]);
                } else {
                    const uint32_t w2 = *reinterpret_cast<const uint32_t*>(po + s * rows_g * D);
                    v[u][0] = bf16_to_f((uint16_t)(w2 & 0xffffu));
                    v[u][1] = bf16_to_f((uint16_t)(w2 >> 16));
                }
            }
#pragma unroll
            for (int u = 0; u < kMergeUnroll; ++u) {
                if (s0 + u < nsplit) {
                    const float w = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wl), s0 + u));
#pragma unroll
                    for (int e = 0; e < PER; ++e) acc[e] += w * v[u][e];
                }
            }
        }
        const float inv = L > 0.f ? 1.f / L : 0.f;
#pragma unroll
        for (int e = 0; e < PER; ++e) acc[e] *= inv;
    }
    if constexpr (PER == 1) {
        *op = f_to_bf16(acc[0]);
    } else {
        static_assert(PER == 2, "head_dim 64 or 128");
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
    p.rb = kAttnRowBlocks;
    p.waves = kAttnWaves / p.rb;
    p.rows_per_tile = p.waves * kRowsPerWave * p.rb;
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
    a.splits = p.splits;
    a.split_len = p.split_len;
    a.n_tasks = (int32_t)p.tasks;
    a.compact = p.compact ? 1 : 0;
    a.n_blocks = (int32_t)p.blocks;
    a.scale_log2 = d->scale * kLog2e;
    const dim3 block(p.waves * kWave), grid((unsigned)p.blocks);
    constexpr int RB = kAttnRowBlocks, NW = kAttnWaves / kAttnRowBlocks;
    if (d->head_dim == 64)
        tree_attn_bf16_kernel<64, NW, RB><<<grid, block, 0, stream>>>(a);
    else
        tree_attn_bf16_kernel<128, NW, RB><<<grid, block, 0, stream>>>(a);
    presto_status st = check_launch("tree_attn_bf16_kernel");
    if (st != PRESTO_OK || p.splits == 1) return st;
    const int64_t merge_rows = (int64_t)d->batch * d->hkv * p.G * d->n_max;
    const unsigned mgrid = (unsigned)((merge_rows + 3) / 4);
    if (d->head_dim == 64)
        tree_attn_merge_kernel<64><<<mgrid, 256, 0, stream>>>(a);
    else
        tree_attn_merge_kernel<128><<<mgrid, 256, 0, stream>>>(a);
    return check_launch("tree_attn_merge_kernel");
}

}  // namespace presto_host
