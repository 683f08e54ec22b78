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
// bf16 path (matrix cores, v_mfma_f32_16x16x32_bf16).  Each wave owns 32
// query rows.  Scores are computed transposed, S^T = K Q^T, so that each
// lane holds one query row and 4+4 keys of a 32-key step: the row max/sum
// need only two cross-lane steps, and the probabilities already sit in the
// B-operand layout of O^T = V^T P^T; V is staged transposed in LDS to feed
// the A operand.  The context is split across workgroups when a sequence
// alone cannot fill the chip; partial (max, sum, accumulator) triples are
// then merged by a second kernel.
#include <math.h>

#include "common.hpp"

namespace presto {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kKeyTile = 64;  // keys per LDS tile
constexpr int kRowsPerWave = 32;
constexpr int kMaxRowsPerTile = 256;  // 8 waves: two per SIMD, 256 registers each
constexpr int kKPad = 8;      // bf16 padding of a K row in LDS (bank spread)
constexpr int kVPad = 8;      // bf16 padding of a V^T row in LDS
constexpr float kLog2e = 1.4426950408889634f;

struct AttnArgs {
    const uint16_t* q;
    const uint16_t* kc;
    const uint16_t* vc;
    const int32_t* ctx_off;
    const uint16_t* kt;
    const uint16_t* vt;
    const uint64_t* anc;
    const int32_t* n_nodes;
    uint16_t* out;
    float* part;  // [batch, hkv, rows_pad, splits, D + 2] when splits > 1
    int32_t batch, n_max, hq, hkv, G, W;
    int32_t row_tiles, rows_per_tile, rows_pad, splits, split_len;
    int32_t n_tasks, n_blocks;
    float scale_log2;  // scale * log2(e)
};

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

template <int D>
__global__ __launch_bounds__(512) void tree_attn_bf16_kernel(AttnArgs a) {
    constexpr int DB = D / 16;  // 16-wide blocks of the head dimension
    constexpr int KS = D / 32;  // 32-deep contraction steps over the head dimension
    constexpr int KROW = D + kKPad;
    constexpr int VROW = kKeyTile + kVPad;
    __shared__ __align__(16) uint16_t sK[kKeyTile * KROW];
    __shared__ __align__(16) uint16_t sV[D * VROW];

    const int task = xcd_task(blockIdx.x, a.n_blocks);
    if (task >= a.n_tasks) return;
    const int rt = task % a.row_tiles;
    const int split = (task / a.row_tiles) % a.splits;
    const int g = (task / a.row_tiles / a.splits) % a.hkv;
    const int b = task / a.row_tiles / a.splits / a.hkv;

    const int c0 = a.ctx_off[b];
    const int ctx = a.ctx_off[b + 1] - c0;
    const int nn = clamp_nodes(a.n_nodes[b], a.n_max);
    const int keys = ctx + nn;
    const int k_begin = split * a.split_len;
    if (k_begin >= keys) return;  // nothing of this sequence in this split
    const int k_end = min(keys, k_begin + a.split_len);
    const int live_rows = a.G * nn;

    const int tid = threadIdx.x, nthr = blockDim.x;
    const int wave = tid / kWave, lane = lane_id();
    const int li = lane & 15, lg = lane >> 4;  // row within a 16-block, lane group
    const int row0 = rt * a.rows_per_tile + wave * kRowsPerWave;

    // Q fragments (B operand of S^T = K Q^T): lane holds row li, d = ks*32 + lg*8 .. +8
    bf16x8 qf[2][KS];
    int node_of[2];
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
        const int rho = row0 + blk * 16 + li;
        const int n = rho / a.G, hh = rho - n * a.G;
        node_of[blk] = n;
        const bool ok = rho < a.G * a.n_max;
        const uint16_t* qp = a.q + (((int64_t)b * a.n_max + n) * a.hq + g * a.G + hh) * D;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            uint4 u = make_uint4(0, 0, 0, 0);
            if (ok) u = *reinterpret_cast<const uint4*>(qp + ks * 32 + lg * 8);
            qf[blk][ks] = __builtin_bit_cast(bf16x8, u);
        }
    }

    floatx4 o[2][DB];
    float m_run[2], l_run[2];
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
        m_run[blk] = -INFINITY;
        l_run[blk] = 0.f;
#pragma unroll
        for (int db = 0; db < DB; ++db) o[blk][db] = floatx4{0.f, 0.f, 0.f, 0.f};
    }

    const int64_t kv_stride = (int64_t)a.hkv * D;  // elements between consecutive positions
    for (int t0 = k_begin; t0 < k_end; t0 += kKeyTile) {
        // ---- stage K (row major) and V (transposed) of keys t0 .. t0+63
        constexpr int PIECES = kKeyTile * D / 8;
        for (int p = tid; p < PIECES; p += nthr) {
            const int kk = p / (D / 8), c8 = p % (D / 8);
            const int j = t0 + kk;
            uint4 ku = make_uint4(0, 0, 0, 0), vu = make_uint4(0, 0, 0, 0);
            if (j < k_end) {
                const uint16_t *ks, *vs;
                if (j < ctx) {
                    const int64_t off = (int64_t)(c0 + j) * kv_stride + (int64_t)g * D + c8 * 8;
                    ks = a.kc + off;
                    vs = a.vc + off;
                } else {
                    const int64_t off = (((int64_t)b * a.n_max + (j - ctx)) * a.hkv + g) * D + c8 * 8;
                    ks = a.kt + off;
                    vs = a.vt + off;
                }
                ku = *reinterpret_cast<const uint4*>(ks);
                vu = *reinterpret_cast<const uint4*>(vs);
            }
            *reinterpret_cast<uint4*>(&sK[kk * KROW + c8 * 8]) = ku;
            const uint32_t vw[4] = {vu.x, vu.y, vu.z, vu.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                sV[(c8 * 8 + 2 * e) * VROW + kk] = (uint16_t)(vw[e] & 0xffffu);
                sV[(c8 * 8 + 2 * e + 1) * VROW + kk] = (uint16_t)(vw[e] >> 16);
            }
        }
        __syncthreads();

        if (row0 < live_rows) {
#pragma unroll
            for (int blk = 0; blk < 2; ++blk) {
                // ---- S^T for 64 keys: 4 key blocks of 16
                floatx4 s[4];
#pragma unroll
                for (int kb = 0; kb < 4; ++kb) {
                    floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int ks = 0; ks < KS; ++ks) {
                        const uint4 u = *reinterpret_cast<const uint4*>(
                            &sK[(kb * 16 + li) * KROW + ks * 32 + lg * 8]);
                        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                            __builtin_bit_cast(bf16x8, u), qf[blk][ks], acc, 0, 0, 0);
                    }
                    s[kb] = acc;
                }
                // ---- scale, mask (end of sequence, tree ancestry), running max
                const int n = node_of[blk];
                const uint64_t* arow = a.anc + ((int64_t)b * a.n_max + min(n, a.n_max - 1)) * a.W;
                float mx = -INFINITY;
#pragma unroll
                for (int kb = 0; kb < 4; ++kb) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int j = t0 + kb * 16 + lg * 4 + e;
                        bool vis = j < k_end;
                        if (vis && j >= ctx) {
                            const int m = j - ctx;
                            vis = (arow[m >> 6] >> (m & 63)) & 1ull;
                        }
                        const float v = vis ? s[kb][e] * a.scale_log2 : -INFINITY;
                        s[kb][e] = v;
                        mx = fmaxf(mx, v);
                    }
                }
                mx = fmaxf(mx, __shfl_xor(mx, 16, kWave));
                mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
                const float m_new = fmaxf(m_run[blk], mx);
                const float m_use = m_new == -INFINITY ? 0.f : m_new;
                const float alpha = exp2f(m_run[blk] - m_use);
                m_run[blk] = m_new;
                float ls = 0.f;
                uint32_t pk[4][2];
#pragma unroll
                for (int kb = 0; kb < 4; ++kb) {
                    float p[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        p[e] = exp2f(s[kb][e] - m_use);
                        ls += p[e];
                    }
                    pk[kb][0] = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)p[0]) |
                                ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)p[1]) << 16);
                    pk[kb][1] = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)p[2]) |
                                ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)p[3]) << 16);
                }
                l_run[blk] = l_run[blk] * alpha + ls;
#pragma unroll
                for (int db = 0; db < DB; ++db) o[blk][db] *= alpha;
                // ---- O^T += V^T P^T over two 32-key steps
#pragma unroll
                for (int st = 0; st < 2; ++st) {
                    const uint4 pb = make_uint4(pk[2 * st][0], pk[2 * st][1], pk[2 * st + 1][0],
                                                pk[2 * st + 1][1]);
                    const bf16x8 bop = __builtin_bit_cast(bf16x8, pb);
#pragma unroll
                    for (int db = 0; db < DB; ++db) {
                        const uint16_t* vrow = &sV[(db * 16 + li) * VROW + st * 32 + lg * 4];
                        const uint2 lo = *reinterpret_cast<const uint2*>(vrow);
                        const uint2 hi = *reinterpret_cast<const uint2*>(vrow + 16);
                        const uint4 av = make_uint4(lo.x, lo.y, hi.x, hi.y);
                        o[blk][db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                            __builtin_bit_cast(bf16x8, av), bop, o[blk][db], 0, 0, 0);
                    }
                }
            }
        }
        __syncthreads();
    }

    // ---- epilogue
#pragma unroll
    for (int blk = 0; blk < 2; ++blk) {
        float l = l_run[blk];
        l += __shfl_xor(l, 16, kWave);
        l += __shfl_xor(l, 32, kWave);
        const int rho = row0 + blk * 16 + li;
        if (rho >= a.G * a.n_max) continue;
        const int n = rho / a.G, hh = rho - n * a.G;
        if (a.splits == 1) {
            uint16_t* op = a.out + (((int64_t)b * a.n_max + n) * a.hq + g * a.G + hh) * D;
            const bool live = rho < live_rows;
            const float inv = live && l > 0.f ? 1.f / l : 0.f;
#pragma unroll
            for (int db = 0; db < DB; ++db) {
                const floatx4 v = o[blk][db] * inv;
                uint2 w;
                w.x = (uint32_t)f_to_bf16(v[0]) | ((uint32_t)f_to_bf16(v[1]) << 16);
                w.y = (uint32_t)f_to_bf16(v[2]) | ((uint32_t)f_to_bf16(v[3]) << 16);
                *reinterpret_cast<uint2*>(op + db * 16 + lg * 4) = w;
            }
        } else {
            float* pp = a.part + ((((int64_t)b * a.hkv + g) * a.rows_pad + rho) * a.splits + split) * (D + 2);
#pragma unroll
            for (int db = 0; db < DB; ++db)
                *reinterpret_cast<floatx4*>(pp + db * 16 + lg * 4) = o[blk][db];
            if (lg == 0) {
                pp[D] = m_run[blk];
                pp[D + 1] = l;
            }
        }
    }
}

// Merge of the split partials: one thread per (row, 4 output dims).
template <int D>
__global__ __launch_bounds__(256) void tree_attn_merge_kernel(AttnArgs a) {
    const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    constexpr int Q = D / 4;
    const int64_t rows = (int64_t)a.batch * a.hkv * a.G * a.n_max;
    if (gid >= rows * Q) return;
    const int q4 = (int)(gid % Q);
    const int64_t r = gid / Q;
    const int rho = (int)(r % (a.G * a.n_max));
    const int g = (int)((r / (a.G * a.n_max)) % a.hkv);
    const int b = (int)(r / ((int64_t)a.G * a.n_max * a.hkv));
    const int n = rho / a.G, hh = rho - n * a.G;
    const int nn = clamp_nodes(a.n_nodes[b], a.n_max);
    uint16_t* op = a.out + (((int64_t)b * a.n_max + n) * a.hq + g * a.G + hh) * D + q4 * 4;
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    if (rho < a.G * nn) {
        const int keys = a.ctx_off[b + 1] - a.ctx_off[b] + nn;
        const int nsplit = min(a.splits, (keys + a.split_len - 1) / a.split_len);
        const float* pp = a.part + (((int64_t)b * a.hkv + g) * a.rows_pad + rho) * a.splits * (D + 2);
        float M = -INFINITY;
        for (int s = 0; s < nsplit; ++s) M = fmaxf(M, pp[s * (D + 2) + D]);
        float L = 0.f;
        for (int s = 0; s < nsplit; ++s) {
            const float* ps = pp + s * (D + 2);
            const float w = ps[D] == -INFINITY ? 0.f : exp2f(ps[D] - M);
            L += w * ps[D + 1];
            const floatx4 v = *reinterpret_cast<const floatx4*>(ps + q4 * 4);
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[e] += w * v[e];
        }
        const float inv = L > 0.f ? 1.f / L : 0.f;
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[e] *= inv;
    }
    uint2 w;
    w.x = (uint32_t)f_to_bf16(acc[0]) | ((uint32_t)f_to_bf16(acc[1]) << 16);
    w.y = (uint32_t)f_to_bf16(acc[2]) | ((uint32_t)f_to_bf16(acc[3]) << 16);
    *reinterpret_cast<uint2*>(op) = w;
}

// fp32 path: one wave per (b, n, h) row, plain fp32 arithmetic.  Each lane
// runs an online softmax over a strided subset of keys; lanes are merged
// through LDS at the end.
template <int D>
__global__ __launch_bounds__(kWave) void tree_attn_f32_kernel(
    const float* __restrict__ q, const float* __restrict__ kc, const float* __restrict__ vc,
    const int32_t* __restrict__ ctx_off, const float* __restrict__ kt,
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
    const int c0 = ctx_off[b], ctx = ctx_off[b + 1] - c0;
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
    int G, rows, row_tiles, rows_per_tile, rows_pad, waves, splits, split_len;
    int64_t tasks, blocks;
};

static AttnPlan attn_plan(const presto_attn_desc* d) {
    AttnPlan p;
    p.G = d->hq / d->hkv;
    p.rows = p.G * d->n_max;
    p.row_tiles = (p.rows + kMaxRowsPerTile - 1) / kMaxRowsPerTile;
    const int per = (p.rows + p.row_tiles - 1) / p.row_tiles;
    p.rows_per_tile = (per + kRowsPerWave - 1) / kRowsPerWave * kRowsPerWave;
    p.waves = p.rows_per_tile / kRowsPerWave;
    p.rows_pad = p.rows_per_tile * p.row_tiles;
    const int64_t base = (int64_t)d->batch * d->hkv * p.row_tiles;
    const int keys = d->max_ctx + d->n_max;
    const int max_splits = (keys + 255) / 256;
    int splits = (int)((512 + base - 1) / base);
    splits = splits < 1 ? 1 : (splits > max_splits ? max_splits : splits);
    int len = (keys + splits - 1) / splits;
    len = (len + kKeyTile - 1) / kKeyTile * kKeyTile;
    p.split_len = len;
    p.splits = (keys + len - 1) / len;
    p.tasks = base * p.splits;
    p.blocks = (p.tasks + 7) / 8 * 8;
    return p;
}

size_t attn_workspace_bytes(const presto_attn_desc* d) {
    if (d->dt != PRESTO_DT_BF16) return 0;
    const AttnPlan p = attn_plan(d);
    if (p.splits <= 1) return 0;
    return (size_t)d->batch * d->hkv * p.rows_pad * p.splits * (d->head_dim + 2) * sizeof(float) + 256;
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
    a.kt = (const uint16_t*)k_tree;
    a.vt = (const uint16_t*)v_tree;
    a.anc = anc;
    a.n_nodes = n_nodes;
    a.out = (uint16_t*)out;
    a.part = (float*)ws;
    a.batch = d->batch;
    a.n_max = d->n_max;
    a.hq = d->hq;
    a.hkv = d->hkv;
    a.G = p.G;
    a.W = (d->n_max + 63) / 64;
    a.row_tiles = p.row_tiles;
    a.rows_per_tile = p.rows_per_tile;
    a.rows_pad = p.rows_pad;
    a.splits = p.splits;
    a.split_len = p.split_len;
    a.n_tasks = (int32_t)p.tasks;
    a.n_blocks = (int32_t)p.blocks;
    a.scale_log2 = d->scale * kLog2e;
    const dim3 block(p.waves * kWave);
    if (d->head_dim == 64)
        tree_attn_bf16_kernel<64><<<(unsigned)p.blocks, block, 0, stream>>>(a);
    else
        tree_attn_bf16_kernel<128><<<(unsigned)p.blocks, block, 0, stream>>>(a);
    presto_status st = check_launch("tree_attn_bf16_kernel");
    if (st != PRESTO_OK || p.splits == 1) return st;
    const int64_t threads = (int64_t)d->batch * d->hkv * p.G * d->n_max * (d->head_dim / 4);
    const unsigned grid = (unsigned)((threads + 255) / 256);
    if (d->head_dim == 64)
        tree_attn_merge_kernel<64><<<grid, 256, 0, stream>>>(a);
    else
        tree_attn_merge_kernel<128><<<grid, 256, 0, stream>>>(a);
    return check_launch("tree_attn_merge_kernel");
}

}  // namespace presto_host
