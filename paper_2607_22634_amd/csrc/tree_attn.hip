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
// bf16 path (matrix cores, v_mfma_f32_32x32x16_bf16).  A workgroup is four
// waves, one per SIMD, each owning 64 query rows (two 32-row MFMA blocks, so
// every K/V fragment read from LDS feeds two MFMAs).  Scores are computed
// transposed, S^T = K Q^T: a lane then holds one query row and 16 of the 32
// keys of a block, the row max/sum need one cross-half swap, and the bf16
// probabilities are already in the B-operand layout of O^T = V^T P^T.  K and
// V sit in LDS row-major; the V^T operand comes from transposed LDS reads
// (ds_read_b64_tr_b16).  The next K/V tile is fetched into registers while
// the current one is consumed.  The context is split across workgroups when
// the batch alone cannot fill the chip; partial (max, sum, accumulator)
// triples are then merged by a second kernel.
#include <math.h>

#include "common.hpp"

namespace presto {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef short short4_t __attribute__((ext_vector_type(4)));

constexpr int kKeyTile = 64;      // keys per LDS tile
constexpr int kRowsPerWave = 64;  // two 32-row MFMA blocks per wave
constexpr int kAttnWaves = 4;     // one wave per SIMD (about 300 registers each)
constexpr int kAttnThreads = kAttnWaves * kWave;
constexpr int kRowsPerTile = kAttnWaves * kRowsPerWave;
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
    int32_t row_tiles, rows_pad, splits, split_len;
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
__global__ __launch_bounds__(kAttnThreads, 1) void tree_attn_bf16_kernel(AttnArgs a) {
    constexpr int KS = D / 16;                 // S^T contraction steps over the head dimension
    constexpr int DB = D / 32;                 // 32-wide blocks of the output head dimension
    constexpr int KROW = D + 8;                // K row in LDS (bf16): bank spread for b128 reads
    constexpr int VROW = D + 16;               // V row in LDS: bank spread for transposed reads
    constexpr int PIECES = kKeyTile * D / 8;   // 16-byte pieces of one K (or V) tile
    constexpr int PT = PIECES / kAttnThreads;  // pieces per thread
    __shared__ __align__(16) uint16_t sK[kKeyTile * KROW];
    __shared__ __align__(16) uint16_t sV[kKeyTile * VROW];

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
    const int all_rows = a.G * a.n_max;

    const int tid = threadIdx.x;
    const int wave = tid / kWave, lane = lane_id();
    const int l32 = lane & 31, h = lane >> 5;
    const int rbase = rt * kRowsPerTile + wave * kRowsPerWave;  // two 32-row blocks per wave
    const bool active = rbase < live_rows;

    // Q fragments, B operand of S^T = K Q^T: lane holds row l32, d = ks*16 + h*8 .. +8
    bf16x8 qf[2][KS];
    int node_of[2];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
        const int rho = rbase + nb * 32 + l32;
        const int n = rho / a.G, hh = rho - n * a.G;
        node_of[nb] = min(n, a.n_max - 1);
        const uint16_t* qp = a.q + (((int64_t)b * a.n_max + n) * a.hq + g * a.G + hh) * D;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            uint4 u = make_uint4(0, 0, 0, 0);
            if (rho < all_rows) u = *reinterpret_cast<const uint4*>(qp + ks * 16 + h * 8);
            qf[nb][ks] = __builtin_bit_cast(bf16x8, u);
        }
    }

    floatx16 o[2][DB];
    float m_run[2], l_run[2];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
        m_run[nb] = -INFINITY;
        l_run[nb] = 0.f;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int i = 0; i < 16; ++i) o[nb][db][i] = 0.f;
    }

    // K/V tile staging: PT 16-byte pieces of K and of V per thread, fetched into
    // registers one tile ahead and written to LDS row-major.
    const int64_t kv_stride = (int64_t)a.hkv * D;
    uint4 kreg[PT], vreg[PT];
    auto fetch = [&](int t0) {
#pragma unroll
        for (int i = 0; i < PT; ++i) {
            const int p = tid + i * kAttnThreads;
            const int kk = p / (D / 8), c8 = p % (D / 8);
            const int jr = t0 + kk;
            const int j = min(jr, k_end - 1);  // clamped: every load is in bounds
            const bool in_ctx = j < ctx;
            const int64_t off = in_ctx
                ? (int64_t)(c0 + j) * kv_stride + (int64_t)g * D + c8 * 8
                : (((int64_t)b * a.n_max + (j - ctx)) * a.hkv + g) * D + c8 * 8;
            const uint4 ku = *reinterpret_cast<const uint4*>((in_ctx ? a.kc : a.kt) + off);
            const uint4 vu = *reinterpret_cast<const uint4*>((in_ctx ? a.vc : a.vt) + off);
            const bool ok = jr < k_end;
            kreg[i] = ok ? ku : make_uint4(0, 0, 0, 0);
            vreg[i] = ok ? vu : make_uint4(0, 0, 0, 0);
        }
    };
    auto stage = [&]() {
#pragma unroll
        for (int i = 0; i < PT; ++i) {
            const int p = tid + i * kAttnThreads;
            const int kk = p / (D / 8), c8 = p % (D / 8);
            *reinterpret_cast<uint4*>(&sK[kk * KROW + c8 * 8]) = kreg[i];
            *reinterpret_cast<uint4*>(&sV[kk * VROW + c8 * 8]) = vreg[i];
        }
    };

    fetch(k_begin);
    for (int t0 = k_begin; t0 < k_end; t0 += kKeyTile) {
        __syncthreads();  // the previous tile has been consumed
        stage();
        __syncthreads();
        if (t0 + kKeyTile < k_end) fetch(t0 + kKeyTile);
        if (!active) continue;
        const bool plain = t0 + kKeyTile <= min(ctx, k_end);  // no mask inside this tile
        // ancestor words covering the tree keys of this tile, per row block
        uint64_t aw[2][2] = {{0ull, 0ull}, {0ull, 0ull}};
        int wbase = 0;
        if (!plain && t0 + kKeyTile > ctx) {
            wbase = max(0, t0 - ctx) >> 6;
#pragma unroll
            for (int nb = 0; nb < 2; ++nb) {
                const uint64_t* arow = a.anc + ((int64_t)b * a.n_max + node_of[nb]) * a.W;
                aw[nb][0] = arow[wbase];
                aw[nb][1] = wbase + 1 < a.W ? arow[wbase + 1] : 0ull;
            }
        }
#pragma unroll
        for (int kb = 0; kb < kKeyTile / 32; ++kb) {
            // ---- S^T (32 keys x 64 rows): A = K rows from LDS, B = Q fragments
            floatx16 s[2];
#pragma unroll
            for (int nb = 0; nb < 2; ++nb)
#pragma unroll
                for (int i = 0; i < 16; ++i) s[nb][i] = 0.f;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const uint4 u = *reinterpret_cast<const uint4*>(
                    &sK[(kb * 32 + l32) * KROW + ks * 16 + h * 8]);
                const bf16x8 ka = __builtin_bit_cast(bf16x8, u);
                s[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[0][ks], s[0], 0, 0, 0);
                s[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[1][ks], s[1], 0, 0, 0);
            }
            // ---- online softmax; element i of lane holds key 8(i/4) + 4h + i%4 of the block
            uint32_t pk[2][8];
#pragma unroll
            for (int nb = 0; nb < 2; ++nb) {
                float mx = -INFINITY;
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    float v = s[nb][i] * a.scale_log2;
                    if (!plain) {
                        // visible: inside the sequence, and a cached key or an ancestor
                        const int j = t0 + kb * 32 + 8 * (i >> 2) + 4 * h + (i & 3);
                        const int m = max(j - ctx, 0);
                        const uint64_t wd = ((m >> 6) - wbase) == 0 ? aw[nb][0] : aw[nb][1];
                        const bool anc_bit = (wd >> (m & 63)) & 1ull;
                        const bool vis = (j < k_end) & ((j < ctx) | anc_bit);
                        v = vis ? v : -INFINITY;
                    }
                    s[nb][i] = v;
                    mx = fmaxf(mx, v);
                }
                {
                    const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx),
                                                                     __float_as_uint(mx), false, false);
                    mx = fmaxf(mx, __uint_as_float(h == 0 ? sw[1] : sw[0]));
                }
                const float m_new = fmaxf(m_run[nb], mx);
                const float m_use = m_new == -INFINITY ? 0.f : m_new;
                const float alpha = __builtin_amdgcn_exp2f(m_run[nb] - m_use);
                m_run[nb] = m_new;
                float ls = 0.f;
#pragma unroll
                for (int i = 0; i < 16; i += 2) {
                    const float p0 = __builtin_amdgcn_exp2f(s[nb][i] - m_use);
                    const float p1 = __builtin_amdgcn_exp2f(s[nb][i + 1] - m_use);
                    ls += p0 + p1;
                    pk[nb][i >> 1] = (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)p0) |
                                     ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)p1) << 16);
                }
                l_run[nb] = l_run[nb] * alpha + ls;
                if (__ballot(alpha != 1.f)) {
#pragma unroll
                    for (int db = 0; db < DB; ++db) o[nb][db] *= alpha;
                }
            }
            // ---- O^T += V^T P^T over two 16-key steps; V^T fragments by transposed LDS reads
#pragma unroll
            for (int st = 0; st < 2; ++st) {
                bf16x8 pb[2];
#pragma unroll
                for (int nb = 0; nb < 2; ++nb)
                    pb[nb] = __builtin_bit_cast(
                        bf16x8, make_uint4(pk[nb][4 * st], pk[nb][4 * st + 1], pk[nb][4 * st + 2],
                                           pk[nb][4 * st + 3]));
                const int kbase = kb * 32 + st * 16 + 4 * h;
                const int t16 = lane & 15, dhalf = (lane >> 4) & 1;
#pragma unroll
                for (int db = 0; db < DB; ++db) {
                    const int d0 = db * 32 + dhalf * 16;
                    const uint16_t* v0 = &sV[(kbase + (t16 >> 2)) * VROW + d0 + 4 * (t16 & 3)];
                    const short4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                        (__attribute__((address_space(3))) short4_t*)(v0));
                    const short4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                        (__attribute__((address_space(3))) short4_t*)(v0 + 8 * VROW));
                    const bf16x8 va = __builtin_bit_cast(
                        bf16x8, make_uint4(__builtin_bit_cast(uint2, lo).x, __builtin_bit_cast(uint2, lo).y,
                                           __builtin_bit_cast(uint2, hi).x, __builtin_bit_cast(uint2, hi).y));
                    o[0][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb[0], o[0][db], 0, 0, 0);
                    o[1][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb[1], o[1][db], 0, 0, 0);
                }
            }
        }
    }

    // ---- epilogue: lane holds row l32 of each block, d = db*32 + 8(i/4) + 4h + i%4
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
        float l = l_run[nb];
        {
            const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(l), __float_as_uint(l),
                                                             false, false);
            l += __uint_as_float(h == 0 ? sw[1] : sw[0]);
        }
        const int rho = rbase + nb * 32 + l32;
        if (rho >= all_rows) continue;
        const int n = rho / a.G, hh = rho - n * a.G;
        if (a.splits == 1) {
            uint16_t* op = a.out + (((int64_t)b * a.n_max + n) * a.hq + g * a.G + hh) * D;
            const float inv = (rho < live_rows && l > 0.f) ? 1.f / l : 0.f;
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
                for (int q4 = 0; q4 < 4; ++q4) {
                    const int dd = db * 32 + 8 * q4 + 4 * h;
                    uint2 w;
                    w.x = (uint32_t)f_to_bf16(o[nb][db][4 * q4] * inv) |
                          ((uint32_t)f_to_bf16(o[nb][db][4 * q4 + 1] * inv) << 16);
                    w.y = (uint32_t)f_to_bf16(o[nb][db][4 * q4 + 2] * inv) |
                          ((uint32_t)f_to_bf16(o[nb][db][4 * q4 + 3] * inv) << 16);
                    *reinterpret_cast<uint2*>(op + dd) = w;
                }
        } else {
            float* pp = a.part + ((((int64_t)b * a.hkv + g) * a.rows_pad + rho) * a.splits + split) * (D + 2);
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
                for (int q4 = 0; q4 < 4; ++q4) {
                    const int dd = db * 32 + 8 * q4 + 4 * h;
                    *reinterpret_cast<float4*>(pp + dd) =
                        make_float4(o[nb][db][4 * q4], o[nb][db][4 * q4 + 1], o[nb][db][4 * q4 + 2],
                                    o[nb][db][4 * q4 + 3]);
                }
            if (h == 0) {
                pp[D] = m_run[nb];
                pp[D + 1] = l;
            }
        }
    }
}

// Merge of the split partials: one wave per query row; lanes first read the
// splits' (max, sum), then each lane combines its D/64 output dimensions.
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
        const int keys = a.ctx_off[b + 1] - a.ctx_off[b] + nn;
        const int nsplit = min(a.splits, (keys + a.split_len - 1) / a.split_len);
        const float* pp = a.part + (((int64_t)b * a.hkv + g) * a.rows_pad + rho) * a.splits * (D + 2);
        float ms = -INFINITY, ls = 0.f;
        for (int s = lane; s < nsplit; s += kWave) {
            ms = fmaxf(ms, pp[s * (D + 2) + D]);
        }
        const float M = wave_max_f32_dpp(ms);
        float wl = 0.f;  // this lane's split weight (lane s holds split s, s < 64)
        for (int s = lane; s < nsplit; s += kWave) {
            const float m = pp[s * (D + 2) + D];
            const float w = m == -INFINITY ? 0.f : exp2f(m - M);
            ls += w * pp[s * (D + 2) + D + 1];
            if (s < kWave) wl = w;
        }
        const float L = wave_sum_f32_dpp(ls);
        for (int s = 0; s < nsplit; ++s) {
            const float* ps = pp + s * (D + 2);
            const float m = ps[D];
            const float w = s < kWave ? __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wl), s))
                                      : (m == -INFINITY ? 0.f : exp2f(m - M));
#pragma unroll
            for (int e = 0; e < PER; ++e) acc[e] += w * ps[lane * PER + e];
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
    p.row_tiles = (p.rows + kRowsPerTile - 1) / kRowsPerTile;
    p.rows_per_tile = kRowsPerTile;
    p.waves = kAttnWaves;
    p.rows_pad = p.rows_per_tile * p.row_tiles;
    const int64_t base = (int64_t)d->batch * d->hkv * p.row_tiles;
    const int keys = d->max_ctx + d->n_max;
    const int max_splits = (keys + 255) / 256;
    int splits = (int)((384 + base - 1) / base);
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
    a.rows_pad = p.rows_pad;
    a.splits = p.splits;
    a.split_len = p.split_len;
    a.n_tasks = (int32_t)p.tasks;
    a.n_blocks = (int32_t)p.blocks;
    a.scale_log2 = d->scale * kLog2e;
    const dim3 block(kAttnThreads);
    if (d->head_dim == 64)
        tree_attn_bf16_kernel<64><<<(unsigned)p.blocks, block, 0, stream>>>(a);
    else
        tree_attn_bf16_kernel<128><<<(unsigned)p.blocks, block, 0, stream>>>(a);
    presto_status st = check_launch("tree_attn_bf16_kernel");
    if (st != PRESTO_OK || p.splits == 1) return st;
    const int64_t merge_rows = (int64_t)d->batch * d->hkv * p.G * d->n_max;
    const unsigned grid = (unsigned)((merge_rows + 3) / 4);
    if (d->head_dim == 64)
        tree_attn_merge_kernel<64><<<grid, 256, 0, stream>>>(a);
    else
        tree_attn_merge_kernel<128><<<grid, 256, 0, stream>>>(a);
    return check_launch("tree_attn_merge_kernel");
}

}  // namespace presto_host
