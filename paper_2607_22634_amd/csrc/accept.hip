// Stage 4: greedy verification of the tree and the bonus token.
//
// Kernel 1 streams every live node's target logit row from HBM once (rows of
// padding nodes are never read) and leaves, per wave-sized chunk, the chunk
// maximum and the lowest id holding it, packed into one orderable 64-bit
// key.  Kernel 2, queued right behind, runs one workgroup per sequence: its
// waves reduce the chunk keys of the live nodes to the target's greedy
// prediction a[n] (into LDS), then find the accepted root path in parallel
// (pointer jumping over the parent links) instead of walking it.
#include <math.h>

#include "common.hpp"

namespace presto {

constexpr int kArgmaxWavesPerBlock = 4;
constexpr int kWalkThreads = 1024;
constexpr int kMaxNodes = 1024;
constexpr int kNodesPerWave = 8;
constexpr int kKeyCols = 3;  // chunk keys per lane and node loaded at once

template <bool BF16, int NLOAD>
__global__ __launch_bounds__(kArgmaxWavesPerBlock * kWave) void argmax_partial_kernel(
    const void* __restrict__ logits, int32_t batch, int32_t n_max, int32_t vocab,
    int64_t row_stride, const int32_t* __restrict__ n_nodes, int32_t chunks, bool aligned,
    uint64_t* __restrict__ part, int32_t* __restrict__ flags) {
    constexpr int P = BF16 ? 8 : 4;
    constexpr int E = NLOAD * P;
    constexpr int64_t CH = (int64_t)kWave * E;
    const int wave = threadIdx.x / kWave, lane = lane_id();
    const int64_t gw = (int64_t)blockIdx.x * kArgmaxWavesPerBlock + wave;
    const int64_t rows = (int64_t)batch * n_max;
    if (gw >= rows * chunks) return;
    const int64_t row = gw / chunks;
    const int32_t chunk = (int32_t)(gw % chunks);
    const int b = (int)(row / n_max), n = (int)(row % n_max);
    if (n >= min(max(n_nodes[b], 1), n_max)) return;  // padding node: never read, never used
    const int64_t c0 = (int64_t)chunk * CH;
    const char* rowp = static_cast<const char*>(logits) + row * row_stride * (BF16 ? 2 : 4);
    const bool full = aligned && (c0 + CH <= vocab);

    float v[E];
    if (full) {
        const uint4* src = reinterpret_cast<const uint4*>(rowp + c0 * (BF16 ? 2 : 4));
        uint4 raw[NLOAD];
#pragma unroll
        for (int i = 0; i < NLOAD; ++i) raw[i] = load_stream16(&src[i * kWave + lane]);
#pragma unroll
        for (int i = 0; i < NLOAD; ++i) {
            const uint32_t w[4] = {raw[i].x, raw[i].y, raw[i].z, raw[i].w};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if constexpr (BF16) {
                    v[i * P + 2 * j] = bf16lo(w[j]);
                    v[i * P + 2 * j + 1] = bf16hi(w[j]);
                } else {
                    v[i * P + j] = __uint_as_float(w[j]);
                }
            }
        }
    } else {
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const int64_t idx = c0 + (int64_t)((e / P) * kWave + lane) * P + (e % P);
            float x = -INFINITY;
            if (idx < vocab)
                x = BF16 ? bf16_to_f(reinterpret_cast<const uint16_t*>(rowp)[idx])
                         : reinterpret_cast<const float*>(rowp)[idx];
            v[e] = x;
        }
    }
    // lane maximum with NaN propagation (a NaN anywhere in the lane makes it
    // NaN, which is how NaN rows are detected)
    float lm = v[0];
#pragma unroll
    for (int e = 1; e < E; ++e) lm = __builtin_elementwise_maximum(lm, v[e]);
    const bool nan_lane = !(lm == lm);
    const float M = wave_max_f32_dpp(nan_lane ? -INFINITY : lm);
    // lowest vocabulary id holding the chunk maximum: a lane's elements
    // ascend in id, so its candidate is its first element equal to M
    int first = E;
#pragma unroll
    for (int e = E - 1; e >= 0; --e) first = v[e] == M ? e : first;
    uint32_t best = 0xffffffffu;
    if (first < E) {
        const int64_t idx = c0 + (int64_t)((first / P) * kWave + lane) * P + (first % P);
        if (full || idx < vocab) best = (uint32_t)idx;
    }
    best = wave_min_u32_dpp(best);
    const bool any_nan = __ballot(nan_lane) != 0ull;
    if (lane == 0) {
        part[gw] = vocab_key(M, best);
        if (any_nan) raise_flag(flags, PRESTO_FLAG_NAN_TARGET);
    }
}

// One workgroup per sequence: per-node argmax from the chunk keys, then the
// accepted path without a sequential walk.  Node c is "good" when its token
// is the target's prediction after its parent, a[parent(c)]; siblings carry
// distinct tokens, so every node has at most one good child and the accepted
// path is the chain of nodes whose whole root path is good.  Pointer jumping
// (ceil(log2(depth + 1)) rounds) gives every node that property and its
// depth at once; the accepted nodes then write themselves into the path.
// The node count, parents and tokens are loaded together; the chunk keys of
// the live nodes are then all requested before the first is used, so the
// kernel waits for memory twice.
__global__ __launch_bounds__(kWalkThreads) void accept_walk_kernel(
    int32_t n_max, int32_t depth, int32_t chunks, const uint64_t* __restrict__ part,
    const int32_t* __restrict__ parent, const int32_t* __restrict__ token,
    const int32_t* __restrict__ n_nodes, int32_t* __restrict__ accept_len,
    int32_t* __restrict__ path, int32_t* __restrict__ bonus, int32_t* __restrict__ target_argmax) {
    __shared__ int32_t s_a[kMaxNodes];
    __shared__ int32_t s_jmp[2][kMaxNodes];
    __shared__ int32_t s_dep[2][kMaxNodes];  // edges to the jump target; -1: a bad node on the way
    __shared__ int32_t s_len;
    const int b = blockIdx.x;
    const int tid = threadIdx.x;
    const int wave = tid / kWave, lane = lane_id();
    const int nwaves = blockDim.x / kWave;
    const int64_t rb = (int64_t)b * n_max;
    // node tid's parent and token (blockDim.x >= n_max), and the node count
    const int my_par = tid < n_max ? parent[rb + tid] : 0;
    const int my_tok = tid < n_max ? token[rb + tid] : 0;
    const int nn_raw = n_nodes[b];
    if (tid == 0) s_len = 0;
    // each wave reduces the chunk keys of kNodesPerWave live nodes at a time,
    // up to kKeyCols chunk keys per lane and node with every load in flight
    // before the first reduction (one memory round trip for a 151936-entry
    // bf16 row); padding nodes have no keys (the argmax kernel skips them)
    const int nn = min(max(nn_raw, 1), n_max);
    for (int n0 = wave * kNodesPerWave; n0 < nn; n0 += nwaves * kNodesPerWave) {
        uint64_t best[kNodesPerWave];
#pragma unroll
        for (int u = 0; u < kNodesPerWave; ++u) best[u] = 0ull;
        for (int c0 = 0; c0 < chunks; c0 += kKeyCols * kWave) {
            uint64_t x[kKeyCols][kNodesPerWave];
#pragma unroll
            for (int t = 0; t < kKeyCols; ++t) {
                const int c = c0 + t * kWave + lane;
#pragma unroll
                for (int u = 0; u < kNodesPerWave; ++u)
                    x[t][u] = (c < chunks && n0 + u < nn) ? part[(rb + n0 + u) * chunks + c] : 0ull;
            }
#pragma unroll
            for (int t = 0; t < kKeyCols; ++t)
#pragma unroll
                for (int u = 0; u < kNodesPerWave; ++u) best[u] = x[t][u] > best[u] ? x[t][u] : best[u];
        }
#pragma unroll
        for (int u = 0; u < kNodesPerWave; ++u) {
            const uint64_t m = wave_max_u64_dpp(best[u]);
            if (lane == 0 && n0 + u < nn) s_a[n0 + u] = (int32_t)key_id(m);
        }
    }
    __syncthreads();
    if (tid < n_max) {
        if (target_argmax) target_argmax[rb + tid] = tid < nn ? s_a[tid] : -1;
        if (tid < nn) {
            // (a parent outside 0 .. nn-1 can only come from a malformed tree:
            // clamped, so that it costs a wrong answer, never a bad access)
            const int p = tid == 0 ? 0 : min(max(my_par, 0), nn - 1);
            const bool good = tid == 0 || my_tok == s_a[p];
            s_jmp[0][tid] = p;
            s_dep[0][tid] = good ? (tid == 0 ? 0 : 1) : -1;
        }
    }
    __syncthreads();
    int cur = 0;
    for (int reach = 1; reach < depth + 1; reach *= 2) {
        if (tid < nn) {
            const int j = s_jmp[cur][tid], dn = s_dep[cur][tid], dj = s_dep[cur][j];
            s_jmp[cur ^ 1][tid] = s_jmp[cur][j];
            s_dep[cur ^ 1][tid] = (dn < 0 || dj < 0) ? -1 : dn + dj;
        }
        cur ^= 1;
        __syncthreads();
    }
    // accepted nodes: a good root path no longer than `depth` moves
    int32_t* pth = path + (int64_t)b * (depth + 1);
    if (tid < nn) {
        const int dn = s_dep[cur][tid];
        if (dn >= 0 && dn <= depth) {
            pth[dn] = tid;
            atomicMax(&s_len, dn);
        }
    }
    __syncthreads();
    const int L = s_len;
    for (int i = L + 1 + tid; i <= depth; i += blockDim.x) pth[i] = -1;
    if (tid < nn && s_dep[cur][tid] == L) {
        accept_len[b] = L;
        bonus[b] = s_a[tid];
    }
}

}  // namespace presto

namespace presto_host {

using namespace presto;

static int argmax_nload(int64_t rows, int32_t vocab, bool bf16) {
    const int64_t ch8 = (int64_t)kWave * 8 * (bf16 ? 8 : 4);
    return rows * ((vocab + ch8 - 1) / ch8) >= 4 * 256 * 4 ? 8 : 4;
}

size_t accept_workspace_bytes(int32_t batch, int32_t n_max, int32_t vocab) {
    const int64_t chunks = (vocab + (int64_t)kWave * 16 - 1) / ((int64_t)kWave * 16);
    return (size_t)batch * n_max * chunks * sizeof(uint64_t) + 256;
}

presto_status launch_accept(bool bf16, const void* logits, int32_t vocab, int64_t row_stride,
                            int32_t batch, int32_t n_max, int32_t depth, const int32_t* parent,
                            const int32_t* token, const int32_t* n_nodes, int32_t* accept_len,
                            int32_t* path, int32_t* bonus, int32_t* target_argmax, int32_t* flags,
                            void* ws, hipStream_t stream) {
    const int64_t rows = (int64_t)batch * n_max;
    const int nload = argmax_nload(rows, vocab, bf16);
    const int64_t ch = (int64_t)kWave * nload * (bf16 ? 8 : 4);
    const int64_t chunks = (vocab + ch - 1) / ch;
    const size_t esz = bf16 ? 2 : 4;
    const bool aligned = ((uintptr_t)logits % 16 == 0) && ((row_stride * (int64_t)esz) % 16 == 0);
    uint64_t* part = static_cast<uint64_t*>(ws);
    const int64_t waves = rows * chunks;
    const dim3 block(kArgmaxWavesPerBlock * kWave);
    const dim3 grid((unsigned)((waves + kArgmaxWavesPerBlock - 1) / kArgmaxWavesPerBlock));
#define PRESTO_ARGMAX(BF, NL)                                                                  \
    argmax_partial_kernel<BF, NL><<<grid, block, 0, stream>>>(logits, batch, n_max, vocab,      \
                                                              row_stride, n_nodes,             \
                                                              (int32_t)chunks, aligned, part, flags)
    if (bf16) {
        if (nload == 8) PRESTO_ARGMAX(true, 8); else PRESTO_ARGMAX(true, 4);
    } else {
        if (nload == 8) PRESTO_ARGMAX(false, 8); else PRESTO_ARGMAX(false, 4);
    }
#undef PRESTO_ARGMAX
    presto_status st = check_launch("argmax_partial_kernel");
    if (st != PRESTO_OK) return st;
    // one thread per node (n_max <= 1024), at least 16 waves for the key reduction
    accept_walk_kernel<<<batch, kWalkThreads, 0, stream>>>(n_max, depth, (int32_t)chunks, part, parent,
                                                      token, n_nodes, accept_len, path, bonus,
                                                      target_argmax);
    return check_launch("accept_walk_kernel");
}

}  // namespace presto_host
