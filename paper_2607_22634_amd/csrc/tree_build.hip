// Stage 2: prefix-aligned scoring and best-first tree construction.
//
// One wavefront builds one sequence's tree; the batch runs in parallel.
// The candidate table (log q, token ids), lambda, the trigram lattice (when
// it fits), the per-node child tables and the ancestor bitmask rows live in
// LDS.  The frontier lives in registers, spread over the 64 lanes (SL slots
// per lane), so a pop is a per-lane scan plus one wave-wide max.
//
// Frontier policy.  Committing nodes in pop order yields the B best prefixes
// under the total order (S desc, rank path asc).  Instead of pushing all of
// a node's children at once, the frontier holds, for every committed node,
// only its next not-yet-committed child in that order: committing a node
// pushes its first child, committing a child pushes its next sibling.  The
// best uncommitted prefix always has a committed parent and committed
// better siblings, so it is always in the frontier; the frontier never
// holds more than (committed + 1) entries.
#include <math.h>

#include "common.hpp"

// Scores must round exactly as fl(log q + fl(lambda * log rho)) and
// fl(S(parent) + s): no fused multiply-add anywhere in this file.
#pragma clang fp contract(off)

namespace presto {

struct TreeArgs {
    int32_t D, k, branch, budget, N, W, wbits;
    const int32_t* ids;
    const float* logprob;
    const float* log_rho;
    const float* lambda;
    const int32_t* root_token;
    int32_t* n_nodes;
    int32_t* parent;
    int32_t* token;
    int32_t* depth;
    int32_t* rank;
    float* score;
    uint64_t* anc;
    bool rho_in_lds;
    // LDS byte offsets
    int o_lp, o_ids, o_lam, o_rho, o_dep, o_rank, o_prank, o_crank, o_cs, o_anc;
};

// 128-bit rank-path key as (hi, lo); digit (rank + 1) of depth d (1-based)
// sits wbits wide at bit 128 - d * wbits, so a prefix sorts before its
// extensions and siblings sort by rank.
__device__ __forceinline__ void key_set_digit(uint64_t& hi, uint64_t& lo, int d, int wbits,
                                              uint32_t digit) {
    const int shift = 128 - d * wbits;
    const uint64_t mask = (1ull << wbits) - 1ull;
    if (shift >= 64) {
        hi = (hi & ~(mask << (shift - 64))) | ((uint64_t)digit << (shift - 64));
    } else {
        lo = (lo & ~(mask << shift)) | ((uint64_t)digit << shift);
        if (shift + wbits > 64) {
            const int up = 64 - shift;  // bits of the digit that spill into hi
            hi = (hi & ~(mask >> up)) | ((uint64_t)digit >> up);
        }
    }
}

__device__ __forceinline__ bool entry_before(uint32_t sa, uint64_t ha, uint64_t la, uint32_t sb,
                                             uint64_t hb, uint64_t lb) {
    if (sa != sb) return sa > sb;
    if (ha != hb) return ha < hb;
    return la < lb;
}

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const uint64_t w = shfl_xor_u64(v, o);
        v = w < v ? w : v;
    }
    return v;
}

__device__ __forceinline__ float rd_f(float x, int lane) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), lane));
}

// Child table of node n (depth d, own rank rn, parent's rank rp, score Sn):
// the top-`branch` candidates by token score, stored in the order in which
// the best-first search will commit them (child S desc, rank asc).
__device__ __forceinline__ void expand_node(const TreeArgs& a, char* lds, int n, int d, int rn,
                                            int rp, float Sn) {
    const int lane = lane_id();
    const float* s_lp = reinterpret_cast<const float*>(lds + a.o_lp);
    const float* s_lam = reinterpret_cast<const float*>(lds + a.o_lam);
    uint8_t* s_crank = reinterpret_cast<uint8_t*>(lds + a.o_crank);
    float* s_cs = reinterpret_cast<float*>(lds + a.o_cs);
    const int k = a.k, row = d;
    const int ctx2 = d >= 2 ? rp : 0;  // grandparent slot of the trigram
    const int ctx1 = d >= 1 ? rn : 0;  // parent slot of the trigram
    float s = -INFINITY;
    if (lane < k) {
        const float lq = s_lp[row * k + lane];
        if (a.log_rho) {
            const int64_t ri = (((int64_t)row * k + ctx2) * k + ctx1) * k + lane;
            const float lr = a.rho_in_lds ? reinterpret_cast<const float*>(lds + a.o_rho)[ri]
                                          : a.log_rho[ri];
            const float t = s_lam[row] * lr;
            s = lq + t;
        } else {
            s = lq;
        }
        s = (s == s) ? s : -INFINITY;
    }
    // selection by token score: larger s first, lower rank on ties
    int sel = 0;
    for (int j = 0; j < k; ++j) {
        const float sj = rd_f(s, j);
        sel += (sj > s || (sj == s && j < lane)) ? 1 : 0;
    }
    const bool in_set = lane < k && sel < a.branch;
    const float sc = Sn + s;
    // commit order among the chosen children: child S desc, rank asc
    int pos = 0;
    for (int j = 0; j < k; ++j) {
        const float cj = rd_f(sc, j);
        const int selj = __builtin_amdgcn_readlane(sel, j);
        if (selj < a.branch) pos += (cj > sc || (cj == sc && j < lane)) ? 1 : 0;
    }
    if (in_set) {
        s_crank[n * a.branch + pos] = (uint8_t)lane;
        s_cs[n * a.branch + pos] = sc;
    }
    __builtin_amdgcn_wave_barrier();
}

template <int SL>
__global__ __launch_bounds__(kWave) void tree_build_kernel(TreeArgs a) {
    extern __shared__ __align__(16) char lds[];
    const int lane = lane_id();
    const int b = blockIdx.x;
    const int D = a.D, k = a.k, N = a.N, W = a.W;
    float* s_lp = reinterpret_cast<float*>(lds + a.o_lp);
    int32_t* s_ids = reinterpret_cast<int32_t*>(lds + a.o_ids);
    float* s_lam = reinterpret_cast<float*>(lds + a.o_lam);
    int32_t* s_dep = reinterpret_cast<int32_t*>(lds + a.o_dep);
    int32_t* s_rank = reinterpret_cast<int32_t*>(lds + a.o_rank);
    int32_t* s_prank = reinterpret_cast<int32_t*>(lds + a.o_prank);
    const uint8_t* s_crank = reinterpret_cast<const uint8_t*>(lds + a.o_crank);
    const float* s_cs = reinterpret_cast<const float*>(lds + a.o_cs);
    uint64_t* s_anc = reinterpret_cast<uint64_t*>(lds + a.o_anc);

    // stage the candidate table of this sequence
    const int64_t tb = (int64_t)b * D * k;
    for (int i = lane; i < D * k; i += kWave) {
        s_lp[i] = a.logprob[tb + i];
        s_ids[i] = a.ids[tb + i];
    }
    for (int i = lane; i < D; i += kWave) s_lam[i] = a.lambda[i];
    if (a.log_rho && a.rho_in_lds) {
        float* s_rho = reinterpret_cast<float*>(lds + a.o_rho);
        const int64_t rn = (int64_t)D * k * k * k;
        const float* src = a.log_rho + (int64_t)b * rn;
        for (int64_t i = lane; i < rn; i += kWave) s_rho[i] = src[i];
    }
    for (int i = lane; i < N * W; i += kWave) s_anc[i] = 0ull;
    __builtin_amdgcn_wave_barrier();

    int32_t* o_par = a.parent + (int64_t)b * N;
    int32_t* o_tok = a.token + (int64_t)b * N;
    int32_t* o_dep = a.depth + (int64_t)b * N;
    int32_t* o_rank = a.rank + (int64_t)b * N;
    float* o_score = a.score + (int64_t)b * N;
    uint64_t* o_anc = a.anc + (int64_t)b * N * W;

    // root
    if (lane == 0) {
        s_dep[0] = 0;
        s_rank[0] = 0;
        s_prank[0] = 0;
        s_anc[0] = 1ull;
        o_par[0] = -1;
        o_tok[0] = a.root_token[b];
        o_dep[0] = 0;
        o_rank[0] = -1;
        o_score[0] = 0.f;
    }
    for (int w = lane; w < W; w += kWave) o_anc[w] = w == 0 ? 1ull : 0ull;
    __builtin_amdgcn_wave_barrier();
    expand_node(a, lds, 0, 0, 0, 0, 0.f);

    // frontier slots: slot j of lane l is entry j * 64 + l
    uint32_t fS[SL];
    uint64_t fH[SL], fL[SL];
    int32_t fP[SL], fO[SL];
#pragma unroll
    for (int j = 0; j < SL; ++j) {
        fS[j] = 0u;
        fH[j] = fL[j] = 0ull;
        fP[j] = fO[j] = 0;
    }
    if (lane == 0 && D > 0) {
        uint64_t h = 0, l = 0;
        key_set_digit(h, l, 1, a.wbits, (uint32_t)s_crank[0] + 1u);
        fS[0] = ord32(s_cs[0]);
        fH[0] = h;
        fL[0] = l;
        fP[0] = 0;
        fO[0] = 0;
    }
    int fcount = 1;
    int committed = 1;

    while (committed - 1 < a.budget) {
        // best entry of this lane
        uint32_t bS = 0u;
        uint64_t bH = ~0ull, bL = ~0ull;
        int bP = 0, bO = 0, bSlot = 0;
#pragma unroll
        for (int j = 0; j < SL; ++j) {
            if (fS[j] != 0u && entry_before(fS[j], fH[j], fL[j], bS, bH, bL)) {
                bS = fS[j];
                bH = fH[j];
                bL = fL[j];
                bP = fP[j];
                bO = fO[j];
                bSlot = j;
            }
        }
        const uint32_t mS = wave_max_u32(bS);
        if (mS == 0u) break;  // frontier exhausted: the whole candidate tree is committed
        uint64_t tied = __ballot(bS == mS);
        int w;
        if (__popcll(tied) == 1) {
            w = __ffsll((unsigned long long)tied) - 1;
        } else {
            const bool t1 = bS == mS;
            const uint64_t mh = wave_min_u64(t1 ? bH : ~0ull);
            const bool t2 = t1 && bH == mh;
            const uint64_t ml = wave_min_u64(t2 ? bL : ~0ull);
            w = __ffsll((unsigned long long)__ballot(t2 && bL == ml)) - 1;
        }
        const uint64_t eH = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(bH >> 32), w) << 32) |
                            (uint32_t)__builtin_amdgcn_readlane((int)bH, w);
        const uint64_t eL = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(bL >> 32), w) << 32) |
                            (uint32_t)__builtin_amdgcn_readlane((int)bL, w);
        const int p = __builtin_amdgcn_readlane(bP, w);
        const int o = __builtin_amdgcn_readlane(bO, w);
        const int eslot = __builtin_amdgcn_readlane(bSlot, w);

        // commit node n
        const int n = committed;
        const int r = s_crank[p * a.branch + o];
        const int d = s_dep[p] + 1;
        const float S = s_cs[p * a.branch + o];
        const int rp = s_rank[p];
        if (lane == 0) {
            s_dep[n] = d;
            s_rank[n] = r;
            s_prank[n] = rp;
            o_par[n] = p;
            o_tok[n] = s_ids[(d - 1) * k + r];
            o_dep[n] = d;
            o_rank[n] = r;
            o_score[n] = S;
        }
        for (int ww = lane; ww < W; ww += kWave) {
            uint64_t word = s_anc[p * W + ww];
            if (ww == (n >> 6)) word |= 1ull << (n & 63);
            s_anc[n * W + ww] = word;
            o_anc[(int64_t)n * W + ww] = word;
        }
        ++committed;
        __builtin_amdgcn_wave_barrier();

        // pushes: the first child of n, then the next sibling of n
        bool has_child = d < D;
        if (has_child) expand_node(a, lds, n, d, r, rp, S);
        const bool has_sib = o + 1 < a.branch;
        uint32_t cS = 0u, sS = 0u;
        uint64_t cH = eH, cL = eL, sH = eH, sL = eL;
        if (has_child) {
            cS = ord32(s_cs[n * a.branch]);
            key_set_digit(cH, cL, d + 1, a.wbits, (uint32_t)s_crank[n * a.branch] + 1u);
        }
        if (has_sib) {
            sS = ord32(s_cs[p * a.branch + o + 1]);
            key_set_digit(sH, sL, d, a.wbits, (uint32_t)s_crank[p * a.branch + o + 1] + 1u);
        }
        // first push reuses the popped slot, the second takes a fresh slot
        uint32_t xS = 0u;
        uint64_t xH = 0, xL = 0;
        int xP = 0, xO = 0;
        bool second = false;
        uint32_t yS = 0u;
        uint64_t yH = 0, yL = 0;
        int yP = 0, yO = 0;
        if (has_child) {
            xS = cS; xH = cH; xL = cL; xP = n; xO = 0;
            if (has_sib) {
                second = true;
                yS = sS; yH = sH; yL = sL; yP = p; yO = o + 1;
            }
        } else if (has_sib) {
            xS = sS; xH = sH; xL = sL; xP = p; xO = o + 1;
        }
        const int ylane = fcount & (kWave - 1), yslot = fcount >> 6;
#pragma unroll
        for (int j = 0; j < SL; ++j) {
            if (lane == w && j == eslot) {
                fS[j] = xS; fH[j] = xH; fL[j] = xL; fP[j] = xP; fO[j] = xO;
            }
            if (second && lane == ylane && j == yslot) {
                fS[j] = yS; fH[j] = yH; fL[j] = yL; fP[j] = yP; fO[j] = yO;
            }
        }
        if (second) ++fcount;
    }

    // padding rows
    for (int i = committed + lane; i < N; i += kWave) {
        o_par[i] = -1;
        o_tok[i] = -1;
        o_dep[i] = -1;
        o_rank[i] = -1;
        o_score[i] = -INFINITY;
    }
    for (int64_t i = (int64_t)committed * W + lane; i < (int64_t)N * W; i += kWave) o_anc[i] = 0ull;
    if (lane == 0) a.n_nodes[b] = committed;
}

}  // namespace presto

namespace presto_host {

using namespace presto;

static int align16(int x) { return (x + 15) & ~15; }

struct TreeLayout {
    int total_no_rho, total_with_rho;
    int o_lp, o_ids, o_lam, o_dep, o_rank, o_prank, o_crank, o_cs, o_anc, o_rho;
};

static TreeLayout tree_layout(int D, int k, int branch, int N) {
    TreeLayout L;
    const int W = (N + 63) / 64;
    int off = 0;
    L.o_lp = off; off = align16(off + D * k * 4);
    L.o_ids = off; off = align16(off + D * k * 4);
    L.o_lam = off; off = align16(off + D * 4);
    L.o_dep = off; off = align16(off + N * 4);
    L.o_rank = off; off = align16(off + N * 4);
    L.o_prank = off; off = align16(off + N * 4);
    L.o_crank = off; off = align16(off + N * branch);
    L.o_cs = off; off = align16(off + N * branch * 4);
    L.o_anc = off; off = align16(off + N * W * 8);
    L.total_no_rho = off;
    L.o_rho = off;
    L.total_with_rho = align16(off + D * k * k * k * 4);
    return L;
}

static constexpr int kTreeLdsBudget = 64 * 1024;

bool tree_build_fits(int D, int k, int branch, int N) {
    return tree_layout(D, k, branch, N).total_no_rho <= kTreeLdsBudget;
}

presto_status launch_build_tree(const presto_tree_desc* desc, const int32_t* ids,
                                const float* logprob, const float* log_rho, const float* lambda,
                                const int32_t* root_token, int32_t* n_nodes, int32_t* parent,
                                int32_t* token, int32_t* depth, int32_t* rank, float* score,
                                uint64_t* anc, hipStream_t stream) {
    TreeArgs a;
    a.D = desc->depth;
    a.k = desc->k;
    a.branch = desc->branch;
    a.budget = desc->budget;
    a.N = desc->budget + 1;
    a.W = (a.N + 63) / 64;
    int wbits = 1;
    while ((1 << wbits) < a.k + 1) ++wbits;
    a.wbits = wbits;
    a.ids = ids;
    a.logprob = logprob;
    a.log_rho = log_rho;
    a.lambda = lambda;
    a.root_token = root_token;
    a.n_nodes = n_nodes;
    a.parent = parent;
    a.token = token;
    a.depth = depth;
    a.rank = rank;
    a.score = score;
    a.anc = anc;
    const TreeLayout L = tree_layout(a.D, a.k, a.branch, a.N);
    a.o_lp = L.o_lp; a.o_ids = L.o_ids; a.o_lam = L.o_lam; a.o_dep = L.o_dep;
    a.o_rank = L.o_rank; a.o_prank = L.o_prank; a.o_crank = L.o_crank; a.o_cs = L.o_cs;
    a.o_anc = L.o_anc; a.o_rho = L.o_rho;
    a.rho_in_lds = log_rho != nullptr && L.total_with_rho <= kTreeLdsBudget;
    const int lds = a.rho_in_lds ? L.total_with_rho : L.total_no_rho;
    const int SL = (a.N + kWave - 1) / kWave;
#define PRESTO_TREE(S) tree_build_kernel<S><<<desc->batch, kWave, lds, stream>>>(a)
    if (SL <= 1) PRESTO_TREE(1);
    else if (SL <= 2) PRESTO_TREE(2);
    else if (SL <= 4) PRESTO_TREE(4);
    else PRESTO_TREE(8);
#undef PRESTO_TREE
    return check_launch("tree_build_kernel");
}

}  // namespace presto_host
