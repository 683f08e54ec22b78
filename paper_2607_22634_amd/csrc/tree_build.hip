// Stage 2: prefix-aligned scoring and best-first tree construction.
//
// One wavefront builds one sequence's tree; the batch runs in parallel.
// LDS holds the candidate table (log q, token ids), the trigram lattice when
// it fits, and per committed node one 8-byte record (parent, rank, depth, S)
// plus its children in commit order (ranked once, when the node is
// committed).  The frontier lives in registers spread over the 64 lanes (SL
// slots per lane), each slot only (S, packed metadata): a pop is a per-lane
// max, one DPP wave max and a ballot; the next sibling of a popped node is
// one LDS read.  Rank-path keys are only derived when several frontier
// entries share the best S (from the parent records, up to the nearest node
// whose key an earlier tie stored); token ids, the output rows and the
// ancestor bitmasks are produced after the search, in parallel over the
// nodes.
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

#include <type_traits>

#include "common.hpp"

// Scores must round exactly as fl(log q + fl(lambda * log rho)) and
// fl(S(parent) + s): no fused multiply-add anywhere in this file.
#pragma clang fp contract(off)

namespace presto {

constexpr int kBeamCandSlots = 4;  // beam search: W * k <= 4 * 64 candidates per depth

struct TreeArgs {
    int32_t D, k, branch, budget, N, W, wbits, per_word;
    const int32_t* ids;
    const float* logprob;
    const float* log_rho;
    const float* lambda;
    int32_t lambda_stride;  // 0: one lambda row shared by the batch, D: one per sequence
    const int32_t* root_token;
    int32_t* n_nodes;
    int32_t* parent;
    int32_t* token;
    int32_t* depth;
    int32_t* rank;
    float* score;
    uint64_t* anc;
    bool rho_in_lds;
    int32_t beam_width;  // beam search only
    // LDS byte offsets
    int o_lp, o_ids, o_kord, o_krank, o_rec, o_pkey, o_ktab, o_beam, o_kbeam, o_rho;
    // literal Alg. 2 only: T (capacity budget + branch - 1) in LDS
    int o_tmeta, o_tS, o_tkey, o_tplace;
    // frontier sweeps only: lambda, the sorted best set, the pending
    // prefixes and the parent positions
    int o_lam, o_sw_t, o_sw_p, o_sw_p2, o_sw_par, o_sw_cnt, o_sw_np;
    uint32_t mag_k, mag_k3;  // ceil(2^32 / k), ceil(2^32 / k^3) (k > 1): n / d = umulhi(n, mag) for n < 2^20
};

// Frontier metadata in one word: parent node (10 bits), candidate rank (4),
// depth (6), rank of the parent (4), position among the parent's children
// in commit order (4).
__device__ __forceinline__ uint32_t pack_meta(int p, int r, int d, int rp, int pos) {
    return (uint32_t)p | ((uint32_t)r << 10) | ((uint32_t)d << 14) | ((uint32_t)rp << 20) |
           ((uint32_t)pos << 24);
}

// Number of lanes of this lane's row of 16 holding a larger key (row
// rotations by 1..R, each another lane of the row exactly once).
template <int R>
__device__ __forceinline__ int row_count_greater(uint64_t key) {
    if constexpr (R == 0) {
        return 0;
    } else {
        return (dpp_u64<0x120 + R>(0ull, key) > key ? 1 : 0) + row_count_greater<R - 1>(key);
    }
}

// One compare-exchange layer of a bitonic sort, descending: lane i pairs
// with the lane that DPP control CTRL reads (i ^ m within the group), and
// the lower lane of the pair (bit LOWBIT of i clear) keeps the larger key.
template <int CTRL, int LOWBIT>
__device__ __forceinline__ uint64_t bitonic_layer(uint64_t key, int lane) {
    const uint64_t t = dpp_u64<CTRL>(0ull, key);
    const bool lower = ((lane >> LOWBIT) & 1) == 0;
    return (lower == (t > key)) ? t : key;
}

// Keys of lanes 0..7 of every row sorted descending in place (lane 0 of the
// group holds the largest): blocks of 2, 4, 8, each merged by a flip
// (i ^ (s - 1)) and half-cleaners (i ^ s/4, ..., i ^ 1).
__device__ __forceinline__ uint64_t sort8_desc(uint64_t key, int lane) {
    key = bitonic_layer<0xb1, 0>(key, lane);   // i ^ 1
    key = bitonic_layer<0x1b, 1>(key, lane);   // i ^ 3 (quad_perm [3,2,1,0])
    key = bitonic_layer<0xb1, 0>(key, lane);   // i ^ 1
    key = bitonic_layer<0x141, 2>(key, lane);  // i ^ 7 (row_half_mirror)
    key = bitonic_layer<0x4e, 1>(key, lane);   // i ^ 2
    key = bitonic_layer<0xb1, 0>(key, lane);   // i ^ 1
    return key;
}

// Same within this lane's quad (quad_perm rotations by 1, 2, 3).
__device__ __forceinline__ int quad_count_greater(uint64_t key) {
    return (dpp_u64<0x39>(0ull, key) > key ? 1 : 0) + (dpp_u64<0x4e>(0ull, key) > key ? 1 : 0) +
           (dpp_u64<0x93>(0ull, key) > key ? 1 : 0);
}

// Loads up to U words per lane of src[base ..] (batches of 64 words while
// fewer than n; indices clamped, so every load is unconditional) into r.
template <int U>
__device__ __forceinline__ void load_words(uint32_t (&r)[U], const uint32_t* src, int n, int base, int lane) {
#pragma unroll
    for (int u = 0; u < U; ++u)
        if (base + u * kWave < n) r[u] = src[min(base + u * kWave + lane, n - 1)];
}
template <int U>
__device__ __forceinline__ void store_words(uint32_t* dst, const uint32_t (&r)[U], int n, int base, int lane) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int i = base + u * kWave + lane;
        if (i < n) dst[i] = r[u];
    }
}

// Copies n 32-bit words from global memory to LDS with one wave, 16 loads
// in flight per lane before the first store.
__device__ __forceinline__ void stage_words(uint32_t* dst, const uint32_t* src, int n, int lane) {
    constexpr int U = 16;
    for (int base = 0; base < n; base += U * kWave) {
        uint32_t r[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int i = base + u * kWave + lane;
            r[u] = i < n ? src[i] : 0u;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int i = base + u * kWave + lane;
            if (i < n) dst[i] = r[u];
        }
    }
}

// x with lane l replaced by v (v and l are read from the first lane, so they
// are scalar operands whatever registers hold them).
__device__ __forceinline__ uint32_t write_lane(uint32_t x, uint32_t v, int l) {
    const uint32_t sv = (uint32_t)__builtin_amdgcn_readfirstlane(v);
    const uint32_t sl = (uint32_t)__builtin_amdgcn_readfirstlane(l);
    asm("v_writelane_b32 %0, %1, m0" : "+v"(x) : "s"(sv), "{m0}"(sl));
    return x;
}

// Number of frontier slots per lane a pop works on (a compile-time tag).
template <int A>
struct SlotCount {
    static constexpr int value = A;
};

// One entry of a beam (beam search): score, candidate rank, rank of its
// parent, and its place in rank-path order among the entries of its depth.
struct BeamEntry {
    float S;
    int32_t rank, prank, path;
};

// RHO: 0 no lattice (s = log q), 1 lattice staged in LDS, 2 lattice read
// from global memory.  KQ: k <= 4, children ranked within a quad.  BEAM:
// beam search with global retention (Alg. 1): a level-by-level beam pass
// fixes the retained set T, then the best-first pass below, restricted to
// T, emits TopB(T) in the total order.
template <int SL, int RHO, bool KQ, bool BEAM>
__global__ __launch_bounds__(kWave) void tree_build_kernel(TreeArgs a) {
    extern __shared__ __align__(16) char lds[];
    const int lane = lane_id();
    const int b = blockIdx.x;
    const int D = a.D, k = a.k, N = a.N, W = a.W, wbits = a.wbits, per_word = a.per_word;
    float* s_lp = reinterpret_cast<float*>(lds + a.o_lp);
    int32_t* s_ids = reinterpret_cast<int32_t*>(lds + a.o_ids);
    // children of every committed node in commit order: ord(S) (0 ends the
    // list) and candidate rank
    uint32_t* s_kord = reinterpret_cast<uint32_t*>(lds + a.o_kord);  // [N][k]
    uint8_t* s_krank = reinterpret_cast<uint8_t*>(lds + a.o_krank);  // [N][k]
    uint2* s_rec = reinterpret_cast<uint2*>(lds + a.o_rec);          // [N] (meta, S bits)
    float* s_rho = reinterpret_cast<float*>(lds + a.o_rho);
    const int rho_n = D * k * k * k;
    const float* g_rho = RHO ? a.log_rho + (int64_t)b * rho_n : nullptr;

    const float lam_lane =
        lane < D ? a.lambda[(int64_t)b * a.lambda_stride + lane] : 0.f;  // lambda_d held by lane d
    // stage the candidate table of this sequence (and the lattice when it
    // fits): the table, lambda and the lattice's first 1024 words are all
    // requested before the first store, so the common sizes cost one memory
    // round trip
    const int64_t tb = (int64_t)b * D * k;
    {
        const uint32_t* g_lp = reinterpret_cast<const uint32_t*>(a.logprob + tb);
        const uint32_t* g_ids = reinterpret_cast<const uint32_t*>(a.ids + tb);
        constexpr int UT = 8;  // D * k <= 512 words
        uint32_t r_lp[UT], r_ids[UT], r_rho[16];
        load_words(r_lp, g_lp, D * k, 0, lane);
        load_words(r_ids, g_ids, D * k, 0, lane);
        if constexpr (RHO == 1) load_words(r_rho, reinterpret_cast<const uint32_t*>(g_rho), rho_n, 0, lane);
        store_words(reinterpret_cast<uint32_t*>(s_lp), r_lp, D * k, 0, lane);
        store_words(reinterpret_cast<uint32_t*>(s_ids), r_ids, D * k, 0, lane);
        if constexpr (RHO == 1) {
            store_words(reinterpret_cast<uint32_t*>(s_rho), r_rho, rho_n, 0, lane);
            if (rho_n > 16 * kWave)
                stage_words(reinterpret_cast<uint32_t*>(s_rho) + 16 * kWave,
                            reinterpret_cast<const uint32_t*>(g_rho) + 16 * kWave, rho_n - 16 * kWave,
                            lane);
        }
    }
    __builtin_amdgcn_wave_barrier();

    // token score of candidate r at drafter row `row` under the trigram
    // context (ctx2, ctx1): fl(log q + fl(lambda * log rho)), NaN -> -inf
    auto token_score = [&](int row, int ctx2, int ctx1, int r) {
        const float lam_d = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(lam_lane), row));
        const float lq = s_lp[row * k + r];
        float s = lq;
        if constexpr (RHO != 0) {
            const int ri = ((row * k + ctx2) * k + ctx1) * k + r;
            float lr;
            if constexpr (RHO == 1)
                lr = s_rho[ri];
            else
                lr = g_rho[ri];
            const float t = lam_d * lr;
            s = lq + t;
        }
        return (s == s) ? s : -INFINITY;
    };

    // ---- beam pass (Alg. 1): per depth, every beam entry's top-`branch`
    // children join T; the W best (total order) form the next beam.  The
    // table ktab[d][beam entry of the parent][rank] records, for every node of
    // depth d, whether it is in T (-1) and if so whether it is in the beam of
    // its depth (its index there, >= 0); -2: not in T.
    int8_t* s_ktab = reinterpret_cast<int8_t*>(lds + a.o_ktab);
    BeamEntry* s_beam = reinterpret_cast<BeamEntry*>(lds + a.o_beam);  // [2][Wb]
    // [N][k]: the table entry above of every child of a committed node, by
    // candidate rank (written when the node is expanded)
    int8_t* s_kbeam = reinterpret_cast<int8_t*>(lds + a.o_kbeam);
    const int Wb = a.beam_width;
    if constexpr (BEAM) {
        const int tab = (D + 1) * Wb * k;
        for (int i = lane; i < tab; i += kWave) s_ktab[i] = -2;
        if (lane == 0) s_beam[0] = BeamEntry{0.f, 0, 0, 0};  // the root
        __builtin_amdgcn_wave_barrier();
        int nb = 1, cur = 0, nT = 0;
        constexpr int CS = kBeamCandSlots;
        // One depth: candidates c = q * 64 + lane of the nb beam entries
        // (nb * k of them, in ceil(nb * k / 64) <= CS slots per lane: the
        // per-slot work only covers the slots that hold candidates).
        auto beam_depth = [&](auto act, int d) {
            constexpr int A = decltype(act)::value;
            const int row = d - 1;  // drafter row of depth d
            const BeamEntry* bc = s_beam + cur * Wb;
            uint64_t key[CS];
            int cpb[CS], cr[CS];
            int count = 0;
#pragma unroll
            for (int q = 0; q < A; ++q) {
                const int ci = q * kWave + lane;
                const bool valid = ci < nb * k;
                const int pb = valid ? ci / k : 0, r = valid ? ci % k : 0;
                const BeamEntry e = bc[pb];
                const float sv = token_score(row, row >= 2 ? e.prank : 0, row >= 1 ? e.rank : 0, r);
                bool in = valid;
                if (a.branch < k) {
                    // top-`branch` of the parent's k candidates by token score
                    int sel = 0;
                    for (int j = 0; j < k; ++j) {
                        const float sj = token_score(row, row >= 2 ? e.prank : 0, row >= 1 ? e.rank : 0, j);
                        sel += (sj > sv || (sj == sv && j < r)) ? 1 : 0;
                    }
                    in = in && sel < a.branch;
                }
                const float S = e.S + sv;
                key[q] = in ? ((uint64_t)ord32(S) << 32) | (uint64_t)(0xffffffffu - (uint32_t)(e.path * 16 + r))
                            : 0ull;
                cpb[q] = pb;
                cr[q] = r;
                if (in) s_ktab[(d * Wb + pb) * k + r] = -1;
                count += __popcll(__ballot(in));
            }
            nT += count;
            // the W best candidates, in the total order (S desc, rank path asc)
            const int nn = min(Wb, count);
            BeamEntry mine{0.f, 0, 0, 0};
            int mine_pb = 0;
            int okey = 0;
            if constexpr (A == 1) {
                // at most 64 candidates: each takes its place among them by
                // comparing every key once (keys are distinct, 0 = not in T);
                // the nn best hand themselves to lanes 0 .. nn-1 through the
                // next beam's LDS buffer (path holds the rank-path key there)
                int rk = 0;
                const int ncand = nb * k;
                for (int c = 0; c < ncand; ++c) rk += readlane_u64(key[0], c) > key[0] ? 1 : 0;
                if (key[0] != 0ull && rk < nn) {
                    const BeamEntry pe = bc[cpb[0]];
                    s_ktab[(d * Wb + cpb[0]) * k + cr[0]] = (int8_t)rk;
                    s_beam[(cur ^ 1) * Wb + rk] =
                        BeamEntry{unord32((uint32_t)(key[0] >> 32)), cr[0], pe.rank, pe.path * 16 + cr[0]};
                }
                __builtin_amdgcn_wave_barrier();
                if (lane < nn) {
                    mine = s_beam[(cur ^ 1) * Wb + lane];
                    okey = mine.path;
                }
            }
            for (int j = 0; A > 1 && j < nn; ++j) {
                uint64_t lm = 0ull;
#pragma unroll
                for (int q = 0; q < A; ++q) lm = key[q] > lm ? key[q] : lm;
                const uint64_t m = wave_max_u64_dpp(lm);
                int wq = 0, wl = 0;
#pragma unroll
                for (int q = A - 1; q >= 0; --q) {
                    const uint64_t hit = __ballot(key[q] == m);
                    if (hit) {
                        wq = q;
                        wl = __ffsll((unsigned long long)hit) - 1;
                    }
                }
                int lpb = 0, lr = 0;
#pragma unroll
                for (int q = 0; q < A; ++q) {
                    lpb = q == wq ? cpb[q] : lpb;
                    lr = q == wq ? cr[q] : lr;
                }
                const int pb = __builtin_amdgcn_readlane(lpb, wl);
                const int r = __builtin_amdgcn_readlane(lr, wl);
                if (lane == j) {
                    mine = BeamEntry{unord32((uint32_t)(m >> 32)), r, bc[pb].rank, 0};
                    mine_pb = pb;
                }
                if (lane == 0) s_ktab[(d * Wb + pb) * k + r] = (int8_t)j;
#pragma unroll
                for (int q = 0; q < A; ++q) key[q] = (q == wq && lane == wl) ? 0ull : key[q];
            }
            // place of each new entry in rank-path order: (parent's place, rank)
            if constexpr (A > 1) okey = bc[mine_pb].path * 16 + mine.rank;
            int place = 0;
            for (int j = 0; j < nn; ++j) {
                const int oj = __builtin_amdgcn_readlane(okey, j);
                place += (oj < okey) ? 1 : 0;
            }
            mine.path = place;
            __builtin_amdgcn_wave_barrier();
            if (lane < nn) s_beam[(cur ^ 1) * Wb + lane] = mine;
            __builtin_amdgcn_wave_barrier();
            cur ^= 1;
            nb = nn;
        };
        for (int d = 1; d <= D && nT < a.budget && nb > 0; ++d) {
            const int slots = (nb * k + kWave - 1) / kWave;
            if (slots <= 1) beam_depth(SlotCount<1>{}, d);
            else if (slots <= 2) beam_depth(SlotCount<2>{}, d);
            else beam_depth(SlotCount<CS>{}, d);
        }
        __builtin_amdgcn_wave_barrier();
    }

    // Children of node n (depth d, own rank rn, parent's rank rp, score Sn):
    // lane r < k scores candidate r, the children are ranked by (S desc,
    // rank asc) with in-row rotations and stored in that order; returns the
    // first child as (ord S, rank), ord 0 if none.  A node at the depth limit
    // (d == D) has no children: nothing is stored and ord 0 is returned.
    auto expand = [&](int n, int d, int rn, int rp, float Sn, int bidx, uint32_t& c_ord, int& c_rank) {
        const bool live = d < D;
        const int dr = min(d, D - 1);      // drafter row read (clamped at the depth limit)
        const int ctx2 = d >= 2 ? rp : 0;  // grandparent slot of the trigram
        const int ctx1 = d >= 1 ? rn : 0;  // parent slot of the trigram
        const float lam_d = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(lam_lane), dr));
        // every lane reads (lanes >= k at a clamped index) so that no branch
        // separates the reads from their use; only lanes < k are kept
        const int rl = min(lane, k - 1);
        float s;
        {
            const float lq = s_lp[dr * k + rl];
            if constexpr (RHO != 0) {
                const int ri = ((dr * k + ctx2) * k + ctx1) * k + rl;
                float lr;
                if constexpr (RHO == 1)
                    lr = s_rho[ri];
                else
                    lr = g_rho[ri];
                const float t = lam_d * lr;
                s = lq + t;
            } else {
                s = lq;
            }
            s = (s == s && lane < k) ? s : -INFINITY;
        }
        bool in = lane < k && live;
        if constexpr (BEAM) {
            // the children in T (the beam pass applied the branch filter);
            // their table entries are kept for their own pops
            const int tv = s_ktab[((d + 1) * Wb + bidx) * k + rl];
            in = in && tv >= -1;
            if (lane < k && live) s_kbeam[n * k + lane] = (int8_t)tv;
        } else if (a.branch < k) {
            // keep the top-`branch` by token score (larger s, then lower rank)
            int sel = 0;
            for (int j = 0; j < k; ++j) {
                const float sj = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(s), j));
                sel += (sj > s || (sj == s && j < lane)) ? 1 : 0;
            }
            in = in && sel < a.branch;
        }
        const float sc = Sn + s;
        const uint32_t o = ord32(sc);  // nonzero for every non-NaN score
        const uint64_t key = in ? (((uint64_t)o << 8) | (uint64_t)(255 - lane)) : 0ull;
        if (!KQ && k <= 8) {
            // sorted in place: lane p holds the p-th child (key 0 past the
            // last child, which writes the end marker)
            const uint64_t sk = sort8_desc(key, lane);
            if (lane < k && live) {
                s_kord[n * k + lane] = (uint32_t)(sk >> 8);
                s_krank[n * k + lane] = (uint8_t)(255 - (uint32_t)(sk & 255));
            }
            const uint64_t top = readlane_u64(sk, 0);
            c_ord = (uint32_t)(top >> 8);
            c_rank = c_ord ? 255 - (int)(top & 255) : 0;
        } else {
            int pos;
            if constexpr (KQ)
                pos = quad_count_greater(key);
            else
                pos = row_count_greater<15>(key);
            // the lanes that are not children all land on the first free
            // position and write the end marker there
            if (lane < k && live) {
                s_kord[n * k + pos] = in ? o : 0u;
                s_krank[n * k + pos] = (uint8_t)lane;
            }
            const uint64_t first = __ballot(in && pos == 0);
            c_rank = first ? __ffsll((unsigned long long)first) - 1 : 0;
            c_ord = first ? (uint32_t)__builtin_amdgcn_readlane((int)o, c_rank) : 0u;
        }
    };

    // Rank-path keys (four 32-bit words, most significant first): the key of
    // a node is its parent's key with the digit rank + 1 at its depth.  They
    // only break ties of S, so they are derived when a tie needs them: the
    // parent chain of a tied entry is walked up to the nearest node whose key
    // is known (the root, or a node whose key an earlier tie stored: every
    // non-root key has a nonzero first word) and the parent's key is stored.
    uint4* s_pkey = reinterpret_cast<uint4*>(lds + a.o_pkey);  // [N], 0 = not known yet
    const uint32_t pw_magic = (65536u + per_word - 1) / per_word;  // t / per_word = t * magic >> 16 (t < 128)
    auto add_digit = [&](uint4 key, int d, int r) {
        const uint32_t t = (uint32_t)(d - 1);
        const uint32_t wi = (t * pw_magic) >> 16;
        const uint32_t v = (uint32_t)(r + 1) << (32 - (t - wi * per_word + 1) * wbits);
        key.x |= wi == 0 ? v : 0u;
        key.y |= wi == 1 ? v : 0u;
        key.z |= wi == 2 ? v : 0u;
        key.w |= wi == 3 ? v : 0u;
        return key;
    };
    for (int i = lane; i < N; i += kWave) s_pkey[i] = make_uint4(0u, 0u, 0u, 0u);

    if (lane == 0) s_rec[0] = make_uint2(0xffffffffu, __float_as_uint(0.f));
    uint32_t c_ord;
    int c_rank;
    expand(0, 0, 0, 0, 0.f, 0, c_ord, c_rank);

    // frontier slots: slot j of lane l is entry j * 64 + l
    uint32_t fS[SL], fM[SL];
#pragma unroll
    for (int j = 0; j < SL; ++j) fS[j] = fM[j] = 0u;
    if (lane == 0) {
        fS[0] = c_ord;
        fM[0] = pack_meta(0, c_rank, 1, 0, 0);
    }
    int fcount = 1, committed = 1;

    // One pop: commit the best frontier entry and push its successors;
    // false once the frontier is exhausted.  Slots fill lane-major (slot j
    // holds entries 64 j .. 64 j + 63), so only the first A slots of every
    // lane can be occupied, A = fcount / 64 + 1 counting the next fresh one:
    // the per-slot work follows the frontier allocated so far.
    auto pop = [&](auto act) -> bool {
        constexpr int A = decltype(act)::value;
        uint32_t lm = 0u;
#pragma unroll
        for (int j = 0; j < A; ++j) lm = max(lm, fS[j]);
        const uint32_t M = wave_max_u32_dpp(lm);
        if (M == 0u) return false;  // frontier exhausted: the whole candidate tree is committed

        // winner: the unique entry holding M, else the one with the smallest path key
        int cnt = 0, jsel = 0;
#pragma unroll
        for (int j = A - 1; j >= 0; --j) {
            const bool hit = fS[j] == M;
            cnt += hit ? 1 : 0;
            jsel = hit ? j : jsel;
        }
        const uint64_t any = __ballot(cnt > 0);
        int w;
        if (__popcll(any) == 1 && __ballot(cnt > 1) == 0ull) {
            w = __ffsll((unsigned long long)any) - 1;
        } else {
            uint32_t bk[4] = {~0u, ~0u, ~0u, ~0u};
            int bj = 0;
            for (int j = 0; j < A; ++j) {
                if (fS[j] == M) {
                    const int p = fM[j] & 1023;
                    uint4 acc = make_uint4(0u, 0u, 0u, 0u);
                    int y = p;
                    uint4 st = s_pkey[y];
                    uint32_t m = s_rec[y].x;
                    while (y != 0 && st.x == 0u) {
                        acc = add_digit(acc, (m >> 14) & 63, (m >> 10) & 15);
                        y = m & 1023;
                        st = s_pkey[y];
                        m = s_rec[y].x;
                    }
                    const uint4 kp = make_uint4(acc.x | st.x, acc.y | st.y, acc.z | st.z, acc.w | st.w);
                    if (y != p) s_pkey[p] = kp;  // lanes storing the same node store the same key
                    const uint4 kv = add_digit(kp, (fM[j] >> 14) & 63, (fM[j] >> 10) & 15);
                    const uint32_t kw[4] = {kv.x, kv.y, kv.z, kv.w};
                    const bool less =
                        kw[0] != bk[0] ? kw[0] < bk[0]
                                       : (kw[1] != bk[1] ? kw[1] < bk[1]
                                                         : (kw[2] != bk[2] ? kw[2] < bk[2] : kw[3] < bk[3]));
                    if (less) {
                        bk[0] = kw[0]; bk[1] = kw[1]; bk[2] = kw[2]; bk[3] = kw[3];
                        bj = j;
                    }
                }
            }
            bool t = cnt > 0;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint32_t mq = wave_min_u32_dpp(t ? bk[q] : ~0u);
                t = t && bk[q] == mq;
            }
            w = __ffsll((unsigned long long)__ballot(t)) - 1;
            jsel = bj;
        }
        uint32_t lmeta = 0u;
#pragma unroll
        for (int j = 0; j < A; ++j) lmeta = j == jsel ? fM[j] : lmeta;
        const uint32_t meta = (uint32_t)__builtin_amdgcn_readlane((int)lmeta, w);
        const int eslot = __builtin_amdgcn_readlane(jsel, w);
        const int p = meta & 1023, r = (meta >> 10) & 15, d = (meta >> 14) & 63, rp = (meta >> 20) & 15;
        const int pos = (meta >> 24) & 15;
        const float S = unord32(M);

        // commit node n: one record; everything else is derived after the search
        const int n = committed++;
        if (lane == 0) s_rec[n] = make_uint2(meta, __float_as_uint(S));
        int bidx = 0;  // beam search: n's entry in the beam of its depth, or < 0
        if constexpr (BEAM) {
            bidx = s_kbeam[p * k + r];  // recorded when p was expanded
        }

        // next sibling of n: the next entry of its parent's ordered children
        // (read unconditionally, at a clamped index, so that its latency
        // overlaps the expansion's reads)
        const int si = p * k + min(pos + 1, k - 1);
        const uint32_t sib_raw = s_kord[si];
        const int sib_rank = s_krank[si];
        // first child of n
        uint32_t kid_ord = 0u;
        int kid_rank = 0;
        if (!BEAM || (d < D && bidx >= 0)) expand(n, d, r, rp, S, bidx, kid_ord, kid_rank);
        const uint32_t sib_ord = pos + 1 < k ? sib_raw : 0u;

        // pushes: the first reuses the popped slot, the second takes a fresh slot
        uint32_t xS = 0u, xM = 0u, yS = 0u, yM = 0u;
        if (kid_ord != 0u) {
            xS = kid_ord;
            xM = pack_meta(n, kid_rank, d + 1, r, 0);
        }
        if (sib_ord != 0u) {
            const uint32_t m = pack_meta(p, sib_rank, d, rp, pos + 1);
            if (xS != 0u) {
                yS = sib_ord;
                yM = m;
            } else {
                xS = sib_ord;
                xM = m;
            }
        }
        const bool second = yS != 0u;
        const int ylane = fcount & (kWave - 1), yslot = fcount >> 6;
        if constexpr (A <= 2) {
            // one lane of one slot each: lane writes from scalar values (with
            // a single slot in use both go to slot 0)
#pragma unroll
            for (int j = 0; j < A; ++j) {
                if (A == 1 || j == eslot) {
                    fS[j] = write_lane(fS[j], xS, w);
                    fM[j] = write_lane(fM[j], xM, w);
                }
                if (second && (A == 1 || j == yslot)) {
                    fS[j] = write_lane(fS[j], yS, ylane);
                    fM[j] = write_lane(fM[j], yM, ylane);
                }
            }
        } else {
            // more slots: one select per slot instead of a branch per slot
#pragma unroll
            for (int j = 0; j < A; ++j) {
                const bool px = lane == w && j == eslot;
                const bool py = second && lane == ylane && j == yslot;
                fS[j] = px ? xS : (py ? yS : fS[j]);
                fM[j] = px ? xM : (py ? yM : fM[j]);
            }
        }
        if (second) ++fcount;
        return true;
    };
    while (committed - 1 < a.budget) {
        const int need = min((fcount >> 6) + 1, SL);
        bool go;
        if (need <= 1) go = pop(SlotCount<1>{});
        else if (SL <= 2 || need <= 2) go = pop(SlotCount<(SL < 2 ? SL : 2)>{});
        else if (SL <= 3 || need <= 3) go = pop(SlotCount<(SL < 3 ? SL : 3)>{});
        else if (SL <= 4 || need <= 4) go = pop(SlotCount<(SL < 4 ? SL : 4)>{});
        else if (SL <= 5 || need <= 5) go = pop(SlotCount<(SL < 5 ? SL : 5)>{});
        else if (SL <= 8 || need <= 8) go = pop(SlotCount<(SL < 8 ? SL : 8)>{});
        else go = pop(SlotCount<SL>{});
        if (!go) break;
    }
    __builtin_amdgcn_wave_barrier();

    // Output rows and ancestor masks, one node per lane: the mask of node n has
    // the bits of n and of every node on its parent chain (SL >= W =
    // ceil(N / 64) words suffice).
    const int64_t ob = (int64_t)b * N;
    const int root_tok = __builtin_amdgcn_readfirstlane(a.root_token[b]);
    for (int i = lane; i < N; i += kWave) {
        uint64_t words[SL];
#pragma unroll
        for (int q = 0; q < SL; ++q) words[q] = 0ull;
        if (i < committed) {
            const uint2 rec = s_rec[i];
            const int p = i == 0 ? -1 : (int)(rec.x & 1023);
            const int r = (rec.x >> 10) & 15, d = i == 0 ? 0 : (rec.x >> 14) & 63;
            a.parent[ob + i] = p;
            a.token[ob + i] = i == 0 ? root_tok : s_ids[(d > 0 ? d - 1 : 0) * k + r];
            a.depth[ob + i] = d;
            a.rank[ob + i] = i == 0 ? -1 : r;
            a.score[ob + i] = __uint_as_float(rec.y);
            int x = i;
            while (true) {
#pragma unroll
                for (int q = 0; q < SL; ++q) words[q] |= q == (x >> 6) ? 1ull << (x & 63) : 0ull;
                if (x == 0) break;
                x = (int)(s_rec[x].x & 1023);
            }
        } else {
            a.parent[ob + i] = -1;
            a.token[ob + i] = -1;
            a.depth[ob + i] = -1;
            a.rank[ob + i] = -1;
            a.score[ob + i] = -INFINITY;
        }
#pragma unroll
        for (int q = 0; q < SL; ++q)
            if (q < W) a.anc[(ob + i) * W + q] = words[q];
    }
    if (lane == 0) a.n_nodes[b] = committed;
}


// Literal Alg. 2 (Sec. 4.2): T grows by whole expansions.  The root is
// expanded first; every later pop takes the best node of T not yet expanded
// (total order: S desc, rank path asc) and appends its top-`branch`
// children to T.  The search stops once T holds `budget` non-root nodes (the
// last expansion may overshoot by branch - 1) or nothing is left to expand,
// and the tree is TopB(T): the `budget` best nodes of T, in the total order,
// after the root.  One wavefront per sequence: T lives in LDS (per node the
// parent, rank and depth in one word, S, and the rank-path key, built from
// the parent's key when the node is appended); node e of T is "not yet
// expanded" while slot e / 64 of lane e % 64 holds ord(S) (0 once expanded).
// TopB(T) places every node by counting the nodes before it.
template <int SLT, int RHO>
__global__ __launch_bounds__(kWave) void tree_alg2_kernel(TreeArgs a) {
    extern __shared__ __align__(16) char lds[];
    const int lane = lane_id();
    const int b = blockIdx.x;
    const int D = a.D, k = a.k, N = a.N, W = a.W, wbits = a.wbits, per_word = a.per_word;
    const int branch = a.branch, budget = a.budget;
    float* s_lp = reinterpret_cast<float*>(lds + a.o_lp);
    int32_t* s_ids = reinterpret_cast<int32_t*>(lds + a.o_ids);
    float* s_rho = reinterpret_cast<float*>(lds + a.o_rho);
    // T node c: (parent + 1, 0 for the root) | rank << 11 | depth << 15
    // (T holds up to budget + branch - 1 <= 1038 nodes: 11 bits of parent)
    uint32_t* s_tmeta = reinterpret_cast<uint32_t*>(lds + a.o_tmeta);
    float* s_tS = reinterpret_cast<float*>(lds + a.o_tS);
    uint4* s_tkey = reinterpret_cast<uint4*>(lds + a.o_tkey);  // x: most significant word
    int32_t* s_tplace = reinterpret_cast<int32_t*>(lds + a.o_tplace);
    const int rho_n = D * k * k * k;
    const float* g_rho = RHO ? a.log_rho + (int64_t)b * rho_n : nullptr;

    // every load of the tables requested before the first store, as in the
    // best-first kernel
    const float lam_lane = lane < D ? a.lambda[(int64_t)b * a.lambda_stride + lane] : 0.f;
    const int64_t tb = (int64_t)b * D * k;
    {
        uint32_t r_lp[8], r_ids[8], r_rho[16];  // D * k <= 512 words
        load_words(r_lp, reinterpret_cast<const uint32_t*>(a.logprob + tb), D * k, 0, lane);
        load_words(r_ids, reinterpret_cast<const uint32_t*>(a.ids + tb), D * k, 0, lane);
        if constexpr (RHO == 1) load_words(r_rho, reinterpret_cast<const uint32_t*>(g_rho), rho_n, 0, lane);
        store_words(reinterpret_cast<uint32_t*>(s_lp), r_lp, D * k, 0, lane);
        store_words(reinterpret_cast<uint32_t*>(s_ids), r_ids, D * k, 0, lane);
        if constexpr (RHO == 1) {
            store_words(reinterpret_cast<uint32_t*>(s_rho), r_rho, rho_n, 0, lane);
            if (rho_n > 16 * kWave)
                stage_words(reinterpret_cast<uint32_t*>(s_rho) + 16 * kWave,
                            reinterpret_cast<const uint32_t*>(g_rho) + 16 * kWave, rho_n - 16 * kWave,
                            lane);
        }
    }
    __builtin_amdgcn_wave_barrier();

    // Appends the top-`branch` children (by s desc, rank asc) of the node v
    // (T index, -1 for the root; depth d < D, own rank rn, parent's rank rp,
    // score Sv, key kv) to T at index nT.  Lane r scores candidate r.
    auto expand = [&](int v, int d, int rn, int rp, float Sv, uint4 kv, int nT) {
        const int ctx2 = d >= 2 ? rp : 0;
        const int ctx1 = d >= 1 ? rn : 0;
        const int rl = min(lane, k - 1);
        float s = s_lp[d * k + rl];
        if constexpr (RHO != 0) {
            const float lam_d = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(lam_lane), d));
            const int ri = ((d * k + ctx2) * k + ctx1) * k + rl;
            const float lr = RHO == 1 ? s_rho[ri] : g_rho[ri];
            const float t = lam_d * lr;
            s = s + t;
        }
        s = (s == s && lane < k) ? s : -INFINITY;
        int sel = 0;
        for (int j = 0; j < k; ++j) {
            const float sj = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(s), j));
            sel += (sj > s || (sj == s && j < lane)) ? 1 : 0;
        }
        if (lane < k && sel < branch) {
            const int c = nT + sel;
            s_tmeta[c] = (uint32_t)(v + 1) | ((uint32_t)lane << 11) | ((uint32_t)(d + 1) << 15);
            s_tS[c] = Sv + s;
            const int wi = d / per_word, sh = 32 - (d % per_word + 1) * wbits;
            const uint32_t dig = (uint32_t)(lane + 1) << sh;
            s_tkey[c] = make_uint4(kv.x | (wi == 0 ? dig : 0u), kv.y | (wi == 1 ? dig : 0u),
                                   kv.z | (wi == 2 ? dig : 0u), kv.w | (wi == 3 ? dig : 0u));
        }
        __builtin_amdgcn_wave_barrier();
    };
    // marks T nodes n0 .. n0 + cnt - 1 as not yet expanded
    uint32_t fO[SLT];
#pragma unroll
    for (int j = 0; j < SLT; ++j) fO[j] = 0u;
    auto mark_open = [&](int n0, int cnt) {
#pragma unroll
        for (int j = 0; j < SLT; ++j) {
            const int e = j * kWave + lane;
            if (e >= n0 && e < n0 + cnt) fO[j] = ord32(s_tS[e]);
        }
    };
    auto key_less = [](uint4 x, uint4 y) {
        return x.x != y.x ? x.x < y.x : (x.y != y.y ? x.y < y.y : (x.z != y.z ? x.z < y.z : x.w < y.w));
    };

    expand(-1, 0, 0, 0, 0.f, make_uint4(0u, 0u, 0u, 0u), 0);  // depth >= 1: the root has children
    mark_open(0, branch);
    int nT = branch;
    while (nT < budget) {
        uint32_t lm = 0u;
#pragma unroll
        for (int j = 0; j < SLT; ++j) lm = max(lm, fO[j]);
        const uint32_t M = wave_max_u32_dpp(lm);
        if (M == 0u) break;  // every node of T expanded
        int cnt = 0, jsel = 0;
#pragma unroll
        for (int j = SLT - 1; j >= 0; --j) {
            const bool hit = fO[j] == M;
            cnt += hit ? 1 : 0;
            jsel = hit ? j : jsel;
        }
        const uint64_t any = __ballot(cnt > 0);
        int w;
        if (__popcll(any) == 1 && __ballot(cnt > 1) == 0ull) {
            w = __ffsll((unsigned long long)any) - 1;
        } else {
            // several nodes share the best S: the smallest rank-path key wins
            uint4 bk = make_uint4(~0u, ~0u, ~0u, ~0u);
            int bj = 0;
            for (int j = 0; j < SLT; ++j) {
                if (fO[j] == M) {
                    const uint4 kj = s_tkey[j * kWave + lane];
                    if (key_less(kj, bk)) {
                        bk = kj;
                        bj = j;
                    }
                }
            }
            bool t = cnt > 0;
            uint32_t m;
            m = wave_min_u32_dpp(t ? bk.x : ~0u); t = t && bk.x == m;
            m = wave_min_u32_dpp(t ? bk.y : ~0u); t = t && bk.y == m;
            m = wave_min_u32_dpp(t ? bk.z : ~0u); t = t && bk.z == m;
            m = wave_min_u32_dpp(t ? bk.w : ~0u); t = t && bk.w == m;
            w = __ffsll((unsigned long long)__ballot(t)) - 1;
            jsel = bj;
        }
        const int es = __builtin_amdgcn_readlane(jsel, w);
        const int e = es * kWave + w;
#pragma unroll
        for (int j = 0; j < SLT; ++j) fO[j] = (lane == w && j == es) ? 0u : fO[j];
        const uint32_t meta = s_tmeta[e];
        const int d = (meta >> 15) & 63;
        if (d < D) {
            const int pv = (int)(meta & 2047) - 1;
            const int rp = pv >= 0 ? (int)((s_tmeta[pv] >> 11) & 15) : 0;
            expand(e, d, (meta >> 11) & 15, rp, s_tS[e], s_tkey[e], nT);
            mark_open(nT, branch);
            nT += branch;
        }
    }

    // TopB(T): the place of node i in the total order is the number of nodes
    // of T before it (S larger, or S equal and rank-path key smaller)
    const int keep = min(nT, budget);
    uint32_t oT[SLT];
#pragma unroll
    for (int q = 0; q < SLT; ++q) {
        const int i = q * kWave + lane;
        oT[q] = i < nT ? ord32(s_tS[i]) : 0u;
    }
    int place[SLT];
#pragma unroll
    for (int q = 0; q < SLT; ++q) place[q] = 0;
#pragma unroll
    for (int sj = 0; sj < SLT; ++sj) {
        for (int l = 0; l < kWave; ++l) {
            const int j = sj * kWave + l;
            if (j >= nT) break;
            const uint32_t oj = (uint32_t)__builtin_amdgcn_readlane((int)oT[sj], l);
            bool tie = false;
#pragma unroll
            for (int q = 0; q < SLT; ++q) {
                place[q] += oj > oT[q] ? 1 : 0;
                tie = tie || (oj == oT[q] && q * kWave + lane != j && q * kWave + lane < nT);
            }
            if (__ballot(tie)) {
                const uint4 kj = s_tkey[j];
#pragma unroll
                for (int q = 0; q < SLT; ++q) {
                    const int i = q * kWave + lane;
                    if (oj == oT[q] && i != j && i < nT && key_less(kj, s_tkey[i])) ++place[q];
                }
            }
        }
    }
#pragma unroll
    for (int q = 0; q < SLT; ++q) {
        const int i = q * kWave + lane;
        if (i < nT) s_tplace[i] = place[q];
    }
    __builtin_amdgcn_wave_barrier();

    // output: row 0 the root, rows 1 .. keep the kept nodes in order, then padding
    const int64_t ob = (int64_t)b * N;
    constexpr int SLW = SLT + 1;  // mask words: N = budget + 1 <= 64 * SLT + 1
    for (int i = lane; i < nT; i += kWave) {
        const int pl = s_tplace[i];
        if (pl >= keep) continue;
        const int o = pl + 1;
        const uint32_t meta = s_tmeta[i];
        const int pv = (int)(meta & 2047) - 1, r = (meta >> 11) & 15, d = (meta >> 15) & 63;
        int po = 0;
        if (pv >= 0) po = s_tplace[pv] < keep ? s_tplace[pv] + 1 : -2;
        a.parent[ob + o] = po;
        a.token[ob + o] = s_ids[(d - 1) * k + r];
        a.depth[ob + o] = d;
        a.rank[ob + o] = r;
        a.score[ob + o] = s_tS[i];
        // ancestor bits: this node, then the parent chain until the root
        // (or a parent that TopB(T) dropped, which ends the chain)
        uint64_t words[SLW];
#pragma unroll
        for (int q = 0; q < SLW; ++q) words[q] = 0ull;
        int x = i, xo = o;
        while (true) {
#pragma unroll
            for (int q = 0; q < SLW; ++q) words[q] |= q == (xo >> 6) ? 1ull << (xo & 63) : 0ull;
            const int xv = (int)(s_tmeta[x] & 2047) - 1;
            if (xv < 0) {
                words[0] |= 1ull;  // the root
                break;
            }
            if (s_tplace[xv] >= keep) break;
            x = xv;
            xo = s_tplace[xv] + 1;
        }
#pragma unroll
        for (int q = 0; q < SLW; ++q)
            if (q < W) a.anc[(ob + o) * W + q] = words[q];
    }
    const int root_tok = __builtin_amdgcn_readfirstlane(a.root_token[b]);
    for (int i = lane; i < N; i += kWave) {
        if (i != 0 && i <= keep) continue;
        const bool root = i == 0;
        a.parent[ob + i] = -1;
        a.token[ob + i] = root ? root_tok : -1;
        a.depth[ob + i] = root ? 0 : -1;
        a.rank[ob + i] = -1;
        a.score[ob + i] = root ? 0.f : -INFINITY;
        for (int q = 0; q < W; ++q) a.anc[(ob + i) * W + q] = (root && q == 0) ? 1ull : 0ull;
    }
    if (lane == 0) a.n_nodes[b] = keep + 1;
}

// ---------------------------------------------------------------------------
// Best-first tree by frontier sweeps.
//
// Every token score is <= 0, so S never increases along a path and an
// ancestor precedes its descendants in the total order (S desc, rank path
// asc): the nodes that best-first search commits, in pop order, are the
// `budget` best non-root prefixes in that order (the closed form of Sec.
// 4.2), sorted.  This kernel finds that set without popping one node at a
// time.  One workgroup per sequence keeps in LDS
//   T: the best (at most budget) prefixes materialised so far, sorted;
//   P: pending prefixes, each the next sibling (in child order: S desc,
//      rank asc, among the top-`branch` candidates) or a member of the
//      first-child chain (below) of a prefix that entered T, not
//      materialised yet.
// A sweep merges all of P into T (every entry's new place from counting
// comparisons; entries pushed past the budget are dropped for good, since
// T's last entry only ever improves) and then, for every prefix of P that
// entered T, pushes its next sibling and, if it ends a chain, the chain of
// its first child, that child's first child, ... (CL levels; only a chain's
// last member pushes the next chain), keeping a push while T is not full or
// when it precedes T's last entry.  A prefix of the optimal tree is always
// pushed (its parent, or its previous sibling, or the head of its chain
// precedes it and so enters T when materialised) and never dropped (it
// precedes every last entry T ever has), so T is the optimal tree once
// nothing is pending.  A prefix is pushed at most once, and a sweep pushes
// at most CL + 1 prefixes per entry that entered T, so P never holds more
// than (CL + 1) budget.  The number of sweeps follows the depth of the tree
// and the chain length, not the budget (at depth 16 and budget 64: about 15
// with CL = 1, 6 with CL = 3).
//
// Every record carries its full rank-path key, its parent's S and the ranks
// of its trigram context, so that a push reads no other record; a node's
// parent is found after the search by a binary search of T for the
// parent's (S, key).

// A record: ord(S), rank-path key (k0 most significant), ord(S) of the
// parent, and rank | depth << 4 | parent's rank << 10 | grandparent's rank
// << 14 | chain end << 18.  In LDS two 16-byte words: (o, k0, k1, k2),
// (k3, po, meta, 0).
struct SwRec {
    uint32_t o, k0, k1, k2, k3, po, meta;
};

__device__ __forceinline__ SwRec sw_load(const uint4* base, int i) {
    const uint4 x = base[2 * i], y = base[2 * i + 1];
    return SwRec{x.x, x.y, x.z, x.w, y.x, y.y, y.z};
}
__device__ __forceinline__ void sw_store(uint4* base, int i, const SwRec& r) {
    base[2 * i] = make_uint4(r.o, r.k0, r.k1, r.k2);
    base[2 * i + 1] = make_uint4(r.k3, r.po, r.meta, 0u);
}
// The rank-path key of x is smaller than that of y.  Written with bitwise
// operators throughout: short-circuit forms compile to divergent branches.
__device__ __forceinline__ bool sw_key_less(const SwRec& x, const SwRec& y) {
    const uint64_t xa = ((uint64_t)x.k0 << 32) | (uint64_t)x.k1;
    const uint64_t ya = ((uint64_t)y.k0 << 32) | (uint64_t)y.k1;
    const uint64_t xb = ((uint64_t)x.k2 << 32) | (uint64_t)x.k3;
    const uint64_t yb = ((uint64_t)y.k2 << 32) | (uint64_t)y.k3;
    return (xa < ya) | ((xa == ya) & (xb < yb));
}
// x precedes y in the total order (keys of distinct prefixes differ)
__device__ __forceinline__ bool sw_before(const SwRec& x, const SwRec& y) {
    return (x.o > y.o) | ((x.o == y.o) & sw_key_less(x, y));
}
__device__ __forceinline__ SwRec sw_readlane(const SwRec& r, int l) {
    SwRec y;
    y.o = (uint32_t)__builtin_amdgcn_readlane((int)r.o, l);
    y.k0 = (uint32_t)__builtin_amdgcn_readlane((int)r.k0, l);
    y.k1 = (uint32_t)__builtin_amdgcn_readlane((int)r.k1, l);
    y.k2 = (uint32_t)__builtin_amdgcn_readlane((int)r.k2, l);
    y.k3 = (uint32_t)__builtin_amdgcn_readlane((int)r.k3, l);
    y.po = 0u;
    y.meta = 0u;
    return y;
}
__device__ __forceinline__ int lanes_below(uint64_t m) {
    return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

constexpr int kSweepWaves = 4;  // one wave per SIMD
// An entry that enters T pushes its next sibling and, when it ends a chain,
// the chain of its first child, that child's first child, ... CL levels
// deep; only the last of a chain pushes the next chain (every prefix is
// still pushed once: a first child by its parent's chain).  A chain advances
// a path of first children CL levels per sweep: at budget 64 and depth 16
// the sweeps drop from about 15 to 8 with CL = 2 and to 6 with CL = 3.
constexpr uint32_t kChainEnd = 1u << 18;  // record meta: this entry pushes the next chain

// MT: slots per lane of T (budget <= 64 MT), MP: slots per lane of P
// ((CL + 1) budget <= 64 MP), KM: k <= KM, RHO as in tree_build_kernel, CL:
// chain length.
//
// One workgroup of four waves per sequence.  Every wave holds all of T and
// P in registers (from 8 slots of T on, only P's ord S: its records stay in
// LDS, in two buffers, one read and one written by a sweep); the merge's comparisons are split over the waves (each
// takes every fourth P entry in turn and its partial counts are summed
// through LDS); the push candidates are scored before the merge, split into
// tasks (first children, next siblings) per slot of P, and each task
// reserves its places in the next P with one LDS atomic.  A sweep has two
// barriers: after the partial counts, and after the stores and pushes.
template <int MT, int MP, int KM, int RHO, int CL>
__global__ __launch_bounds__(kSweepWaves * kWave) void tree_sweep_kernel(TreeArgs a) {
    constexpr int NWV = kSweepWaves, NT = NWV * kWave;
    extern __shared__ __align__(16) char lds[];
    const int tid = threadIdx.x, lane = lane_id();
    const int wv = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int b = blockIdx.x;
    const int D = a.D, k = a.k, N = a.N, W = a.W, wbits = a.wbits, per_word = a.per_word;
    const int NB = N - 1;             // non-root nodes of a full tree
    const int cap_p = (CL + 1) * NB;  // P's capacity
    float* s_lp = reinterpret_cast<float*>(lds + a.o_lp);
    int32_t* s_ids = reinterpret_cast<int32_t*>(lds + a.o_ids);
    float* s_lam = reinterpret_cast<float*>(lds + a.o_lam);
    uint4* s_t = reinterpret_cast<uint4*>(lds + a.o_sw_t);          // [NB] records, sorted
    constexpr bool PL = MT >= 8;  // P's records in LDS only
    uint4* s_pc = reinterpret_cast<uint4*>(lds + a.o_sw_p);         // [cap_p] records: P of this sweep
    uint4* s_pn = PL ? reinterpret_cast<uint4*>(lds + a.o_sw_p2) : s_pc;  // the pushes
    int32_t* s_par = reinterpret_cast<int32_t*>(lds + a.o_sw_par);  // [N] parent of node i
    int32_t* s_cnt = reinterpret_cast<int32_t*>(lds + a.o_sw_cnt);  // [NWV][MT + MP][64] partial counts
    int32_t* s_np = reinterpret_cast<int32_t*>(lds + a.o_sw_np);    // [2] pending counts, alternating
    float* s_rho = reinterpret_cast<float*>(lds + a.o_rho);
    const int rho_n = D * k * k * k;
    const float* g_rho = RHO ? a.log_rho + (int64_t)b * rho_n : nullptr;

    const int64_t tb = (int64_t)b * D * k;
    if (wv == 0) {
        uint32_t r_lp[8], r_ids[8];  // D * k <= 512 words
        load_words(r_lp, reinterpret_cast<const uint32_t*>(a.logprob + tb), D * k, 0, lane);
        load_words(r_ids, reinterpret_cast<const uint32_t*>(a.ids + tb), D * k, 0, lane);
        const float lam = lane < D ? a.lambda[(int64_t)b * a.lambda_stride + lane] : 0.f;
        store_words(reinterpret_cast<uint32_t*>(s_lp), r_lp, D * k, 0, lane);
        store_words(reinterpret_cast<uint32_t*>(s_ids), r_ids, D * k, 0, lane);
        if (lane < D) s_lam[lane] = lam;
    }
    // Token scores fl(log q + fl(lambda * log rho)), NaN -> -inf, computed
    // once per trigram context in place of the lattice (or of the log q
    // table without one), so that scoring a node's children reads k values.
    // Every thread stages the lattice with up to 32 words in flight, the
    // first batch requested before the barrier that publishes log q and
    // lambda.  A lattice of at most 8 words per thread takes a copy of the
    // loop unrolled 8 times (its cold instruction fetch is part of every
    // launch).  A lattice read from global memory is scored on the fly.
    if constexpr (RHO == 1) {
        const uint32_t* gr = reinterpret_cast<const uint32_t*>(g_rho);
        auto stage = [&](auto uc) __attribute__((always_inline)) {
            constexpr int U = decltype(uc)::value;
            for (int base = 0; base < rho_n; base += U * NT) {
                // words of this batch per thread that exist for some thread
                // (bounded in the small copy only: in the large one the
                // bound's branches would split the batch's requests)
                const int nu = U > 8 ? U : min(U, (rho_n - base + NT - 1) / NT);
                float x[U];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int i = base + u * NT + tid;
                    x[u] = (u < nu && i < rho_n) ? __uint_as_float(gr[i]) : 0.f;
                }
                if (base == 0) __syncthreads();
                // every log q and lambda of the batch read before the first
                // store (a store between them would order each read after it)
                float lq[U], lm[U];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    lq[u] = lm[u] = 0.f;
                    if (u < nu) {
                        const int i = min(base + u * NT + tid, rho_n - 1);
                        const int row = k == 1 ? i : (int)__umulhi((uint32_t)i, a.mag_k3);
                        const int r = k == 1 ? 0 : i - (int)__umulhi((uint32_t)i, a.mag_k) * k;
                        lq[u] = s_lp[row * k + r];
                        lm[u] = s_lam[row];
                    }
                }
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int i = base + u * NT + tid;
                    const float t = lm[u] * x[u];
                    const float v = lq[u] + t;
                    if (u < nu && i < rho_n) s_rho[i] = (v == v) ? v : -INFINITY;
                }
            }
        };
        if (rho_n <= 8 * NT)
            stage(std::integral_constant<int, 8>{});
        else
            stage(std::integral_constant<int, 32>{});
    } else {
        __syncthreads();
        if constexpr (RHO == 0) {
            for (int i = tid; i < D * k; i += NT) {
                const float v = s_lp[i];
                s_lp[i] = (v == v) ? v : -INFINITY;
            }
        }
    }
    __syncthreads();

    const uint32_t pw_magic = (65536u + per_word - 1) / per_word;  // t / per_word = t * magic >> 16 (t < 128)
    // the key with the digit of depth d set to rank r + 1 (cleared first)
    auto with_digit = [&](SwRec x, int d, int r) {
        const uint32_t t = (uint32_t)(d - 1);
        const uint32_t wi = (t * pw_magic) >> 16;
        const uint32_t sh = 32u - (t - wi * (uint32_t)per_word + 1u) * (uint32_t)wbits;
        const uint32_t m = ((1u << wbits) - 1u) << sh;
        const uint32_t v = (uint32_t)(r + 1) << sh;
        x.k0 = wi == 0 ? (x.k0 & ~m) | v : x.k0;
        x.k1 = wi == 1 ? (x.k1 & ~m) | v : x.k1;
        x.k2 = wi == 2 ? (x.k2 & ~m) | v : x.k2;
        x.k3 = wi == 3 ? (x.k3 & ~m) | v : x.k3;
        return x;
    };

    // The best child, in child order, of a node with score Sn whose children
    // sit at drafter row `row` in trigram context (c2, c1): with `first`,
    // the first child; otherwise the first one after the child (ao, ar) (its
    // ord S and rank).  The top-`branch` by (token score desc, rank asc) are
    // children.  Returns ord S of the child, 0 if there is none.
    auto child = [&](int row, int c2, int c1, float Sn, bool first, uint32_t ao, int ar, int& r_out,
                     float& S_out) -> uint32_t {
        float s[KM];
        if constexpr (RHO == 2) {
            const float lam = s_lam[row];
#pragma unroll
            for (int r = 0; r < KM; ++r) {
                const int rr = r < k ? r : k - 1;
                const float lq = s_lp[row * k + rr];
                const float lr = g_rho[((row * k + c2) * k + c1) * k + rr];
                const float t = lam * lr;
                const float v = lq + t;
                s[r] = (v == v) ? v : -INFINITY;
            }
        } else {
            const float* sc = RHO == 1 ? s_rho + ((row * k + c2) * k + c1) * k : s_lp + row * k;
            if (KM == 4 && k == 4) {
                const float4 v = *reinterpret_cast<const float4*>(sc);  // 16-byte aligned: offsets are multiples of 4 words
                s[0] = v.x;
                s[1] = v.y;
                s[2] = v.z;
                s[3] = v.w;
            } else {
#pragma unroll
                for (int r = 0; r < KM; ++r) s[r] = sc[r < k ? r : k - 1];
            }
        }
        // candidates kept by the branch filter (a mask), then one key per
        // candidate, (ord S, 255 - rank), and a maximum over them as a tree
        uint32_t selm = k >= 32 ? ~0u : (1u << k) - 1u;
        if (a.branch < k) {
            selm = 0u;
#pragma unroll
            for (int r = 0; r < KM; ++r) {
                int c = 0;
#pragma unroll
                for (int j = 0; j < KM; ++j)
                    c += ((j < k) & ((s[j] > s[r]) | ((s[j] == s[r]) & (j < r)))) ? 1 : 0;
                selm |= ((r < k) & (c < a.branch)) ? 1u << r : 0u;
            }
        }
        uint64_t key[KM];
#pragma unroll
        for (int r = 0; r < KM; ++r) {
            const float Sc = Sn + s[r];
            const uint32_t oc = ord32(Sc);
            const bool after = first | (oc < ao) | ((oc == ao) & (r > ar));
            key[r] = (((selm >> r) & 1u) & after) ? ((uint64_t)oc << 8) | (uint64_t)(255 - r) : 0ull;
        }
#pragma unroll
        for (int w = 1; w < KM; w *= 2)
#pragma unroll
            for (int r = 0; r + w < KM; r += 2 * w) key[r] = key[r + w] > key[r] ? key[r + w] : key[r];
        const uint32_t bo = (uint32_t)(key[0] >> 8);
        r_out = 255 - (int)(key[0] & 255u);
        S_out = unord32(bo);  // S is never -0.0 or NaN here, so this is the sum itself
        return bo;
    };

    // the first child of a record w (chain end flag `end`), or of the root
    auto first_child = [&](const SwRec& w, bool root, bool end, SwRec& c) -> bool {
        const int d = root ? 0 : (int)(w.meta >> 4) & 63, r = (int)(w.meta & 15);
        const int rp = (int)(w.meta >> 10) & 15;
        const int drow = min(max(d, 0), D - 1);  // clamped for lanes without a valid entry
        int cr;
        float cS;
        const uint32_t co = child(drow, d >= 2 ? rp : 0, d >= 1 ? r : 0, root ? 0.f : unord32(w.o), true, 0u,
                                  0, cr, cS);
        c = SwRec{co, root ? 0u : w.k0, root ? 0u : w.k1, root ? 0u : w.k2, root ? 0u : w.k3,
                  root ? ord32(0.f) : w.o,
                  (uint32_t)cr | ((uint32_t)(d + 1) << 4) | ((uint32_t)r << 10) | ((uint32_t)rp << 14) |
                      (end ? kChainEnd : 0u)};
        c = with_digit(c, min(d + 1, D), cr);
        return (d < D) & (co != 0u);
    };

    // P starts as the root's first chain
    if (tid == 0) {
        SwRec par{0u, 0u, 0u, 0u, 0u, 0u, 0u};
        int n = 0;
        for (int i = 0; i < CL; ++i) {
            SwRec c;
            if (!first_child(par, i == 0, i == CL - 1, c)) break;
            sw_store(s_pc, n++, c);
            par = c;
        }
        s_np[0] = n;
        s_np[1] = 0;
    }
    __syncthreads();

    int nt = 0, cur = 0;
    int np = min(s_np[0], cap_p);
    while (np > 0) {
        // P in slots (entry u * 64 + lane), T likewise (position v * 64 + lane)
        SwRec pr[PL ? 1 : MP], tr[MT];  // P's records (register mode)
        uint32_t pS[MP];                // P's ord S
        bool pv[MP], tv[MT];
#pragma unroll
        for (int u = 0; u < MP; ++u) {
            pv[u] = u * kWave + lane < np;
            pS[u] = 0u;
            if constexpr (PL) {
                if (u * kWave < np) pS[u] = reinterpret_cast<const uint32_t*>(s_pc)[8 * min(u * kWave + lane, np - 1)];
            } else {
                pr[u] = SwRec{0u, 0u, 0u, 0u, 0u, 0u, 0u};
                if (u * kWave < np) pr[u] = sw_load(s_pc, min(u * kWave + lane, np - 1));
                pS[u] = pr[u].o;
            }
        }
        // P entry u * 64 + lane as a whole record (from LDS when only its
        // ord S is held)
        auto prec = [&](int u) __attribute__((always_inline)) {
            if constexpr (PL) return sw_load(s_pc, min(u * kWave + lane, np - 1));
            else return pr[u];
        };
        auto prec_at = [&](int u, int l) __attribute__((always_inline)) {
            if constexpr (PL) return sw_load(s_pc, u * kWave + l);
            else return sw_readlane(pr[u], l);
        };
#pragma unroll
        for (int v = 0; v < MT; ++v) {
            tv[v] = v * kWave + lane < nt;
            tr[v] = SwRec{0u, 0u, 0u, 0u, 0u, 0u, 0u};
            if (v * kWave < nt) tr[v] = sw_load(s_t, min(v * kWave + lane, nt - 1));
        }
        // ord S of lanes without an entry: 0, below every score (ord32 of
        // -inf is 0x007fffff), so that comparisons of S need no masks
#pragma unroll
        for (int u = 0; u < MP; ++u) pS[u] = pv[u] ? pS[u] : 0u;
#pragma unroll
        for (int v = 0; v < MT; ++v) tr[v].o = tv[v] ? tr[v].o : 0u;
        if (tid == 0) s_np[cur ^ 1] = 0;  // last read a sweep ago, before two barriers

        // Push candidates: task 2u scores the first-child chains of slot u
        // (of the entries that end a chain), task 2u + 1 the next siblings, on
        // wave 3 - task mod 4.  With at most four slots per lane, slot 0's two
        // tasks are scored before the merge (whether an entry enters T is only
        // known after it), so that with one slot in use they overlap the
        // counting of waves 0 and 1; every other task is scored after it.
        constexpr bool EARLY = MP <= 4;
        auto owner = [&](int t) { return NWV - 1 - t % NWV; };
        auto score_chain = [&](const SwRec& w, bool valid, SwRec (&c)[CL], bool (&ok)[CL])
                               __attribute__((always_inline)) {
            SwRec par = w;
            bool okp = valid & ((par.meta & kChainEnd) != 0u);
#pragma unroll
            for (int i = 0; i < CL; ++i) {
                ok[i] = okp & first_child(par, false, i == CL - 1, c[i]);
                par = c[i];
                okp = ok[i];
            }
        };
        auto score_sibling = [&](const SwRec& w, bool valid, SwRec& c, bool& ok) __attribute__((always_inline)) {
            // next sibling (depth d, drafter row d - 1, the parent's context)
            const int d = (int)(w.meta >> 4) & 63, r = (int)(w.meta & 15);
            const int rp = (int)(w.meta >> 10) & 15, rg = (int)(w.meta >> 14) & 15;
            const int srow = min(max(d - 1, 0), D - 1);
            int sr;
            float sS;
            const uint32_t so =
                child(srow, d - 1 >= 2 ? rg : 0, d - 1 >= 1 ? rp : 0, unord32(w.po), false, w.o, r, sr, sS);
            c = SwRec{so, w.k0, w.k1, w.k2, w.k3, w.po,
                      (uint32_t)sr | ((uint32_t)d << 4) | ((uint32_t)rp << 10) | ((uint32_t)rg << 14) | kChainEnd};
            c = with_digit(c, max(d, 1), sr);
            ok = valid & (so != 0u);
        };
        SwRec ea[CL], eb = SwRec{0u, 0u, 0u, 0u, 0u, 0u, 0u};
        bool oea[CL], oeb = false;
#pragma unroll
        for (int i = 0; i < CL; ++i) {
            oea[i] = false;
            ea[i] = SwRec{0u, 0u, 0u, 0u, 0u, 0u, 0u};
        }
        if (EARLY) {
            if (owner(0) == wv) score_chain(prec(0), pv[0], ea, oea);
            if (owner(1) == wv) score_sibling(prec(0), pv[0], eb, oeb);
        }

        // merged places: a T entry moves down by the P entries before it; a P
        // entry lands after the T and P entries before it.  Each P entry in
        // turn is read from its lane and compared with all entries at once,
        // on S alone unless some S equals its S (then the keys decide); wave
        // w takes the entries l = w (mod 4) of every slot.  AT, AP: the slots
        // that hold entries this sweep.
        int tc[MT], pc[MP];
#pragma unroll
        for (int v = 0; v < MT; ++v) tc[v] = 0;
#pragma unroll
        for (int u = 0; u < MP; ++u) pc[u] = 0;
        // Counts for the P entries at lanes l0 and l1 (l1 < 0: none) of slot
        // u, written so that the two entries' instructions interleave.  Lane
        // masks straight from the compares: T entries before y, T entries y
        // precedes, P entries y precedes; equal S (rare) falls back to keys.
        auto count = [&](auto at, auto ap) __attribute__((always_inline)) {
            constexpr int AT = decltype(at)::value, AP = decltype(ap)::value;
            auto tie_fix = [&](const SwRec& y, int u, int l, int& before) __attribute__((always_inline)) {
                const uint32_t yo = y.o;
#pragma unroll
                for (int v = 0; v < AT; ++v) {
                    const bool e = tr[v].o == yo;
                    const bool g = sw_key_less(tr[v], y);
                    before += __popcll(__ballot(e & g));
                    tc[v] += (e & !g) ? 1 : 0;
                }
#pragma unroll
                for (int q = 0; q < AP; ++q) {
                    const bool e = (pS[q] == yo) & !((q == u) & (lane == l));
                    if (__ballot(e) != 0ull) pc[q] += (e & sw_key_less(y, prec(q))) ? 1 : 0;
                }
            };
#pragma unroll
            for (int u = 0; u < AP; ++u) {
                const int cnt = min(kWave, np - u * kWave);
                for (int l0 = wv; l0 < cnt; l0 += 2 * NWV) {
                    const int l1 = l0 + NWV < cnt ? l0 + NWV : l0;
                    const bool two = l1 != l0;
                    const uint32_t y0 = (uint32_t)__builtin_amdgcn_readlane((int)pS[u], l0);
                    const uint32_t y1 = (uint32_t)__builtin_amdgcn_readlane((int)pS[u], l1);
                    int b0 = 0, b1 = 0;
                    uint64_t e0 = 0ull, e1 = 0ull;
#pragma unroll
                    for (int v = 0; v < AT; ++v) {
                        b0 += __popcll(__builtin_amdgcn_uicmp(tr[v].o, y0, 34));  // T before y: greater ord S
                        b1 += __popcll(__builtin_amdgcn_uicmp(tr[v].o, y1, 34));
                        tc[v] += (tr[v].o < y0 ? 1 : 0) + ((two & (tr[v].o < y1)) ? 1 : 0);
                        e0 |= __builtin_amdgcn_uicmp(tr[v].o, y0, 32);
                        e1 |= __builtin_amdgcn_uicmp(tr[v].o, y1, 32);
                    }
#pragma unroll
                    for (int q = 0; q < AP; ++q) {
                        pc[q] += (pS[q] < y0 ? 1 : 0) + ((two & (pS[q] < y1)) ? 1 : 0);
                        const uint64_t self0 = q == u ? 1ull << l0 : 0ull, self1 = q == u ? 1ull << l1 : 0ull;
                        e0 |= __builtin_amdgcn_uicmp(pS[q], y0, 32) & ~self0;
                        e1 |= __builtin_amdgcn_uicmp(pS[q], y1, 32) & ~self1;
                    }
                    if (e0 != 0ull) tie_fix(prec_at(u, l0), u, l0, b0);
                    if (two && e1 != 0ull) tie_fix(prec_at(u, l1), u, l1, b1);
                    pc[u] += (lane == l0 ? b0 : 0) + ((two & (lane == l1)) ? b1 : 0);
                }
            }
        };
        auto count_p = [&](auto at) __attribute__((always_inline)) {
            if (np <= kWave) count(at, SlotCount<1>{});
            else if (MP <= 2 || np <= 2 * kWave) count(at, SlotCount<(MP < 2 ? MP : 2)>{});
            else if (MP <= 4 || np <= 4 * kWave) count(at, SlotCount<(MP < 4 ? MP : 4)>{});
            else count(at, SlotCount<MP>{});
        };
        if (nt <= kWave) count_p(SlotCount<1>{});
        else if (MT <= 2 || nt <= 2 * kWave) count_p(SlotCount<(MT < 2 ? MT : 2)>{});
        else count_p(SlotCount<MT>{});

        // sum of the four waves' counts
        int32_t* my_cnt = s_cnt + wv * (MT + MP) * kWave;
#pragma unroll
        for (int v = 0; v < MT; ++v)
            if (v * kWave < nt) my_cnt[v * kWave + lane] = tc[v];
#pragma unroll
        for (int u = 0; u < MP; ++u)
            if (u * kWave < np) my_cnt[(MT + u) * kWave + lane] = pc[u];
        __syncthreads();
#pragma unroll
        for (int v = 0; v < MT; ++v) {
            if (v * kWave < nt) {
                int c = 0;
#pragma unroll
                for (int w = 0; w < NWV; ++w) c += s_cnt[(w * (MT + MP) + v) * kWave + lane];
                tc[v] = c;
            }
        }
#pragma unroll
        for (int u = 0; u < MP; ++u) {
            if (u * kWave < np) {
                int c = 0;
#pragma unroll
                for (int w = 0; w < NWV; ++w) c += s_cnt[(w * (MT + MP) + MT + u) * kWave + lane];
                pc[u] = c;
            }
        }

        // moved T entries and the P entries that made it go to their places
        // (every wave read every record before the barrier); slot j of the
        // two lists is stored by wave j mod 4
#pragma unroll
        for (int v = 0; v < MT; ++v) {
            const int to = v * kWave + lane + tc[v];
            if (v % NWV == wv && v * kWave < nt && (tv[v] & (tc[v] != 0) & (to < NB))) sw_store(s_t, to, tr[v]);
        }
#pragma unroll
        for (int u = 0; u < MP; ++u)
            if ((MT + u) % NWV == wv && u * kWave < np && (pv[u] & (pc[u] < NB))) sw_store(s_t, pc[u], prec(u));
        const int nt_new = min(NB, nt + np);
        const bool full = nt_new == NB;
        // T's last entry, from the registers
        SwRec last = SwRec{0u, 0u, 0u, 0u, 0u, 0u, 0u};
        if (full) {
#pragma unroll
            for (int v = 0; v < MT; ++v) {
                if (v * kWave < nt) {
                    const uint64_t m = __ballot(tv[v] & (v * kWave + lane + tc[v] == NB - 1));
                    if (m) last = sw_readlane(tr[v], __ffsll((unsigned long long)m) - 1);
                }
            }
#pragma unroll
            for (int u = 0; u < MP; ++u) {
                if (u * kWave < np) {
                    const uint64_t m = __ballot(pv[u] & (pc[u] == NB - 1));
                    if (m) last = prec_at(u, __ffsll((unsigned long long)m) - 1);
                }
            }
        }

        // pushes of the P entries that entered T, while T is not full or when
        // they precede its last entry; a task takes its places in the next P
        // with one atomic
        auto push = [&](auto& h, auto& c) __attribute__((always_inline)) {
            constexpr int n = sizeof(h) / sizeof(h[0]);
            uint64_t m[n];
            int total = 0;
#pragma unroll
            for (int i = 0; i < n; ++i) {
                m[i] = __ballot(h[i]);
                total += __popcll(m[i]);
            }
            if (total == 0) return;
            int base = 0;
            if (lane == 0) base = atomicAdd(&s_np[cur ^ 1], total);
            base = __builtin_amdgcn_readlane(base, 0);
#pragma unroll
            for (int i = 0; i < n; ++i) {
                const int at = base + lanes_below(m[i]);
                if (h[i] & (at < cap_p)) sw_store(s_pn, at, c[i]);
                base += __popcll(m[i]);
            }
        };
#pragma unroll
        for (int u = 0; u < MP; ++u) {
            if (u * kWave >= np) break;
            const bool in = pv[u] & (pc[u] < NB);
            if (owner(2 * u) == wv) {
                SwRec c[CL];
                bool ok[CL];
                if (EARLY && u == 0) {
#pragma unroll
                    for (int i = 0; i < CL; ++i) {
                        c[i] = ea[i];
                        ok[i] = oea[i];
                    }
                } else {
                    score_chain(prec(u), pv[u], c, ok);
                }
                bool h[CL];
#pragma unroll
                for (int i = 0; i < CL; ++i) h[i] = ok[i] & in & (!full | sw_before(c[i], last));
                push(h, c);
            }
            if (owner(2 * u + 1) == wv) {
                SwRec c[1] = {eb};
                bool ok = oeb;
                if (!(EARLY && u == 0)) score_sibling(prec(u), pv[u], c[0], ok);
                bool h[1] = {(bool)(ok & in & (!full | sw_before(c[0], last)))};
                push(h, c);
            }
        }
        nt = nt_new;
        __syncthreads();
        cur ^= 1;
        np = min(s_np[cur], cap_p);
        if (PL) {
            uint4* t = s_pc;
            s_pc = s_pn;
            s_pn = t;
        }
    }

    // parents: node i >= 1 is T's position i - 1; the parent of a node of
    // depth d > 1 is the T entry with the parent's (S, key), found by binary
    // search (it precedes the node, so its position is smaller)
    if (tid == 0) s_par[0] = -1;
    const int top = nt > 0 ? 1 << (31 - __clz(nt)) : 0;
    for (int p = tid; p < nt; p += NT) {
        const SwRec x = sw_load(s_t, p);
        const int d = (int)(x.meta >> 4) & 63;
        int par = 0;
        if (d > 1) {
            SwRec tg = x;
            tg.o = x.po;
            const uint32_t t = (uint32_t)(d - 1);
            const uint32_t wi = (t * pw_magic) >> 16;
            const uint32_t sh = 32u - (t - wi * (uint32_t)per_word + 1u) * (uint32_t)wbits;
            const uint32_t m = ~(((1u << wbits) - 1u) << sh);
            tg.k0 &= wi == 0 ? m : ~0u;
            tg.k1 &= wi == 1 ? m : ~0u;
            tg.k2 &= wi == 2 ? m : ~0u;
            tg.k3 &= wi == 3 ? m : ~0u;
            int q = 0;
            for (int step = top; step > 0; step >>= 1) {
                const int c = q + step;
                if (c <= nt && sw_before(sw_load(s_t, c - 1), tg)) q = c;
            }
            par = min(q + 1, p);
        }
        s_par[p + 1] = par;
    }
    __syncthreads();

    // output rows and ancestor masks (the parent chain, at most D steps)
    constexpr int SLW = MT + 1;  // W = ceil((budget + 1) / 64) <= MT + 1
    const int64_t ob = (int64_t)b * N;
    const int root_tok = __builtin_amdgcn_readfirstlane(a.root_token[b]);
    for (int i = tid; i < N; i += NT) {
        uint64_t words[SLW];
#pragma unroll
        for (int q = 0; q < SLW; ++q) words[q] = 0ull;
        if (i == 0) {
            a.parent[ob] = -1;
            a.token[ob] = root_tok;
            a.depth[ob] = 0;
            a.rank[ob] = -1;
            a.score[ob] = 0.f;
            words[0] = 1ull;
        } else if (i <= nt) {
            const SwRec x = sw_load(s_t, i - 1);
            const int d = (int)(x.meta >> 4) & 63, r = (int)(x.meta & 15);
            a.parent[ob + i] = s_par[i];
            a.token[ob + i] = s_ids[(d - 1) * k + r];
            a.depth[ob + i] = d;
            a.rank[ob + i] = r;
            a.score[ob + i] = unord32(x.o);
            int y = i;
            for (int step = 0; step <= D && y > 0; ++step) {
#pragma unroll
                for (int q = 0; q < SLW; ++q) words[q] |= q == (y >> 6) ? 1ull << (y & 63) : 0ull;
                y = s_par[y];
            }
            words[0] |= 1ull;
        } else {
            a.parent[ob + i] = -1;
            a.token[ob + i] = -1;
            a.depth[ob + i] = -1;
            a.rank[ob + i] = -1;
            a.score[ob + i] = -INFINITY;
        }
#pragma unroll
        for (int q = 0; q < SLW; ++q)
            if (q < W) a.anc[(ob + i) * W + q] = words[q];
    }
    if (tid == 0) a.n_nodes[b] = nt + 1;
}
}  // namespace presto

namespace presto_host {

using namespace presto;

static int align16(int x) { return (x + 15) & ~15; }

struct TreeLayout {
    int total_no_rho, total_with_rho;
    int o_lp, o_ids, o_kord, o_krank, o_rec, o_pkey, o_ktab, o_beam, o_kbeam, o_rho;
};

static TreeLayout tree_layout(int D, int k, int N, int Wb) {
    TreeLayout L;
    int off = 0;
    L.o_lp = off; off = align16(off + D * k * 4);
    L.o_ids = off; off = align16(off + D * k * 4);
    L.o_kord = off; off = align16(off + N * k * 4);
    L.o_krank = off; off = align16(off + N * k);
    L.o_ktab = off; off = align16(off + (D + 1) * Wb * k);
    L.o_beam = off; off = align16(off + 2 * Wb * (int)sizeof(BeamEntry));
    L.o_kbeam = off; off = align16(off + (Wb > 0 ? N * k : 0));  // beam search only
    L.o_rec = off; off = align16(off + N * 8);
    L.o_pkey = off; off = align16(off + N * 16);
    L.total_no_rho = off;
    L.o_rho = off;
    L.total_with_rho = align16(off + D * k * k * k * 4);
    return L;
}

// gfx950 gives one workgroup up to 160 KiB of LDS; the search runs one wave
// per CU anyway, so the lattice stays in LDS whenever the total fits.
static constexpr int kTreeLdsBudget = 160 * 1024;
static constexpr int kDefaultLds = 64 * 1024;

// Dynamic LDS above the default needs the kernel's own limit raised (once
// per instantiation and process).
template <typename K>
static presto_status allow_lds(K* kernel, int bytes) {
    if (bytes <= kDefaultLds) return PRESTO_OK;
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (e != hipSuccess)
        return set_error(PRESTO_ERR_HIP, "tree build: %d bytes of LDS refused: %s", bytes,
                         hipGetErrorString(e));
    return PRESTO_OK;
}

int tree_key_bits(int k) {
    int wbits = 1;
    while ((1 << wbits) < k + 1) ++wbits;
    return wbits;
}

// Deepest tree whose rank-path key fits four 32-bit words (digits never
// straddle a word).
int tree_max_depth(int k) { return 4 * (32 / tree_key_bits(k)); }

// Literal Alg. 2: candidate table, then T (capacity budget + branch - 1:
// the last expansion may overshoot the budget), then the lattice.
struct Alg2Layout {
    int cap, total_no_rho, total_with_rho;
    int o_lp, o_ids, o_tmeta, o_tS, o_tkey, o_tplace, o_rho;
};

static Alg2Layout alg2_layout(int D, int k, int branch, int budget) {
    Alg2Layout L;
    L.cap = budget + branch - 1;
    int off = 0;
    L.o_lp = off; off = align16(off + D * k * 4);
    L.o_ids = off; off = align16(off + D * k * 4);
    L.o_tmeta = off; off = align16(off + L.cap * 4);
    L.o_tS = off; off = align16(off + L.cap * 4);
    L.o_tkey = off; off = align16(off + L.cap * 16);
    L.o_tplace = off; off = align16(off + L.cap * 4);
    L.total_no_rho = off;
    L.o_rho = off;
    L.total_with_rho = align16(off + D * k * k * k * 4);
    return L;
}

// Frontier sweeps: candidate table, lambda, T, P (capacity 2 budget), the
// parent positions, then the lattice.
struct SweepLayout {
    int total_no_rho, total_with_rho;
    int o_lp, o_ids, o_lam, o_t, o_p, o_p2, o_par, o_cnt, o_np, o_rho;
};

// slots per lane of T and P for a budget (the kernel's MT and MP)
static int sweep_mt(int budget) { return budget <= 64 ? 1 : (budget <= 128 ? 2 : (budget <= 256 ? 4 : 8)); }
// chains of three first children at budgets <= 64 (8 -> 6 sweeps at depth 16 against chains of
// two, 15 with none); at larger budgets the trees are wider and chains added entries without
// removing sweeps
static int sweep_chain(int budget) { return sweep_mt(budget) == 1 ? 3 : 1; }
static int sweep_mp(int budget) { return (sweep_chain(budget) + 1) * sweep_mt(budget); }

static SweepLayout sweep_layout(int D, int k, int N) {
    SweepLayout L;
    const int nb = N - 1;
    int off = 0;
    L.o_lp = off; off = align16(off + D * k * 4);
    L.o_ids = off; off = align16(off + D * k * 4);
    L.o_lam = off; off = align16(off + D * 4);
    L.o_t = off; off = align16(off + nb * 32);
    L.o_p = off; off = align16(off + (sweep_chain(nb) + 1) * nb * 32);
    L.o_p2 = off; off = align16(off + (sweep_mt(nb) >= 8 ? (sweep_chain(nb) + 1) * nb * 32 : 0));  // P's second buffer
    L.o_par = off; off = align16(off + N * 4);
    L.o_cnt = off; off = align16(off + kSweepWaves * (sweep_mt(nb) + sweep_mp(nb)) * kWave * 4);
    L.o_np = off; off = align16(off + 2 * 4);
    L.total_no_rho = off;
    L.o_rho = off;
    L.total_with_rho = align16(off + D * k * k * k * 4);
    return L;
}

// Budgets the sweep kernel takes: above 512 the slots per lane would not
// fit (T's records stay in registers); at 32 and below popping one node at
// a time is faster (a sweep costs about three pops, and a tree of depth 16
// needs about 14 sweeps).
static constexpr int kSweepMinBudget = 33;
static constexpr int kSweepMaxBudget = 512;

bool tree_build_fits(int D, int k, int branch, int N, int beam_width, bool alg2) {
    if (alg2) return alg2_layout(D, k, branch, N - 1).total_no_rho <= kTreeLdsBudget;
    return tree_layout(D, k, N, beam_width).total_no_rho <= kTreeLdsBudget;
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
    a.wbits = tree_key_bits(a.k);
    a.per_word = 32 / a.wbits;
    a.ids = ids;
    a.logprob = logprob;
    a.log_rho = log_rho;
    a.lambda = lambda;
    a.lambda_stride = desc->lambda_per_seq ? desc->depth : 0;
    a.root_token = root_token;
    a.n_nodes = n_nodes;
    a.parent = parent;
    a.token = token;
    a.depth = depth;
    a.rank = rank;
    a.score = score;
    a.anc = anc;
    if (desc->mode == PRESTO_TREE_BEST_FIRST_ALG2) {
        const Alg2Layout L = alg2_layout(a.D, a.k, a.branch, a.budget);
        a.beam_width = 0;
        a.o_lp = L.o_lp; a.o_ids = L.o_ids; a.o_rho = L.o_rho;
        a.o_tmeta = L.o_tmeta; a.o_tS = L.o_tS; a.o_tkey = L.o_tkey; a.o_tplace = L.o_tplace;
        a.rho_in_lds = log_rho != nullptr && L.total_with_rho <= kTreeLdsBudget;
        const int lds = a.rho_in_lds ? L.total_with_rho : L.total_no_rho;
        const int slt = (L.cap + kWave - 1) / kWave;
        const int rho_mode = log_rho == nullptr ? 0 : (a.rho_in_lds ? 1 : 2);
        presto_status st = PRESTO_OK;
        auto go = [&](auto kernel) {
            st = allow_lds(kernel, lds);
            if (st == PRESTO_OK) kernel<<<desc->batch, kWave, lds, stream>>>(a);
        };
#define PRESTO_ALG2(S)                                    \
    if (rho_mode == 0) go(tree_alg2_kernel<S, 0>);        \
    else if (rho_mode == 1) go(tree_alg2_kernel<S, 1>);   \
    else go(tree_alg2_kernel<S, 2>)
        if (slt <= 1) { PRESTO_ALG2(1); }
        else if (slt <= 2) { PRESTO_ALG2(2); }
        else if (slt <= 4) { PRESTO_ALG2(4); }
        else if (slt <= 9) { PRESTO_ALG2(9); }
        else { PRESTO_ALG2(17); }
#undef PRESTO_ALG2
        if (st != PRESTO_OK) return st;
        return check_launch("tree_alg2_kernel");
    }
    const bool beam = desc->mode == PRESTO_TREE_BEAM;
    if (!beam && a.budget >= kSweepMinBudget && a.budget <= kSweepMaxBudget) {
        const SweepLayout L = sweep_layout(a.D, a.k, a.N);
        a.beam_width = 0;
        a.o_lp = L.o_lp; a.o_ids = L.o_ids; a.o_lam = L.o_lam; a.o_rho = L.o_rho;
        a.o_sw_t = L.o_t; a.o_sw_p = L.o_p; a.o_sw_p2 = L.o_p2; a.o_sw_par = L.o_par; a.o_sw_cnt = L.o_cnt;
        a.o_sw_np = L.o_np;
        a.rho_in_lds = log_rho != nullptr && L.total_with_rho <= kTreeLdsBudget;
        const uint64_t k3 = (uint64_t)a.k * a.k * a.k;
        a.mag_k = (uint32_t)(((1ull << 32) + a.k - 1) / a.k);        // k > 1 only
        a.mag_k3 = (uint32_t)(((1ull << 32) + k3 - 1) / k3);
        const int lds = a.rho_in_lds ? L.total_with_rho : L.total_no_rho;
        const int rho_mode = log_rho == nullptr ? 0 : (a.rho_in_lds ? 1 : 2);
        presto_status st = PRESTO_OK;
        auto go = [&](auto kernel) {
            st = allow_lds(kernel, lds);
            if (st == PRESTO_OK) kernel<<<desc->batch, kSweepWaves * kWave, lds, stream>>>(a);
        };
#define PRESTO_SWEEP3(T, P, K, C)                                    \
    if (rho_mode == 0) go(tree_sweep_kernel<T, P, K, 0, C>);        \
    else if (rho_mode == 1) go(tree_sweep_kernel<T, P, K, 1, C>);   \
    else go(tree_sweep_kernel<T, P, K, 2, C>)
#define PRESTO_SWEEP(T, P, C)                                        \
    if (a.k <= 4) { PRESTO_SWEEP3(T, P, 4, C); }                     \
    else if (a.k <= 8) { PRESTO_SWEEP3(T, P, 8, C); }                \
    else { PRESTO_SWEEP3(T, P, 16, C); }
        const int mt = sweep_mt(a.budget);
        if (mt == 1) { PRESTO_SWEEP(1, 4, 3) }
        else if (mt == 2) { PRESTO_SWEEP(2, 4, 1) }
        else if (mt == 4) { PRESTO_SWEEP(4, 8, 1) }
        else { PRESTO_SWEEP(8, 16, 1) }
#undef PRESTO_SWEEP
#undef PRESTO_SWEEP3
        if (st != PRESTO_OK) return st;
        return check_launch("tree_sweep_kernel");
    }
    a.beam_width = beam ? desc->beam_width : 0;
    const TreeLayout L = tree_layout(a.D, a.k, a.N, a.beam_width);
    a.o_lp = L.o_lp; a.o_ids = L.o_ids; a.o_kord = L.o_kord; a.o_krank = L.o_krank; a.o_rec = L.o_rec;
    a.o_pkey = L.o_pkey;
    a.o_ktab = L.o_ktab; a.o_beam = L.o_beam; a.o_kbeam = L.o_kbeam;
    a.o_rho = L.o_rho;
    a.rho_in_lds = log_rho != nullptr && L.total_with_rho <= kTreeLdsBudget;
    const int lds = a.rho_in_lds ? L.total_with_rho : L.total_no_rho;
    const int SL = (a.N + kWave - 1) / kWave;
    const int rho_mode = log_rho == nullptr ? 0 : (a.rho_in_lds ? 1 : 2);
    presto_status st = PRESTO_OK;
    auto go = [&](auto kernel) {
        st = allow_lds(kernel, lds);
        if (st == PRESTO_OK) kernel<<<desc->batch, kWave, lds, stream>>>(a);
    };
#define PRESTO_TREE4(S, R, Q)                         \
    if (beam) go(tree_build_kernel<S, R, Q, true>);   \
    else go(tree_build_kernel<S, R, Q, false>)
#define PRESTO_TREE2(S, R) \
    if (a.k <= 4) { PRESTO_TREE4(S, R, true); } else { PRESTO_TREE4(S, R, false); }
#define PRESTO_TREE(S)                      \
    if (rho_mode == 0) { PRESTO_TREE2(S, 0); } \
    else if (rho_mode == 1) { PRESTO_TREE2(S, 1); } \
    else { PRESTO_TREE2(S, 2); }
    if (SL <= 1) { PRESTO_TREE(1) }
    else if (SL <= 2) { PRESTO_TREE(2) }
    else if (SL <= 3) { PRESTO_TREE(3) }
    else if (SL <= 4) { PRESTO_TREE(4) }
    else if (SL <= 5) { PRESTO_TREE(5) }
    else if (SL <= 8) { PRESTO_TREE(8) }
    else { PRESTO_TREE(16) }
#undef PRESTO_TREE
#undef PRESTO_TREE2
#undef PRESTO_TREE4
    if (st != PRESTO_OK) return st;
    return check_launch("tree_build_kernel");
}

}  // namespace presto_host
