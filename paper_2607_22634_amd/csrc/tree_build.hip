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
