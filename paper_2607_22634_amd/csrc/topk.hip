// Stage 1: log-softmax normaliser and top-k candidates per drafter position.
//
// The vocabulary row of each position is streamed from HBM once.  A row is
// cut into wave-sized chunks; every wave holds its chunk in registers and
// produces, with no block-level synchronisation:
//   * the chunk maximum m and sum exp(z - m)           (for the row's LSE)
//   * the chunk's k best (value desc, id asc) entries  (as 64-bit keys)
// The k-th largest lane maximum (k rounds of wave max, or a ballot bisection
// on its orderable bits for k > 8) is a lower bound on the chunk's k-th value, so only the
// 16-byte groups whose maximum reaches it can hold a top-k entry (at least
// k of them, normally about k); they are appended to a per-wave LDS list of
// up to 256 values and their entries at or above the bound are keyed.  With
// bf16 values, up to 64 such entries take one lane each and are placed in
// the output by their rank among them; otherwise (and for fp32) the k best
// are taken by k rounds of wave max over up to four keys per lane.  A
// chunk with more candidate groups than the list holds (massive ties) falls
// back to k rounds of exact wave-wide selection over the chunk re-read from
// memory, and marks its partial so that the merge can count such chunks.
// A second kernel, queued right behind, merges each row's chunk partials
// with one wave per row.
#include <math.h>

#include <mutex>

#include "common.hpp"

namespace presto {

constexpr int kMaxDevices = 64;
constexpr int kCandCap = 256;  // values of candidate groups a wave's list holds
constexpr int kTopkWavesPerBlock = 4;
constexpr float kLog2eF = 1.4426950408889634f;

template <bool BF16>
struct VecTraits;
template <>
struct VecTraits<true> {
    static constexpr int kPerVec = 8;
};
template <>
struct VecTraits<false> {
    static constexpr int kPerVec = 4;
};

// Element e of a lane's register block: load i = e / kPerVec, j = e % kPerVec;
// vocabulary index c0 + (i * 64 + lane) * kPerVec + j.
template <bool BF16, int NLOAD>
__device__ __forceinline__ void load_chunk(const void* __restrict__ row, int64_t c0, int32_t vocab,
                                           bool vec_ok, float (&v)[NLOAD * VecTraits<BF16>::kPerVec]) {
    constexpr int P = VecTraits<BF16>::kPerVec;
    const int lane = lane_id();
    if (vec_ok) {
        const uint4* src = reinterpret_cast<const uint4*>(
            static_cast<const char*>(row) + c0 * (BF16 ? 2 : 4));
        uint4 raw[NLOAD];
#pragma unroll
        for (int i = 0; i < NLOAD; ++i) raw[i] = load_stream16(&src[i * kWave + lane]);
#pragma unroll
        for (int i = 0; i < NLOAD; ++i) {
            const uint32_t w[4] = {raw[i].x, raw[i].y, raw[i].z, raw[i].w};
            if constexpr (BF16) {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    v[i * P + 2 * j] = bf16lo(w[j]);
                    v[i * P + 2 * j + 1] = bf16hi(w[j]);
                }
            } else {
#pragma unroll
                for (int j = 0; j < 4; ++j) v[i * P + j] = __uint_as_float(w[j]);
            }
        }
    } else {
#pragma unroll
        for (int i = 0; i < NLOAD; ++i) {
#pragma unroll
            for (int j = 0; j < P; ++j) {
                const int64_t idx = c0 + (int64_t)(i * kWave + lane) * P + j;
                float x = -INFINITY;
                if (idx < vocab) {
                    if constexpr (BF16)
                        x = bf16_to_f(static_cast<const uint16_t*>(row)[idx]);
                    else
                        x = static_cast<const float*>(row)[idx];
                }
                v[i * P + j] = x;
            }
        }
    }
}

// The k-th largest value of one u32 per lane (k <= 64).  Small k: k rounds
// of "wave max, then retire one lane holding it"; larger k: bisection on the
// top BITS bits (the others of every x are equal: 16 for ord32 of bf16
// values), counting lanes at or above each probe with a ballot.
template <int BITS = 32>
__device__ __forceinline__ uint32_t wave_kth_largest_u32(uint32_t x, int k) {
    if (k <= (BITS == 32 ? 8 : 4)) {
        const int lane = lane_id();
        uint32_t t = 0u;
        for (int j = 0; j < k; ++j) {
            t = wave_max_u32_dpp(x);
            const int l = __ffsll((unsigned long long)__ballot(x == t)) - 1;
            x = lane == l ? 0u : x;
        }
        return t;
    }
    uint32_t t = 0u;
#pragma unroll
    for (int bit = 31; bit >= 32 - BITS; --bit) {
        const uint32_t c = t | (1u << bit);
        if (__popcll(__ballot(x >= c)) >= k) t = c;
    }
    return t;
}

// ENT: also the chunk's sum of exp(z - m) * (z - m), for the entropy of q.
template <bool BF16, int NLOAD, bool ENT>
__global__ __launch_bounds__(kTopkWavesPerBlock * kWave) void topk_partial_kernel(
    const void* __restrict__ logits, int64_t rows, int32_t vocab, int64_t row_stride, int32_t k,
    int32_t chunks, bool aligned, const int64_t* __restrict__ row_index, int64_t logits_rows,
    float2* __restrict__ part_ms, uint64_t* __restrict__ part_keys, float* __restrict__ part_h,
    uint32_t* __restrict__ n_fallback, int32_t* __restrict__ flags) {
    constexpr int P = VecTraits<BF16>::kPerVec;  // elements per 16-byte load (a "group")
    constexpr int E = NLOAD * P;
    constexpr int64_t CH = (int64_t)kWave * E;
    constexpr int kGroupCap = kCandCap / P;      // candidate groups a wave list holds
    // per-wave candidate list: the values of up to kGroupCap groups and the
    // vocabulary index of each group's first element
    __shared__ __align__(16) float cand_v[kTopkWavesPerBlock][kCandCap];
    __shared__ int32_t cand_i[kTopkWavesPerBlock][kGroupCap];
    __shared__ uint32_t cand_n[kTopkWavesPerBlock];
    __shared__ uint32_t rank_keys[kTopkWavesPerBlock][kWave];  // valid bf16 keys, one per lane

    const int wave = threadIdx.x / kWave, lane = lane_id();
    const int64_t gw = (int64_t)blockIdx.x * kTopkWavesPerBlock + wave;
    if (gw == 0 && lane == 0) *n_fallback = 0u;  // counted by the merge kernel
    if (gw >= rows * chunks) return;
    const int64_t row = gw / chunks;
    const int32_t chunk = (int32_t)(gw % chunks);
    const int64_t c0 = (int64_t)chunk * CH;
    // with a row index, output row `row` reads logits row row_index[row]; an
    // index outside the logits reads as an empty row (and is flagged)
    int64_t src = row;
    if (row_index) {
        src = row_index[row];
        if (src < 0 || src >= logits_rows) {
            if (chunk == 0 && lane_id() == 0) raise_flag(flags, PRESTO_FLAG_BAD_INDEX);
            src = 0;
            vocab = 0;
        }
    }
    const char* rowp = static_cast<const char*>(logits) + src * row_stride * (BF16 ? 2 : 4);
    const bool full = aligned && (c0 + CH <= vocab);

    float v[E];
    load_chunk<BF16, NLOAD>(rowp, c0, vocab, full, v);

    // group maxima (one group = the P elements of one 16-byte load), lane max
    float gmax[NLOAD];
#pragma unroll
    for (int i = 0; i < NLOAD; ++i) {
        float m = v[i * P];
#pragma unroll
        for (int j = 1; j < P; ++j) m = fmaxf(m, v[i * P + j]);
        gmax[i] = m;
    }
    float lm = gmax[0];
#pragma unroll
    for (int i = 1; i < NLOAD; ++i) lm = fmaxf(lm, gmax[i]);
    const float M = wave_max_f32_dpp(lm);
    // For moderate M: exp(z - M) = exp2(fma(z, log2 e, -mo)) * 2^-r with
    // mo = fl(M log2 e) and r = M log2 e - mo taken exactly by one fma (|r| is
    // below 2^-16 here), so one fma and one exp per entry.  Larger |M| takes
    // the plain form exp2((z - M) log2 e).
    // Each entry's exponent is x = fl(z log2 e - mo) = (z - M) log2 e + r, so
    // exp(z - M) = 2^x * 2^-r (corr = 2^-r), and with ENT
    // sum exp(z - M) (z - M) = corr * sum 2^x (x - r) / log2 e.
    float s = 0.f, sx = 0.f;
    float corr = 1.f, rr = 0.f;
    if (fabsf(M) < 256.f) {
        const float mo = M * kLog2eF;
        rr = fmaf(M, kLog2eF, -mo);
        corr = __builtin_amdgcn_exp2f(-rr);
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const float x = fmaf(v[e], kLog2eF, -mo);
            const float ex = __builtin_amdgcn_exp2f(x);
            s += ex;
            // a -inf entry (masked, or padding past the row end) has q = 0 and
            // adds nothing; without the select it would add 0 * -inf
            if constexpr (ENT) sx = fmaf(ex, ex != 0.f ? x - rr : 0.f, sx);
        }
    } else if (M != -INFINITY) {
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const float x = (v[e] - M) * kLog2eF;
            const float ex = __builtin_amdgcn_exp2f(x);
            s += ex;
            if constexpr (ENT) sx = fmaf(ex, ex != 0.f ? x : 0.f, sx);
        }
    }
    const float S = wave_sum_f32_dpp(s) * corr;
    float Hx = 0.f;  // sum over the chunk of exp(z - M) (z - M)
    if constexpr (ENT) Hx = wave_sum_f32_dpp(sx) * corr * (1.f / kLog2eF);
    // the k-th largest lane maximum bounds the chunk's k-th value from below:
    // only groups whose maximum reaches it can hold a top-k entry
    // (bf16: ord32 of every value ends in 0x0000 or 0xffff, so the bisection
    // runs over the top 16 bits and the bound is completed below them)
    float thr;
    if constexpr (BF16) {
        const uint32_t t = wave_kth_largest_u32<16>(ord32(lm) & 0xffff0000u, k);
        thr = unord32(t | ((t & 0x80000000u) ? 0u : 0xffffu));
    } else {
        thr = unord32(wave_kth_largest_u32(ord32(lm), k));
    }

    // A lane appends its candidate groups (values as they are) with one LDS
    // atomic for all of them; the keys are formed afterwards, one candidate
    // per lane, so the divergent part stays a few stores per group.
    if (lane == 0) cand_n[wave] = 0u;
    __builtin_amdgcn_wave_barrier();
    uint32_t npass = 0u;
#pragma unroll
    for (int i = 0; i < NLOAD; ++i) npass += gmax[i] >= thr ? 1u : 0u;
    uint32_t q = 0u;
    if (npass != 0u) q = atomicAdd(&cand_n[wave], npass);
#pragma unroll
    for (int i = 0; i < NLOAD; ++i) {
        if (gmax[i] >= thr) {
            if (q < (uint32_t)kGroupCap) {
                float4* dst = reinterpret_cast<float4*>(&cand_v[wave][q * P]);
#pragma unroll
                for (int j = 0; j < P / 4; ++j)
                    dst[j] = make_float4(v[i * P + 4 * j], v[i * P + 4 * j + 1], v[i * P + 4 * j + 2],
                                         v[i * P + 4 * j + 3]);
                cand_i[wave][q] = (int32_t)(c0 + (int64_t)(i * kWave + lane) * P);
            }
            ++q;
        }
    }
    __builtin_amdgcn_wave_barrier();
    const uint32_t ngroups = __builtin_amdgcn_readfirstlane(cand_n[wave]);
    uint64_t* out = part_keys + gw * k;

    const int total = (int)ngroups * P;
    // key of list entry e (0 if it is past the list, past the row or below
    // the bound)
    auto entry_key = [&](int e) -> uint64_t {
        if (e >= total) return 0ull;
        const float xv = cand_v[wave][e];
        const int64_t idx = (int64_t)cand_i[wave][e / P] + e % P;
        return ((full || idx < vocab) && xv >= thr) ? vocab_key(xv, (uint32_t)idx) : 0ull;
    };
    bool fell_back = false;
    // bf16: a chunk-local 32-bit key, the value's 16-bit order code over
    // 0xffff minus the index within the chunk (chunks hold at most 65536
    // entries), orders the entries exactly as the 64-bit vocabulary key
    auto entry_key32 = [&](int e) -> uint32_t {
        if (e >= total) return 0u;
        const float xv = cand_v[wave][e];
        const int64_t idx = (int64_t)cand_i[wave][e / P] + e % P;
        return ((full || idx < vocab) && xv >= thr)
                   ? (ord32(xv) & 0xffff0000u) | (0xffffu - (uint32_t)(idx - c0))
                   : 0u;
    };
    auto key64 = [&](uint32_t k32) -> uint64_t {
        const uint32_t o = k32 & 0xffff0000u;
        const float xv = unord32(o | ((o & 0x80000000u) ? 0u : 0xffffu));
        return vocab_key(xv, (uint32_t)(c0 + (0xffffu - (k32 & 0xffffu))));
    };
    if (BF16 && total <= kCandCap && ngroups <= (uint32_t)kGroupCap) {
        constexpr int C = kCandCap / kWave;
        uint32_t x[C];
#pragma unroll
        for (int c = 0; c < C; ++c) x[c] = (c == 0 || total > c * kWave) ? entry_key32(c * kWave + lane) : 0u;
        // The valid keys (nonzero: at or above the bound) are usually about
        // k.  Up to a wave of them are packed one per lane, and each finds its
        // output place as its rank among them (keys are unique): one compare
        // per valid key instead of k wave-wide maxima.
        uint64_t bal[C];
        int nv = 0;
#pragma unroll
        for (int c = 0; c < C; ++c) {
            bal[c] = __ballot(x[c] != 0u);
            nv += __popcll(bal[c]);
        }
        if (nv <= kWave) {
            int pos = 0;
#pragma unroll
            for (int c = 0; c < C; ++c) {
                const int below = (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(bal[c] >> 32),
                                                                 __builtin_amdgcn_mbcnt_lo((uint32_t)bal[c], 0u));
                if (x[c] != 0u) rank_keys[wave][pos + below] = x[c];
                pos += __popcll(bal[c]);
            }
            __builtin_amdgcn_wave_barrier();
            const uint32_t my = lane < nv ? rank_keys[wave][lane] : 0u;
            int rank = 0;
            for (int j = 0; j < nv; ++j)
                rank += (uint32_t)__builtin_amdgcn_readlane((int)my, j) > my ? 1 : 0;
            if (lane < nv) {
                if (rank < k) out[rank] = key64(my);
            } else if (lane < k) {
                out[lane] = 0ull;  // fewer than k valid entries
            }
        } else {
            uint32_t mine = 0u;
            const int nc = (total + kWave - 1) / kWave;  // slots holding entries
            for (int j = 0; j < k; ++j) {
                uint32_t lmax = x[0];
#pragma unroll
                for (int c = 1; c < C; ++c) lmax = (c < nc && x[c] > lmax) ? x[c] : lmax;
                const uint32_t m = wave_max_u32_dpp(lmax);
                mine = lane == j ? m : mine;
#pragma unroll
                for (int c = 0; c < C; ++c) x[c] = x[c] == m ? 0u : x[c];
            }
            if (lane < k) out[lane] = mine ? key64(mine) : 0ull;
        }
    } else if (total <= kWave) {
        // one candidate per lane (keys are unique); k rounds of wave max,
        // retiring the lane that held it (0 past the last valid entry)
        uint64_t x = entry_key(lane);
        uint64_t mine = 0ull;
        for (int j = 0; j < k; ++j) {
            const uint64_t m = wave_max_u64_dpp(x);
            mine = lane == j ? m : mine;
            x = x == m ? 0ull : x;
        }
        if (lane < k) out[lane] = mine;
    } else if (ngroups <= (uint32_t)kGroupCap) {
        // up to four candidates per lane (the usual case for k > 8)
        constexpr int C = kCandCap / kWave;
        uint64_t x[C];
#pragma unroll
        for (int c = 0; c < C; ++c) x[c] = entry_key(c * kWave + lane);
        uint64_t mine = 0ull;
        for (int j = 0; j < k; ++j) {
            uint64_t lmax = x[0];
#pragma unroll
            for (int c = 1; c < C; ++c) lmax = x[c] > lmax ? x[c] : lmax;
            const uint64_t m = wave_max_u64_dpp(lmax);
            mine = lane == j ? m : mine;
#pragma unroll
            for (int c = 0; c < C; ++c) x[c] = x[c] == m ? 0ull : x[c];
        }
        if (lane < k) out[lane] = mine;
    } else {
        fell_back = true;
        // massive ties: exact selection, k rounds of "largest key below the
        // last one", re-reading the chunk from memory (rare; keeps the
        // register copy of the chunk out of this path)
        uint64_t last = ~0ull;
        for (int j = 0; j < k; ++j) {
            uint64_t best = 0ull;
#pragma unroll 1
            for (int e = 0; e < E; ++e) {
                const int64_t idx = c0 + (int64_t)((e / P) * kWave + lane) * P + (e % P);
                if (idx < vocab) {
                    const float x = BF16 ? bf16_to_f(reinterpret_cast<const uint16_t*>(rowp)[idx])
                                         : reinterpret_cast<const float*>(rowp)[idx];
                    const uint64_t key = vocab_key(x, (uint32_t)idx);
                    if (key < last && key > best) best = key;
                }
            }
            last = wave_max_u64_dpp(best);
            if (lane == 0) out[j] = last;
        }
    }
    if (lane == 0) {
        // the sum is never negative: its sign bit marks a chunk that took the
        // exact fallback
        part_ms[gw] = make_float2(M, fell_back ? -S : S);
        if constexpr (ENT) part_h[gw] = Hx;
        if (!(S == S)) raise_flag(flags, PRESTO_FLAG_NAN_DRAFTER);
    }
}

// One wave per row: LSE from the chunk (max, sum) pairs, then the k best of
// the chunk keys by k rounds of wave-wide selection over keys held in
// registers (KPL per lane; KPL == 0 re-reads them from memory).
// With ENT also the entropy H = -sum q log q = log S - (sum exp(z - M)(z - M)) / S
// of the row, from the chunks' shifted sums.
template <int KPL, bool ENT>
__global__ __launch_bounds__(kTopkWavesPerBlock * kWave) void topk_merge_kernel(
    int64_t rows, int32_t chunks, int32_t k, const float2* __restrict__ part_ms,
    const uint64_t* __restrict__ part_keys, const float* __restrict__ part_h,
    int32_t* __restrict__ ids, float* __restrict__ logprob, float* __restrict__ lse,
    float* __restrict__ entropy, uint32_t* __restrict__ n_fallback) {
    const int wave = threadIdx.x / kWave, lane = lane_id();
    const int64_t row = (int64_t)blockIdx.x * kTopkWavesPerBlock + wave;
    if (row >= rows) return;
    const float2* ms = part_ms + row * chunks;
    const uint64_t* keys = part_keys + row * chunks * k;
    const int nk = chunks * k;

    uint64_t kr[KPL > 0 ? KPL : 1];
    if constexpr (KPL > 0) {
#pragma unroll
        for (int i = 0; i < KPL; ++i) {
            const int idx = i * kWave + lane;
            kr[i] = idx < nk ? keys[idx] : 0ull;
        }
    }
    // the chunks' (max, sum) pairs: the first kMsRegs per lane are read once
    // into registers (every row up to 256 chunks), the rest read again below
    constexpr int kMsRegs = 4;
    float2 mr[kMsRegs];
#pragma unroll
    for (int i = 0; i < kMsRegs; ++i) {
        const int c = i * kWave + lane;
        mr[i] = c < chunks ? ms[c] : make_float2(-INFINITY, 0.f);
    }
    float m = -INFINITY;
    int nfb = 0;  // chunks of this lane that took the exact fallback
#pragma unroll
    for (int i = 0; i < kMsRegs; ++i) {
        m = fmaxf(m, mr[i].x);
        nfb += __builtin_signbit(mr[i].y) ? 1 : 0;
        mr[i].y = fabsf(mr[i].y);
    }
    for (int c = kMsRegs * kWave + lane; c < chunks; c += kWave) {
        m = fmaxf(m, ms[c].x);
        nfb += __builtin_signbit(ms[c].y) ? 1 : 0;
    }
    const float M = wave_max_f32_dpp(m);
    nfb = wave_sum_i32(nfb);
    if (lane == 0 && nfb > 0) atomicAdd(n_fallback, (uint32_t)nfb);
    float s = 0.f, hx = 0.f;
    // chunk sums shift to the row max: (z - M) = (z - m_c) + (m_c - M)
    auto add_chunk = [&](float2 p, int c) {
        if (p.x != -INFINITY) {
            const float w = __expf(p.x - M);
            const float py = fabsf(p.y);
            s += py * w;
            if constexpr (ENT) hx += w * (part_h[row * chunks + c] + (p.x - M) * py);
        }
    };
    if (M != -INFINITY) {
#pragma unroll
        for (int i = 0; i < kMsRegs; ++i) add_chunk(mr[i], i * kWave + lane);
        for (int c = kMsRegs * kWave + lane; c < chunks; c += kWave) add_chunk(ms[c], c);
    }
    const float S = wave_sum_f32_dpp(s);
    const float logS = __logf(S);
    const float L = (M == -INFINITY) ? -INFINITY : M + logS;
    if constexpr (ENT) {
        const float HX = wave_sum_f32_dpp(hx);
        if (lane == 0) entropy[row] = (M == -INFINITY) ? 0.f : logS - HX / S;
    }

    uint64_t last = ~0ull, mine = 0ull;
    for (int j = 0; j < k; ++j) {
        uint64_t best = 0ull;
        if constexpr (KPL > 0) {
#pragma unroll
            for (int i = 0; i < KPL; ++i) best = (kr[i] < last && kr[i] > best) ? kr[i] : best;
        } else {
            for (int i = lane; i < nk; i += kWave) {
                const uint64_t key = keys[i];
                best = (key < last && key > best) ? key : best;
            }
        }
        last = wave_max_u64_dpp(best);
        if (lane == j) mine = last;
    }
    if (lane < k) {
        ids[row * k + lane] = (int32_t)key_id(mine);
        // (z - M) - log S rather than z - L: z - M is exact for the top
        // entries, so large logits do not lose the ulp of L
        logprob[row * k + lane] = (L == -INFINITY) ? -INFINITY : (key_value(mine) - M) - logS;
    }
    if (lse && lane == 0) lse[row] = L;
}

// Entropy-adaptive interpolation weight: lambda = beta * H / (H + C), per row.
__global__ void entropy_lambda_kernel(int64_t rows, const float* __restrict__ entropy, float beta,
                                      float c, float* __restrict__ lambda) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < rows) {
        const float h = entropy[i];
        lambda[i] = beta * (h / (h + c));
    }
}

}  // namespace presto

namespace presto_host {

using namespace presto;

// The workspace starts with the fallback counter (read by callers that want
// the diagnostic), then the partials.
static constexpr size_t kTopkCounterBytes = 16;

static int topk_nload(bool bf16, int64_t rows, int32_t vocab) {
    auto waves = [&](int nl) {
        const int64_t ch = (int64_t)kWave * nl * (bf16 ? 8 : 4);
        return rows * ((vocab + ch - 1) / ch);
    };
    // 8 loads per lane only when that still leaves >= 16 waves per CU (16
    // loads, 165 registers, measured slower at 1024 rows: 58 -> 70 us)
    return waves(8) >= 16 * 256 ? 8 : 4;
}

size_t topk_workspace_bytes(int64_t rows, int32_t vocab, int32_t k) {
    // sized for the finest chunking any dtype may pick
    const int64_t chunks = (vocab + (int64_t)kWave * 16 - 1) / ((int64_t)kWave * 16);
    const size_t per = (size_t)chunks * (sizeof(float2) + sizeof(uint64_t) * (size_t)k + sizeof(float));
    return (size_t)rows * per + 512 + kTopkCounterBytes;
}

presto_status launch_topk(bool bf16, const void* logits, const int64_t* row_index,
                          int64_t logits_rows, int64_t rows, int32_t vocab, int64_t row_stride,
                          int32_t k, int32_t* ids, float* logprob, float* lse, float* entropy,
                          int32_t* flags, void* ws, hipStream_t stream) {
    const int nload = topk_nload(bf16, rows, vocab);
    const int64_t ch = (int64_t)kWave * nload * (bf16 ? 8 : 4);
    const int64_t chunks = (vocab + ch - 1) / ch;
    const size_t esz = bf16 ? 2 : 4;
    const bool aligned = ((uintptr_t)logits % 16 == 0) && ((row_stride * (int64_t)esz) % 16 == 0);
    uint32_t* n_fallback = static_cast<uint32_t*>(ws);
    float2* ms = reinterpret_cast<float2*>(static_cast<char*>(ws) + kTopkCounterBytes);
    uint64_t* keys = reinterpret_cast<uint64_t*>(
        (reinterpret_cast<uintptr_t>(ms + rows * chunks) + 15) & ~uintptr_t(15));
    float* hs = reinterpret_cast<float*>(
        (reinterpret_cast<uintptr_t>(keys + rows * chunks * k) + 15) & ~uintptr_t(15));
    const bool ent = entropy != nullptr;
    const int64_t waves = rows * chunks;
    const dim3 block(kTopkWavesPerBlock * kWave);
    const dim3 grid((unsigned)((waves + kTopkWavesPerBlock - 1) / kTopkWavesPerBlock));
#define PRESTO_TOPK(BF, NL, EN)                                                              \
    topk_partial_kernel<BF, NL, EN><<<grid, block, 0, stream>>>(logits, rows, vocab, row_stride, \
                                                               k, (int32_t)chunks, aligned,      \
                                                               row_index, logits_rows, ms, keys, \
                                                               hs, n_fallback, flags)
#define PRESTO_TOPK2(BF, NL) \
    if (ent) PRESTO_TOPK(BF, NL, true); else PRESTO_TOPK(BF, NL, false)
    if (bf16) {
        if (nload == 8) { PRESTO_TOPK2(true, 8); } else { PRESTO_TOPK2(true, 4); }
    } else {
        if (nload == 8) { PRESTO_TOPK2(false, 8); } else { PRESTO_TOPK2(false, 4); }
    }
#undef PRESTO_TOPK2
#undef PRESTO_TOPK
    presto_status st = check_launch("topk_partial_kernel");
    if (st != PRESTO_OK) return st;
    const dim3 mgrid((unsigned)((rows + kTopkWavesPerBlock - 1) / kTopkWavesPerBlock));
    const int64_t per_lane = (chunks * k + kWave - 1) / kWave;
#define PRESTO_MERGE(KP, EN)                                                                    \
    topk_merge_kernel<KP, EN><<<mgrid, block, 0, stream>>>(rows, (int32_t)chunks, k, ms, keys, hs, \
                                                           ids, logprob, lse, entropy, n_fallback)
#define PRESTO_MERGE2(KP) \
    if (ent) PRESTO_MERGE(KP, true); else PRESTO_MERGE(KP, false)
    if (per_lane <= 2) { PRESTO_MERGE2(2); }
    else if (per_lane <= 4) { PRESTO_MERGE2(4); }
    else if (per_lane <= 8) { PRESTO_MERGE2(8); }
    else if (per_lane <= 16) { PRESTO_MERGE2(16); }
    else { PRESTO_MERGE2(0); }
#undef PRESTO_MERGE2
#undef PRESTO_MERGE
    return check_launch("topk_merge_kernel");
}

// ---------------------------------------------------------------------------
// Top-k without a caller workspace, for callers that cannot allocate (code
// under graph capture, serving loops that forbid allocation).  The partials
// live in one static device array per GPU; every call on a GPU shares it, so
// calls that overlap on one GPU race.  Nothing in it needs to start at zero
// (the fallback counter is cleared by the partial kernel of each call).

constexpr size_t kTopkScratchBytes = PRESTO_TOPK_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kTopkScratchBytes];

static std::mutex g_scratch_mu;
static void* g_scratch_ptr[kMaxDevices];  // this device's address of `scratch`

presto_status launch_topk_noalloc(bool bf16, const void* logits, int64_t rows, int32_t vocab,
                                  int64_t row_stride, int32_t k, int32_t* ids, float* logprob,
                                  float* lse, float* entropy, int32_t* flags, hipStream_t stream) {
    const size_t need = topk_workspace_bytes(rows, vocab, k);
    if (need > kTopkScratchBytes)
        return set_error(PRESTO_ERR_WORKSPACE,
                         "presto_topk_noalloc: %zu bytes of scratch needed, the static scratch "
                         "holds %zu (fewer rows per call)",
                         need, kTopkScratchBytes);
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return set_error(PRESTO_ERR_HIP, "presto_topk_noalloc: hipGetDevice: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxDevices)
        return set_error(PRESTO_ERR_UNSUPPORTED, "presto_topk_noalloc: device %d", dev);
    void* ptr;
    {
        std::lock_guard<std::mutex> lock(g_scratch_mu);
        if (g_scratch_ptr[dev] == nullptr) {
            // the array's name is a host-side stand-in: its device address
            // (one per GPU) comes from the runtime, with this device current
            void* p = nullptr;
            e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
            if (e != hipSuccess || p == nullptr)
                return set_error(PRESTO_ERR_HIP, "presto_topk_noalloc: hipGetSymbolAddress: %s",
                                 hipGetErrorString(e));
            g_scratch_ptr[dev] = p;
        }
        ptr = g_scratch_ptr[dev];
    }
    return launch_topk(bf16, logits, nullptr, rows, rows, vocab, row_stride, k, ids, logprob, lse,
                       entropy, flags, ptr, stream);
}

presto_status launch_entropy_lambda(int64_t rows, const float* entropy, float beta, float c,
                                    float* lambda, hipStream_t stream) {
    entropy_lambda_kernel<<<(unsigned)((rows + 255) / 256), 256, 0, stream>>>(rows, entropy, beta, c,
                                                                              lambda);
    return check_launch("entropy_lambda_kernel");
}

}  // namespace presto_host
