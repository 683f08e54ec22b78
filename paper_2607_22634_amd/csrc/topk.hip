// Stage 1: log-softmax normaliser and top-k candidates per drafter position.
//
// The vocabulary row of each position is streamed from HBM once.  A row is
// cut into wave-sized chunks; every wave holds its chunk in registers and
// produces, with no block-level synchronisation:
//   * the chunk maximum m and sum exp(z - m)           (for the row's LSE)
//   * the chunk's k best (value desc, id asc) entries  (as 64-bit keys)
// The k-th largest lane maximum (k rounds of wave max, or a ballot bisection
// on its orderable bits for k > 8) is a lower bound on the chunk's k-th value, so only the
// 16-byte groups whose maximum reaches it can hold a top-k entry (normally a
// handful); their entries at or above it are compacted through a small
// per-wave LDS list and the k best taken by k rounds of wave max.  A chunk
// with more candidate groups than the list holds (massive ties) falls back
// to k rounds of exact wave-wide selection over the chunk re-read from
// memory.  A second kernel, queued right behind,
// merges each row's chunk partials with one wave per row.
#include <math.h>

#include "common.hpp"

namespace presto {

constexpr int kCandCap = 64;
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
// bits, counting lanes at or above each probe with a ballot.
__device__ __forceinline__ uint32_t wave_kth_largest_u32(uint32_t x, int k) {
    if (k <= 8) {
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
    for (int bit = 31; bit >= 0; --bit) {
        const uint32_t c = t | (1u << bit);
        if (__popcll(__ballot(x >= c)) >= k) t = c;
    }
    return t;
}

template <bool BF16, int NLOAD>
__global__ __launch_bounds__(kTopkWavesPerBlock * kWave) void topk_partial_kernel(
    const void* __restrict__ logits, int64_t rows, int32_t vocab, int64_t row_stride, int32_t k,
    int32_t chunks, bool aligned, float2* __restrict__ part_ms, uint64_t* __restrict__ part_keys,
    int32_t* __restrict__ flags) {
    constexpr int P = VecTraits<BF16>::kPerVec;  // elements per 16-byte load (a "group")
    constexpr int E = NLOAD * P;
    constexpr int64_t CH = (int64_t)kWave * E;
    constexpr int kGroupCap = kCandCap / P;      // candidate groups a wave list holds
    __shared__ uint64_t cand[kTopkWavesPerBlock][kCandCap];
    __shared__ uint32_t cand_n[kTopkWavesPerBlock];

    const int wave = threadIdx.x / kWave, lane = lane_id();
    const int64_t gw = (int64_t)blockIdx.x * kTopkWavesPerBlock + wave;
    if (gw >= rows * chunks) return;
    const int64_t row = gw / chunks;
    const int32_t chunk = (int32_t)(gw % chunks);
    const int64_t c0 = (int64_t)chunk * CH;
    const char* rowp = static_cast<const char*>(logits) + row * row_stride * (BF16 ? 2 : 4);
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
    // For moderate M: exp(z - M) = exp2(fma(z, log2 e, -mo)) * 2^r with
    // mo = fl(M log2 e) and r = M log2 e - mo taken exactly by one fma (|r| is
    // below 2^-16 here), so one fma and one exp per entry.  Larger |M| takes
    // the plain form exp2((z - M) log2 e).
    float s = 0.f;
    float corr = 1.f;
    if (fabsf(M) < 256.f) {
        const float mo = M * kLog2eF;
        corr = __builtin_amdgcn_exp2f(fmaf(M, kLog2eF, -mo));
#pragma unroll
        for (int e = 0; e < E; ++e) s += __builtin_amdgcn_exp2f(fmaf(v[e], kLog2eF, -mo));
    } else if (M != -INFINITY) {
#pragma unroll
        for (int e = 0; e < E; ++e) s += __builtin_amdgcn_exp2f((v[e] - M) * kLog2eF);
    }
    const float S = wave_sum_f32_dpp(s) * corr;
    // the k-th largest lane maximum bounds the chunk's k-th value from below:
    // only groups whose maximum reaches it can hold a top-k entry
    const float thr = unord32(wave_kth_largest_u32(ord32(lm), k));

    if (lane == 0) cand_n[wave] = 0u;
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int i = 0; i < NLOAD; ++i) {
        if (gmax[i] >= thr) {
            const uint32_t slot = atomicAdd(&cand_n[wave], 1u);
            if (slot < (uint32_t)kGroupCap) {
#pragma unroll
                for (int j = 0; j < P; ++j) {
                    const int64_t idx = c0 + (int64_t)(i * kWave + lane) * P + j;
                    const bool ok = (full || idx < vocab) && v[i * P + j] >= thr;
                    cand[wave][slot * P + j] = ok ? vocab_key(v[i * P + j], (uint32_t)idx) : 0ull;
                }
            }
        }
    }
    __builtin_amdgcn_wave_barrier();
    const uint32_t ngroups = __builtin_amdgcn_readfirstlane(cand_n[wave]);
    uint64_t* out = part_keys + gw * k;

    if (ngroups <= (uint32_t)kGroupCap) {
        // one candidate key per lane (keys are unique); k rounds of wave max,
        // retiring the lane that held it (0 past the last valid entry)
        const int total = (int)ngroups * P;
        uint64_t x = lane < total ? cand[wave][lane] : 0ull;
        uint64_t mine = 0ull;
        for (int j = 0; j < k; ++j) {
            const uint64_t m = wave_max_u64_dpp(x);
            mine = lane == j ? m : mine;
            x = x == m ? 0ull : x;
        }
        if (lane < k) out[lane] = mine;
    } else {
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
        part_ms[gw] = make_float2(M, S);
        if (!(S == S)) raise_flag(flags, PRESTO_FLAG_NAN_DRAFTER);
    }
}

// One wave per row: LSE from the chunk (max, sum) pairs, then the k best of
// the chunk keys by k rounds of wave-wide selection over keys held in
// registers (KPL per lane; KPL == 0 re-reads them from memory).
template <int KPL>
__global__ __launch_bounds__(kTopkWavesPerBlock * kWave) void topk_merge_kernel(
    int64_t rows, int32_t chunks, int32_t k, const float2* __restrict__ part_ms,
    const uint64_t* __restrict__ part_keys, int32_t* __restrict__ ids, float* __restrict__ logprob,
    float* __restrict__ lse) {
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
    float m = -INFINITY;
    for (int c = lane; c < chunks; c += kWave) m = fmaxf(m, ms[c].x);
    const float M = wave_max_f32_dpp(m);
    float s = 0.f;
    if (M != -INFINITY)
        for (int c = lane; c < chunks; c += kWave) {
            const float2 p = ms[c];
            s += p.x == -INFINITY ? 0.f : p.y * __expf(p.x - M);
        }
    const float S = wave_sum_f32_dpp(s);
    const float L = (M == -INFINITY) ? -INFINITY : M + __logf(S);

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
        logprob[row * k + lane] = (L == -INFINITY) ? -INFINITY : key_value(mine) - L;
    }
    if (lse && lane == 0) lse[row] = L;
}

}  // namespace presto

namespace presto_host {

using namespace presto;

static int topk_nload(bool bf16, int64_t rows, int32_t vocab) {
    const int64_t ch8 = (int64_t)kWave * 8 * (bf16 ? 8 : 4);
    const int64_t waves8 = rows * ((vocab + ch8 - 1) / ch8);
    // 8 loads per lane only when that still leaves >= 16 waves per CU
    return waves8 >= 16 * 256 ? 8 : 4;
}

size_t topk_workspace_bytes(int64_t rows, int32_t vocab, int32_t k) {
    // sized for the finest chunking any dtype may pick
    const int64_t chunks = (vocab + (int64_t)kWave * 16 - 1) / ((int64_t)kWave * 16);
    const size_t per = (size_t)chunks * (sizeof(float2) + sizeof(uint64_t) * (size_t)k);
    return (size_t)rows * per + 256;
}

presto_status launch_topk(bool bf16, const void* logits, int64_t rows, int32_t vocab,
                          int64_t row_stride, int32_t k, int32_t* ids, float* logprob, float* lse,
                          int32_t* flags, void* ws, hipStream_t stream) {
    const int nload = topk_nload(bf16, rows, vocab);
    const int64_t ch = (int64_t)kWave * nload * (bf16 ? 8 : 4);
    const int64_t chunks = (vocab + ch - 1) / ch;
    const size_t esz = bf16 ? 2 : 4;
    const bool aligned = ((uintptr_t)logits % 16 == 0) && ((row_stride * (int64_t)esz) % 16 == 0);
    float2* ms = static_cast<float2*>(ws);
    uint64_t* keys = reinterpret_cast<uint64_t*>(
        (reinterpret_cast<uintptr_t>(ms + rows * chunks) + 15) & ~uintptr_t(15));
    const int64_t waves = rows * chunks;
    const dim3 block(kTopkWavesPerBlock * kWave);
    const dim3 grid((unsigned)((waves + kTopkWavesPerBlock - 1) / kTopkWavesPerBlock));
#define PRESTO_TOPK(BF, NL)                                                                 \
    topk_partial_kernel<BF, NL><<<grid, block, 0, stream>>>(logits, rows, vocab, row_stride, \
                                                           k, (int32_t)chunks, aligned, ms,  \
                                                           keys, flags)
    if (bf16) {
        if (nload == 8) PRESTO_TOPK(true, 8); else PRESTO_TOPK(true, 4);
    } else {
        if (nload == 8) PRESTO_TOPK(false, 8); else PRESTO_TOPK(false, 4);
    }
#undef PRESTO_TOPK
    presto_status st = check_launch("topk_partial_kernel");
    if (st != PRESTO_OK) return st;
    const dim3 mgrid((unsigned)((rows + kTopkWavesPerBlock - 1) / kTopkWavesPerBlock));
    const int64_t per_lane = (chunks * k + kWave - 1) / kWave;
#define PRESTO_MERGE(KP)                                                                     \
    topk_merge_kernel<KP><<<mgrid, block, 0, stream>>>(rows, (int32_t)chunks, k, ms, keys, \
                                                       ids, logprob, lse)
    if (per_lane <= 2) PRESTO_MERGE(2);
    else if (per_lane <= 4) PRESTO_MERGE(4);
    else if (per_lane <= 8) PRESTO_MERGE(8);
    else if (per_lane <= 16) PRESTO_MERGE(16);
    else PRESTO_MERGE(0);
#undef PRESTO_MERGE
    return check_launch("topk_merge_kernel");
}

}  // namespace presto_host
