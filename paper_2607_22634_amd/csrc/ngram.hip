// Trigram table for the prefix-aligned signal rho (Sec. 5.1 instantiates rho
// with an n-gram model, n = 3) and the gather that turns it into the lattice
// log_rho[b, d, r2, r1, r] read by the tree builder (Eq. 9).
//
// Table: open addressing with linear probing in caller memory of
// `capacity` slots (a power of two): keys[capacity] uint64, then
// vals[capacity] uint32.  A key packs (t2, t1, t) in 21 bits each; the empty
// key is all ones, which no packed key reaches (bit 63 stays clear).  A value
// is ord32(log rho): monotone as an unsigned integer, so duplicate keys keep
// the largest log rho through one atomicMax, whatever the insertion order.
// The home slot is the splitmix64 output mix (Steele, Lea and Flood, 2014) of
// the key.
//
// The gather runs one lane per lattice entry: a handful of dependent 8-byte
// probes per entry, all entries in flight at once, so the sequential tree
// search never waits on a table lookup.
#include "common.hpp"

namespace presto {

constexpr uint64_t kNgramEmpty = ~0ull;
constexpr uint32_t kNgramTokenLimit = 1u << 21;

__device__ __forceinline__ uint64_t ngram_key(uint32_t t2, uint32_t t1, uint32_t t) {
    return ((uint64_t)t2 << 42) | ((uint64_t)t1 << 21) | (uint64_t)t;
}

__device__ __forceinline__ uint64_t ngram_mix(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    return z ^ (z >> 31);
}

__device__ __forceinline__ bool ngram_token_ok(int32_t t) {
    return t >= 0 && (uint32_t)t < kNgramTokenLimit;
}

__global__ void ngram_clear_kernel(uint64_t* __restrict__ keys, uint32_t* __restrict__ vals,
                                   int64_t capacity) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < capacity;
         i += (int64_t)gridDim.x * blockDim.x) {
        keys[i] = kNgramEmpty;
        vals[i] = 0u;
    }
}

// One lane per entry.  A bad entry (token outside [0, 2^21), log rho not a
// finite value <= 0) is skipped with PRESTO_FLAG_NGRAM_BAD; an entry that
// finds no free slot after a full cycle raises PRESTO_FLAG_NGRAM_FULL.
__global__ void ngram_insert_kernel(uint64_t* __restrict__ keys, uint32_t* __restrict__ vals,
                                    int64_t capacity, int64_t n, const int32_t* __restrict__ t2,
                                    const int32_t* __restrict__ t1, const int32_t* __restrict__ t,
                                    const float* __restrict__ log_rho, int32_t* __restrict__ flags) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const int32_t a = t2[i], b = t1[i], c = t[i];
    const float v = log_rho[i];
    if (!ngram_token_ok(a) || !ngram_token_ok(b) || !ngram_token_ok(c) || !(v <= 0.f) ||
        v == -INFINITY) {
        if (flags) atomicOr(flags, PRESTO_FLAG_NGRAM_BAD);
        return;
    }
    const uint64_t key = ngram_key((uint32_t)a, (uint32_t)b, (uint32_t)c);
    const uint64_t mask = (uint64_t)capacity - 1;
    uint64_t h = ngram_mix(key) & mask;
    for (int64_t p = 0; p < capacity; ++p) {
        const unsigned long long prev =
            atomicCAS(reinterpret_cast<unsigned long long*>(keys + h), kNgramEmpty, key);
        if (prev == kNgramEmpty || prev == key) {
            atomicMax(vals + h, ord32(v));
            return;
        }
        h = (h + 1) & mask;
    }
    if (flags) atomicOr(flags, PRESTO_FLAG_NGRAM_FULL);
}

__device__ __forceinline__ float ngram_lookup(const uint64_t* __restrict__ keys,
                                              const uint32_t* __restrict__ vals, uint64_t mask,
                                              int32_t a, int32_t b, int32_t c, float floor_v) {
    if (!ngram_token_ok(a) || !ngram_token_ok(b) || !ngram_token_ok(c)) return floor_v;
    const uint64_t key = ngram_key((uint32_t)a, (uint32_t)b, (uint32_t)c);
    uint64_t h = ngram_mix(key) & mask;
    for (uint64_t p = 0; p <= mask; ++p) {
        const uint64_t kk = keys[h];
        if (kk == key) return unord32(vals[h]);
        if (kk == kNgramEmpty) break;
        h = (h + 1) & mask;
    }
    return floor_v;
}

// Lattice entry (b, d, r2, r1, r) holds log rho(t | t2, t1) with
//   t  = ids[b, d, r]
//   t1 = ids[b, d-1, r1]                 (d >= 1), the root token (d = 0)
//   t2 = ids[b, d-2, r2]                 (d >= 2), the root token (d = 1),
//        the token before the root       (d = 0)
// and the floor when the trigram is absent.  Slots that a depth never reads
// (r1, r2 at d = 0, r2 at d = 1) repeat the value of slot 0.
__global__ void ngram_gather_kernel(const uint64_t* __restrict__ keys,
                                    const uint32_t* __restrict__ vals, uint64_t mask,
                                    float floor_v, int32_t batch, int32_t D, int32_t k,
                                    const int32_t* __restrict__ ids,
                                    const int32_t* __restrict__ prev_token,
                                    const int32_t* __restrict__ root_token,
                                    float* __restrict__ log_rho) {
    const int64_t k3 = (int64_t)k * k * k;
    const int64_t total = (int64_t)batch * D * k3;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int r = (int)(i % k);
        const int r1 = (int)((i / k) % k);
        const int r2 = (int)((i / ((int64_t)k * k)) % k);
        const int64_t bd = i / k3;  // b * D + d
        const int d = (int)(bd % D);
        const int64_t b = bd / D;
        const int32_t* row = ids + bd * k;
        const int32_t root = root_token[b];
        const int32_t tok = row[r];
        const int32_t t1 = d >= 1 ? row[r1 - k] : root;
        const int32_t t2 = d >= 2 ? row[r2 - 2 * k] : (d == 1 ? root : prev_token[b]);
        log_rho[i] = ngram_lookup(keys, vals, mask, t2, t1, tok, floor_v);
    }
}

}  // namespace presto

namespace presto_host {

using namespace presto;

static unsigned ngram_grid(int64_t work) {
    const int64_t blocks = (work + 255) / 256;
    return (unsigned)(blocks < 8192 ? (blocks > 0 ? blocks : 1) : 8192);
}

static uint32_t* ngram_vals(void* table, int64_t capacity) {
    return reinterpret_cast<uint32_t*>(static_cast<uint64_t*>(table) + capacity);
}

presto_status launch_ngram_clear(void* table, int64_t capacity, hipStream_t stream) {
    ngram_clear_kernel<<<ngram_grid(capacity), 256, 0, stream>>>(
        static_cast<uint64_t*>(table), ngram_vals(table, capacity), capacity);
    return check_launch("ngram_clear_kernel");
}

presto_status launch_ngram_insert(void* table, int64_t capacity, int64_t n, const int32_t* t2,
                                  const int32_t* t1, const int32_t* t, const float* log_rho,
                                  int32_t* flags, hipStream_t stream) {
    ngram_insert_kernel<<<(unsigned)((n + 255) / 256), 256, 0, stream>>>(
        static_cast<uint64_t*>(table), ngram_vals(table, capacity), capacity, n, t2, t1, t,
        log_rho, flags);
    return check_launch("ngram_insert_kernel");
}

presto_status launch_ngram_gather(const void* table, int64_t capacity, float floor_v,
                                  int32_t batch, int32_t D, int32_t k, const int32_t* ids,
                                  const int32_t* prev_token, const int32_t* root_token,
                                  float* log_rho, hipStream_t stream) {
    const uint64_t* keys = static_cast<const uint64_t*>(table);
    const uint32_t* vals = reinterpret_cast<const uint32_t*>(keys + capacity);
    const int64_t total = (int64_t)batch * D * k * k * k;
    ngram_gather_kernel<<<ngram_grid(total), 256, 0, stream>>>(
        keys, vals, (uint64_t)capacity - 1, floor_v, batch, D, k, ids, prev_token, root_token,
        log_rho);
    return check_launch("ngram_gather_kernel");
}

}  // namespace presto_host
