/* Sanitizer driver for the CPU oracle: built together with oracle.c under
 * AddressSanitizer and UndefinedBehaviorSanitizer (no recovery), it calls
 * every oracle entry point on small seeded inputs, edge rows included
 * (ties, -inf rows, NaN, empty contexts, budgets beyond the candidate
 * tree), and checks a few invariants.  Exit status 0 means no report. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "oracle.h"

static uint64_t rng_state = 0x9e3779b97f4a7c15ull;
static uint64_t next_u64(void) { /* splitmix64 */
    uint64_t z = (rng_state += 0x9e3779b97f4a7c15ull);
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    return z ^ (z >> 31);
}
static float uniform(void) { return (float)((next_u64() >> 11) * (1.0 / 9007199254740992.0)); }
static float normal(void) {
    float u = uniform() + 1e-7f, v = uniform();
    return sqrtf(-2.f * logf(u)) * cosf(6.2831853f * v);
}
static uint16_t to_bf16(float f) {
    uint32_t u;
    memcpy(&u, &f, 4);
    return (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

#define CHECK(c)                                                   \
    do {                                                           \
        if (!(c)) {                                                \
            fprintf(stderr, "check failed: %s (line %d)\n", #c, __LINE__); \
            return 1;                                              \
        }                                                          \
    } while (0)

static int topk_and_entropy(void) {
    const int rows = 6, V = 517, k = 5;
    float *x = malloc(sizeof(float) * rows * V);
    uint16_t *xb = malloc(sizeof(uint16_t) * rows * V);
    for (int i = 0; i < rows * V; ++i) x[i] = 3.f * normal();
    for (int v = 0; v < V; ++v) {
        x[1 * V + v] = 1.5f;      /* one tie */
        x[2 * V + v] = -INFINITY; /* a fully masked row */
    }
    x[3 * V + 7] = NAN;
    for (int i = 0; i < rows * V; ++i) xb[i] = to_bf16(x[i]);
    int32_t ids[6 * 5];
    float lp[6 * 5], lse[6];
    double h[6];
    CHECK(oracle_topk(ORACLE_F32, x, rows, V, V, k, ids, lp, lse) == 1);
    CHECK(ids[1 * k] == 0 && ids[1 * k + 4] == 4); /* ties: lowest ids first */
    CHECK(oracle_topk(ORACLE_BF16, xb, rows, V, V, k, ids, lp, lse) == 1);
    oracle_entropy(ORACLE_F32, x, rows, V, V, h);
    CHECK(h[2] == 0.0 && fabs(h[1] - log((double)V)) < 1e-9);
    double lam[6];
    oracle_entropy_lambda(rows, h, 0.5, 2.0, lam);
    free(x);
    free(xb);
    return 0;
}

static int trees(void) {
    const int b = 3, D = 5, k = 3;
    int32_t ids[3 * 5 * 3], root[3] = {7, 8, 9};
    float lp[3 * 5 * 3], rho[3 * 5 * 27], lam[5] = {0.2f, 0.2f, 0.2f, 0.2f, 0.2f};
    for (int i = 0; i < b * D * k; ++i) {
        ids[i] = 100 + i;
        lp[i] = -(float)(next_u64() % 8) * 0.25f; /* quantised: ties in S */
    }
    for (int i = 0; i < b * D * k * k * k; ++i) rho[i] = uniform() < 0.5f ? logf(1e-4f) : logf(uniform() + 1e-3f);
    const int budgets[3] = {1, 17, 400}; /* 400 > the 363-node candidate tree */
    for (int bi = 0; bi < 3; ++bi) {
        const int B = budgets[bi], N = B + 1, W = (N + 63) / 64;
        int32_t *nn = malloc(sizeof(int32_t) * b), *par = malloc(sizeof(int32_t) * b * N),
                *tok = malloc(sizeof(int32_t) * b * N), *dep = malloc(sizeof(int32_t) * b * N),
                *rk = malloc(sizeof(int32_t) * b * N);
        float *sc = malloc(sizeof(float) * b * N);
        uint64_t *anc = malloc(sizeof(uint64_t) * b * N * W);
        for (int mode = 0; mode < 3; ++mode)
            for (int with_rho = 0; with_rho < 2; ++with_rho) {
                CHECK(oracle_build_tree(mode, b, D, k, k - (mode == 1), B, 2, ids, lp,
                                        with_rho ? rho : NULL, lam, 0, root, nn, par, tok, dep, rk,
                                        sc, anc) == 0);
                for (int s = 0; s < b; ++s) {
                    CHECK(nn[s] >= 1 && nn[s] <= N);
                    for (int n = 1; n < nn[s]; ++n) CHECK(par[s * N + n] >= 0 && par[s * N + n] < n);
                }
            }
        free(nn); free(par); free(tok); free(dep); free(rk); free(sc); free(anc);
    }
    return 0;
}

static int attention_and_accept(void) {
    const int b = 3, N = 9, hq = 4, hkv = 2, d = 64, W = 1;
    const int32_t offs[4] = {0, 0, 1, 70}; /* empty, one key, 69 keys */
    const int total = 70;
    float *q = malloc(sizeof(float) * b * N * hq * d), *kc = malloc(sizeof(float) * total * hkv * d),
          *vc = malloc(sizeof(float) * total * hkv * d), *kt = malloc(sizeof(float) * b * N * hkv * d),
          *vt = malloc(sizeof(float) * b * N * hkv * d), *out = malloc(sizeof(float) * b * N * hq * d);
    for (int i = 0; i < b * N * hq * d; ++i) q[i] = normal();
    for (int i = 0; i < total * hkv * d; ++i) { kc[i] = normal(); vc[i] = normal(); }
    for (int i = 0; i < b * N * hkv * d; ++i) { kt[i] = normal(); vt[i] = normal(); }
    int32_t nn[3] = {1, 9, 5}, par[27], tok[27];
    uint64_t anc[27];
    for (int s = 0; s < b; ++s)
        for (int n = 0; n < N; ++n) {
            par[s * N + n] = n == 0 ? -1 : (n - 1) / 2;
            tok[s * N + n] = n < nn[s] ? 10 + n : -1;
            uint64_t m = 0;
            for (int x = n; x >= 0 && n < nn[s]; x = x == 0 ? -1 : (x - 1) / 2) m |= 1ull << x;
            anc[s * N + n] = m;
        }
    oracle_tree_attention(ORACLE_F32, b, N, hq, hkv, d, 0.125, q, kc, vc, offs, kt, vt, anc, nn, out);
    const int32_t rows[6] = {1, 8, 3, 2, 4, 0};
    double ro[2 * 64];
    oracle_tree_attention_rows(ORACLE_F32, b, N, hq, hkv, d, 0.125, q, kc, vc, offs, kt, vt, anc,
                               nn, 2, rows, ro);
    for (int e = 0; e < d; ++e) CHECK(fabs(ro[e] - out[((1 * N + 8) * hq + 3) * d + e]) < 1e-5);
    (void)W;
    const int V = 33;
    float *T = malloc(sizeof(float) * b * N * V);
    for (int i = 0; i < b * N * V; ++i) T[i] = normal();
    T[(1 * N + 0) * V + 11] = 50.f; /* the root of sequence 1 predicts node 1's token */
    int32_t al[3], path[3 * 6], bonus[3], am[27];
    CHECK(oracle_accept(ORACLE_F32, T, V, V, b, N, 5, par, tok, nn, al, path, bonus, am) == 0);
    CHECK(al[1] >= 1 && path[1 * 6 + 1] == 1);
    free(q); free(kc); free(vc); free(kt); free(vt); free(out); free(T);
    return 0;
}

int main(void) {
    oracle_set_threads(2);
    if (topk_and_entropy()) return 1;
    if (trees()) return 1;
    if (attention_and_accept()) return 1;
    printf("oracle driver: ok\n");
    return 0;
}
