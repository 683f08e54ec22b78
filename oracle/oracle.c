/*
 * CPU oracle for the PRESTO draft-to-verify round -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, obviously correct statement of what the four stages of a
 * round compute, following "PRESTO: Prefix-Aligned Tree Drafting for
 * Diffusion Speculative Decoding":
 *
 *   1. per-position log-softmax and top-k candidates  (Sec. 4.1, Eq. 7;
 *      Sec. 4.3 / Appendix C stage II "top-k diffusion candidates")
 *   2. prefix-aligned token score and path score      (Sec. 4.1, Eq. 9)
 *      and best-first tree construction under budget B (Sec. 4.2, Alg. 2;
 *      the closed form "top-B prefixes by S" of Sec. 4.2 with Eq. 3)
 *   3. tree-masked verification attention             (Appendix C stage I:
 *      each draft token attends to the committed prefix and its ancestors)
 *   4. greedy longest-accepted-path walk + bonus       (Eq. 1; Appendix C
 *      stage I)
 *
 * Floating point: log-sum-exp, softmax and attention in fp64 over inputs
 * upcast exactly; the tree score in fp32 with the paper's two-term sum
 * evaluated as fl(log q + fl(lambda * log rho)) and S(child) =
 * fl(S(parent) + s), no contraction (built with -ffp-contract=off).
 *
 * Only the test suite, the smoke check and the bench's CPU-baseline leg may
 * load this library.  It shares no code with the HIP library.
 */
#define _GNU_SOURCE
#include "oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

void oracle_set_threads(int n) {
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

int oracle_get_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ------------------------------------------------------------------------ */
/* element access                                                           */

static float bf16_to_float(uint16_t b) {
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

static uint16_t float_to_bf16(float f) {
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40); /* quiet NaN */
    u += 0x7fffu + ((u >> 16) & 1u);                                         /* round to nearest even */
    return (uint16_t)(u >> 16);
}

static float load_f(int dtype, const void *base, int64_t i) {
    if (dtype == ORACLE_BF16) return bf16_to_float(((const uint16_t *)base)[i]);
    return ((const float *)base)[i];
}

static void store_f(int dtype, void *base, int64_t i, double v) {
    float f = (float)v;
    if (dtype == ORACLE_BF16)
        ((uint16_t *)base)[i] = float_to_bf16(f);
    else
        ((float *)base)[i] = f;
}

/* "a ranks before b" for vocabulary entries: larger value first, lower id on
 * equal values (-0.0 and +0.0 compare equal). */
static int vocab_before(float av, int32_t ai, float bv, int32_t bi) {
    if (av > bv) return 1;
    if (av < bv) return 0;
    return av == bv && ai < bi;
}

/* ------------------------------------------------------------------------ */
/* 1. log-softmax + top-k                                                   */

int oracle_topk(int dtype, const void *logits, int64_t rows, int32_t vocab, int64_t row_stride,
                int32_t k, int32_t *ids, float *logprob, float *lse) {
    int nan_rows = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(+ : nan_rows)
    for (int64_t r = 0; r < rows; ++r) {
        const int64_t base = r * row_stride;
        float *bv = (float *)malloc(sizeof(float) * (size_t)k);
        int32_t *bi = (int32_t *)malloc(sizeof(int32_t) * (size_t)k);
        int have = 0, saw_nan = 0;
        double m = -INFINITY;
        for (int32_t v = 0; v < vocab; ++v) {
            float z = load_f(dtype, logits, base + v);
            if (isnan(z)) saw_nan = 1;
            if ((double)z > m) m = (double)z;
            /* insertion into the sorted list of the best k seen so far */
            if (have < k || vocab_before(z, v, bv[have - 1], bi[have - 1])) {
                int pos = have < k ? have : k - 1;
                while (pos > 0 && vocab_before(z, v, bv[pos - 1], bi[pos - 1])) {
                    bv[pos] = bv[pos - 1];
                    bi[pos] = bi[pos - 1];
                    --pos;
                }
                bv[pos] = z;
                bi[pos] = v;
                if (have < k) ++have;
            }
        }
        /* log sum_v exp(z_v) = m + log sum_v exp(z_v - m), in fp64; log q(t) =
         * z_t - LSE is formed as (z_t - m) - log sum, which keeps the log of
         * the sum even where |m| dwarfs it (a row near -1e30) */
        double l, ls = 0.0;
        if (m == -INFINITY) {
            l = -INFINITY;
        } else {
            double acc = 0.0;
            for (int32_t v = 0; v < vocab; ++v) acc += exp((double)load_f(dtype, logits, base + v) - m);
            ls = log(acc);
            l = m + ls;
        }
        for (int j = 0; j < k; ++j) {
            ids[r * k + j] = bi[j];
            logprob[r * k + j] = (l == -INFINITY) ? -INFINITY : (float)(((double)bv[j] - m) - ls);
        }
        if (lse) lse[r] = (float)l;
        nan_rows += saw_nan;
        free(bv);
        free(bi);
    }
    return nan_rows;
}

/* Entropy of the diffusion marginal, H_d = -sum_w q_d(w) log q_d(w)
 * (Appendix F), with q_d = softmax(z_d) (Eq. 6) formed in fp64 from the
 * row max m and log sum_w exp(z_w - m).  A term whose q is 0 contributes 0 (its limit); a row of
 * only -inf has no distribution and is given H = 0. */
void oracle_entropy(int dtype, const void *logits, int64_t rows, int32_t vocab, int64_t row_stride,
                    double *entropy) {
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t r = 0; r < rows; ++r) {
        const int64_t base = r * row_stride;
        double m = -INFINITY;
        for (int32_t v = 0; v < vocab; ++v) {
            double z = (double)load_f(dtype, logits, base + v);
            if (z > m) m = z;
        }
        if (m == -INFINITY) {
            entropy[r] = 0.0;
            continue;
        }
        double acc = 0.0;
        for (int32_t v = 0; v < vocab; ++v) acc += exp((double)load_f(dtype, logits, base + v) - m);
        const double ls = log(acc);
        double h = 0.0;
        for (int32_t v = 0; v < vocab; ++v) {
            /* log q = (z - m) - log sum, shifted so that |m| >> log sum keeps it */
            const double q = exp(((double)load_f(dtype, logits, base + v) - m) - ls);
            if (q > 0.0) h -= q * log(q);
        }
        entropy[r] = h;
    }
}

/* Entropy-adaptive weight lambda_d(H_d) = beta * H_d / (H_d + C) (Appendix F), fp64. */
void oracle_entropy_lambda(int64_t rows, const double *entropy, double beta, double c,
                           double *lambda) {
    for (int64_t r = 0; r < rows; ++r) lambda[r] = beta * entropy[r] / (entropy[r] + c);
}

/* ------------------------------------------------------------------------ */
/* 2. prefix-aligned score + best-first tree                                */

#define MAXD 128

typedef struct {
    float S;          /* path score S(u) (Eq. 9)               */
    int32_t parent;   /* index of the parent (committed or T)  */
    int32_t rank;     /* candidate rank of the last token      */
    int32_t depth;    /* |u|                                   */
    int32_t token;
    uint8_t path[MAXD]; /* rank path u, one rank per depth     */
} onode;

/* The total order used for "best" and "top-B": larger S first; on equal S the
 * rank path compared lexicographically, a proper prefix before its
 * extensions.  Since every token score is <= 0, S never increases along a
 * path, so an ancestor always precedes its descendants. */
static int node_before(const onode *a, const onode *b) {
    if (a->S > b->S) return 1;
    if (a->S < b->S) return 0;
    int n = a->depth < b->depth ? a->depth : b->depth;
    for (int i = 0; i < n; ++i)
        if (a->path[i] != b->path[i]) return a->path[i] < b->path[i];
    return a->depth < b->depth;
}

typedef struct {
    int32_t D, k, branch;
    const int32_t *ids;    /* [D, k] */
    const float *logprob;  /* [D, k] */
    const float *rho;      /* [D, k, k, k] or NULL */
    const float *lambda;   /* [D] */
} seqctx;

/* Token score s_{d,t}(c_d) = log q_d(t) + lambda_d log rho_d(t | c_d) for the k
 * candidates of the child position of v, with rho a trigram over the two
 * preceding tokens (grandparent rank, parent rank; rank slot 0 for tokens
 * outside the block: the root and the committed context). */
static void token_scores(const seqctx *c, const onode *v, const onode *v_parent, float *s) {
    const int row = v->depth; /* child depth v->depth + 1 reads drafter row v->depth */
    const int a = v->depth >= 2 ? v_parent->rank : 0;
    const int b = v->depth >= 1 ? v->rank : 0;
    for (int r = 0; r < c->k; ++r) {
        float lq = c->logprob[row * c->k + r];
        if (c->rho) {
            float lr = c->rho[(((int64_t)row * c->k + a) * c->k + b) * c->k + r];
            float t = c->lambda[row] * lr;
            s[r] = lq + t;
        } else {
            s[r] = lq;
        }
    }
}

/* Expand(v, b, s): the top-`branch` children of v ranked by token score
 * (higher s first, lower rank on ties).  Writes children to out[], returns count. */
static int expand(const seqctx *c, const onode *v, int32_t v_index, const onode *v_parent,
                  onode *out) {
    if (v->depth >= c->D) return 0;
    float s[64];
    int used[64];
    token_scores(c, v, v_parent, s);
    for (int r = 0; r < c->k; ++r) used[r] = 0;
    for (int j = 0; j < c->branch; ++j) {
        int best = -1;
        for (int r = 0; r < c->k; ++r) {
            if (used[r]) continue;
            if (best < 0 || s[r] > s[best]) best = r;
        }
        used[best] = 1;
        onode *ch = &out[j];
        memcpy(ch->path, v->path, (size_t)v->depth);
        ch->path[v->depth] = (uint8_t)best;
        ch->depth = v->depth + 1;
        ch->rank = best;
        ch->parent = v_index;
        ch->token = c->ids[v->depth * c->k + best];
        ch->S = v->S + s[best];
    }
    return c->branch;
}

static int pop_best(onode *front, int *nfront) {
    int best = 0;
    for (int i = 1; i < *nfront; ++i)
        if (node_before(&front[i], &front[best])) best = i;
    return best;
}

static void write_tree(const onode *nodes, int n, int32_t N, int32_t W, int32_t *n_nodes,
                       int32_t *parent, int32_t *token, int32_t *depth_out, int32_t *rank,
                       float *score, uint64_t *anc) {
    *n_nodes = n;
    for (int i = 0; i < N; ++i) {
        if (i < n) {
            parent[i] = nodes[i].parent;
            token[i] = nodes[i].token;
            depth_out[i] = nodes[i].depth;
            rank[i] = nodes[i].depth == 0 ? -1 : nodes[i].rank;
            score[i] = nodes[i].S;
        } else {
            parent[i] = token[i] = depth_out[i] = rank[i] = -1;
            score[i] = -INFINITY;
        }
        for (int w = 0; w < W; ++w) anc[(int64_t)i * W + w] = 0;
    }
    /* ancestor mask: row i has bit j set iff j is i or an ancestor of i */
    for (int i = 0; i < n; ++i)
        for (int j = i; j >= 0; j = nodes[j].parent) anc[(int64_t)i * W + j / 64] |= 1ull << (j % 64);
}

static int build_best_first(const seqctx *c, int32_t budget, int32_t root_token, onode *nodes,
                            onode *front, onode *kids) {
    memset(&nodes[0], 0, sizeof(onode));
    nodes[0].parent = -1;
    nodes[0].rank = 0;
    nodes[0].token = root_token;
    int n = 1, nfront = expand(c, &nodes[0], 0, NULL, front);
    /* commit on pop: the popped node is the best uncommitted prefix */
    while (n - 1 < budget && nfront > 0) {
        int i = pop_best(front, &nfront);
        nodes[n] = front[i];
        front[i] = front[--nfront];
        int nk = expand(c, &nodes[n], n, &nodes[nodes[n].parent], kids);
        for (int j = 0; j < nk; ++j) front[nfront++] = kids[j];
        ++n;
    }
    return n;
}

static int cmp_index_by_order(const void *pa, const void *pb, void *arg) {
    const onode *T = (const onode *)arg;
    int a = *(const int *)pa, b = *(const int *)pb;
    if (node_before(&T[a], &T[b])) return -1;
    if (node_before(&T[b], &T[a])) return 1;
    return 0;
}

/* Literal Alg. 2: pop the best frontier node, add all its children to T and to
 * the frontier, stop once |T| (non-root) reaches B, return TopB(T). */
static int build_alg2(const seqctx *c, int32_t budget, int32_t root_token, onode *nodes,
                      onode *T, int32_t *front_idx, int *order, int32_t *remap) {
    onode root;
    memset(&root, 0, sizeof(root));
    root.parent = -1;
    root.token = root_token;
    /* T entries reference parents as T indices; -1 is the root */
    int nT = 0, nfront = 0;
    int root_open = 1;
    while (nT < budget && (root_open || nfront > 0)) {
        int v_index; /* -1 = root */
        if (root_open) {
            v_index = -1;
            root_open = 0;
        } else {
            int best = 0;
            for (int i = 1; i < nfront; ++i)
                if (node_before(&T[front_idx[i]], &T[front_idx[best]])) best = i;
            v_index = front_idx[best];
            front_idx[best] = front_idx[--nfront];
        }
        const onode *v = v_index < 0 ? &root : &T[v_index];
        const onode *vp = (v_index < 0 || v->parent < 0) ? &root : &T[v->parent];
        int nk = expand(c, v, v_index, vp, &T[nT]);
        for (int j = 0; j < nk; ++j) front_idx[nfront++] = nT + j;
        nT += nk;
    }
    for (int i = 0; i < nT; ++i) order[i] = i;
    qsort_r(order, (size_t)nT, sizeof(int), cmp_index_by_order, T);
    int keep = nT < budget ? nT : budget;
    nodes[0] = root;
    for (int i = 0; i < nT; ++i) remap[i] = -2;
    for (int i = 0; i < keep; ++i) remap[order[i]] = i + 1;
    for (int i = 0; i < keep; ++i) {
        nodes[i + 1] = T[order[i]];
        int p = T[order[i]].parent;
        nodes[i + 1].parent = p < 0 ? 0 : remap[p];
    }
    return keep + 1;
}

/* Alg. 1, beam search with global retention: the beam starts as {root}; at
 * each depth every beam node is expanded (its top-`branch` children join T
 * and the candidate set), and the W best candidates in the total order form
 * the next beam.  Depths are taken while T holds fewer than `budget`
 * non-root nodes (checked before each depth), at most D of them.  The result
 * is TopB(T): the `budget` best nodes of T (with the root), in the total
 * order.  T is prefix-closed, so TopB(T) is too. */
static int build_beam(const seqctx *c, int32_t budget, int32_t W, int32_t root_token,
                      onode *nodes, onode *T, int32_t *beam, int32_t *cand, int *order,
                      int32_t *remap) {
    onode root;
    memset(&root, 0, sizeof(root));
    root.parent = -1;
    root.token = root_token;
    int nT = 0, nbeam = 1;
    beam[0] = -1; /* -1 = the root; T entries reference parents as T indices */
    for (int d = 1; d <= c->D && nT < budget && nbeam > 0; ++d) {
        int ncand = 0;
        for (int i = 0; i < nbeam; ++i) {
            const int v_index = beam[i];
            const onode *v = v_index < 0 ? &root : &T[v_index];
            const onode *vp = (v_index < 0 || v->parent < 0) ? &root : &T[v->parent];
            const int nk = expand(c, v, v_index, vp, &T[nT]);
            for (int j = 0; j < nk; ++j) cand[ncand++] = nT + j;
            nT += nk;
        }
        qsort_r(cand, (size_t)ncand, sizeof(int32_t), cmp_index_by_order, T);
        nbeam = ncand < W ? ncand : W;
        for (int i = 0; i < nbeam; ++i) beam[i] = cand[i];
    }
    for (int i = 0; i < nT; ++i) order[i] = i;
    qsort_r(order, (size_t)nT, sizeof(int), cmp_index_by_order, T);
    const int keep = nT < budget ? nT : budget;
    nodes[0] = root;
    for (int i = 0; i < nT; ++i) remap[i] = -2;
    for (int i = 0; i < keep; ++i) remap[order[i]] = i + 1;
    for (int i = 0; i < keep; ++i) {
        nodes[i + 1] = T[order[i]];
        const int p = T[order[i]].parent;
        nodes[i + 1].parent = p < 0 ? 0 : remap[p];
    }
    return keep + 1;
}

int oracle_build_tree(int mode, int32_t batch, int32_t depth, int32_t k, int32_t branch,
                      int32_t budget, int32_t beam_width, const int32_t *ids, const float *logprob,
                      const float *log_rho, const float *lambda, int32_t lambda_per_seq,
                      const int32_t *root_token,
                      int32_t *n_nodes, int32_t *parent, int32_t *token, int32_t *depth_out,
                      int32_t *rank, float *score, uint64_t *anc) {
    if (depth < 1 || depth > MAXD || k < 1 || k > 64 || branch < 1 || branch > k || budget < 1)
        return -1;
    if (mode != ORACLE_BEST_FIRST && mode != ORACLE_BEST_FIRST_ALG2 && mode != ORACLE_BEAM) return -1;
    if (mode == ORACLE_BEAM && beam_width < 1) return -1;
    const int32_t N = budget + 1, W = (N + 63) / 64;
    /* T capacity: best-first and Alg. 2 add at most `branch` nodes per pop; beam
     * search adds at most W * branch per depth and exceeds the budget by at most
     * one depth's worth */
    int64_t cap = (int64_t)budget * branch + branch + 1;
    if (mode == ORACLE_BEAM) {
        const int64_t beam_cap = (int64_t)budget + (int64_t)beam_width * branch + 1;
        if (beam_cap > cap) cap = beam_cap;
    }
    int err = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : err)
    for (int b = 0; b < batch; ++b) {
        seqctx c = {depth, k, branch, ids + (int64_t)b * depth * k, logprob + (int64_t)b * depth * k,
                    log_rho ? log_rho + (int64_t)b * depth * k * k * k : NULL,
                    lambda_per_seq ? lambda + (int64_t)b * depth : lambda};
        onode *nodes = (onode *)malloc(sizeof(onode) * (size_t)(N + 1));
        onode *pool = (onode *)malloc(sizeof(onode) * (size_t)(cap + branch));
        onode *kids = (onode *)malloc(sizeof(onode) * (size_t)branch);
        int32_t *fidx = (int32_t *)malloc(sizeof(int32_t) * (size_t)(cap + branch));
        int32_t *beam = (int32_t *)malloc(sizeof(int32_t) * (size_t)(beam_width > 0 ? beam_width : 1));
        int *order = (int *)malloc(sizeof(int) * (size_t)(cap + branch));
        int32_t *remap = (int32_t *)malloc(sizeof(int32_t) * (size_t)(cap + branch));
        if (!nodes || !pool || !kids || !fidx || !order || !remap || !beam) {
            err |= 1;
        } else {
            int n;
            if (mode == ORACLE_BEST_FIRST)
                n = build_best_first(&c, budget, root_token[b], nodes, pool, kids);
            else if (mode == ORACLE_BEST_FIRST_ALG2)
                n = build_alg2(&c, budget, root_token[b], nodes, pool, fidx, order, remap);
            else
                n = build_beam(&c, budget, beam_width, root_token[b], nodes, pool, beam, fidx, order,
                               remap);
            write_tree(nodes, n, N, W, &n_nodes[b], parent + (int64_t)b * N, token + (int64_t)b * N,
                       depth_out + (int64_t)b * N, rank + (int64_t)b * N, score + (int64_t)b * N,
                       anc + (int64_t)b * N * W);
        }
        free(nodes);
        free(pool);
        free(kids);
        free(fidx);
        free(beam);
        free(order);
        free(remap);
    }
    return err ? -1 : 0;
}

/* ------------------------------------------------------------------------ */
/* 3. tree-masked attention                                                 */

static void attend_row(int dtype, int32_t n_max, int32_t hq, int32_t hkv, int32_t d, double scale,
                       const void *q, const void *k_cache, const void *v_cache,
                       const int32_t *ctx_offsets, const void *k_tree, const void *v_tree,
                       const uint64_t *anc, const int32_t *n_nodes, int b, int n, int h,
                       double *o, double *sc) {
    const int32_t W = (n_max + 63) / 64;
    const int g = h / (hq / hkv); /* query head h reads KV head floor(h / group) */
    const int64_t c0 = ctx_offsets[b], ctx = ctx_offsets[b + 1] - ctx_offsets[b];
    const int64_t qo = (((int64_t)b * n_max + n) * hq + h) * d;
    const int nn = n_nodes[b];
    /* visible keys: every cached position, then the tree nodes whose bit is set */
    int64_t nk = 0;
    double m = -INFINITY;
    for (int64_t j = 0; j < ctx; ++j) {
        const int64_t ko = ((c0 + j) * hkv + g) * d;
        double dot = 0.0;
        for (int e = 0; e < d; ++e)
            dot += (double)load_f(dtype, q, qo + e) * (double)load_f(dtype, k_cache, ko + e);
        sc[nk] = dot * scale;
        if (sc[nk] > m) m = sc[nk];
        ++nk;
    }
    for (int t = 0; t < nn; ++t) {
        if (!((anc[((int64_t)b * n_max + n) * W + t / 64] >> (t % 64)) & 1ull)) continue;
        const int64_t ko = (((int64_t)b * n_max + t) * hkv + g) * d;
        double dot = 0.0;
        for (int e = 0; e < d; ++e)
            dot += (double)load_f(dtype, q, qo + e) * (double)load_f(dtype, k_tree, ko + e);
        sc[nk] = dot * scale;
        if (sc[nk] > m) m = sc[nk];
        ++nk;
    }
    double den = 0.0;
    for (int64_t j = 0; j < nk; ++j) {
        sc[j] = exp(sc[j] - m);
        den += sc[j];
    }
    for (int e = 0; e < d; ++e) o[e] = 0.0;
    int64_t j = 0;
    for (int64_t p = 0; p < ctx; ++p, ++j) {
        const int64_t vo = ((c0 + p) * hkv + g) * d;
        for (int e = 0; e < d; ++e) o[e] += sc[j] * (double)load_f(dtype, v_cache, vo + e);
    }
    for (int t = 0; t < nn; ++t) {
        if (!((anc[((int64_t)b * n_max + n) * W + t / 64] >> (t % 64)) & 1ull)) continue;
        const int64_t vo = (((int64_t)b * n_max + t) * hkv + g) * d;
        for (int e = 0; e < d; ++e) o[e] += sc[j] * (double)load_f(dtype, v_tree, vo + e);
        ++j;
    }
    for (int e = 0; e < d; ++e) o[e] /= den;
}

void oracle_tree_attention(int dtype, int32_t batch, int32_t n_max, int32_t hq, int32_t hkv,
                           int32_t head_dim, double scale, const void *q, const void *k_cache,
                           const void *v_cache, const int32_t *ctx_offsets, const void *k_tree,
                           const void *v_tree, const uint64_t *anc, const int32_t *n_nodes,
                           void *out) {
    int64_t max_ctx = 0;
    for (int b = 0; b < batch; ++b)
        if (ctx_offsets[b + 1] - ctx_offsets[b] > max_ctx) max_ctx = ctx_offsets[b + 1] - ctx_offsets[b];
    const int64_t units = (int64_t)batch * n_max * hq;
#pragma omp parallel
    {
        double *o = (double *)malloc(sizeof(double) * (size_t)head_dim);
        double *sc = (double *)malloc(sizeof(double) * (size_t)(max_ctx + n_max));
#pragma omp for schedule(dynamic, 4)
        for (int64_t u = 0; u < units; ++u) {
            const int h = (int)(u % hq), n = (int)((u / hq) % n_max), b = (int)(u / hq / n_max);
            const int64_t oo = u * head_dim;
            if (n >= n_nodes[b]) {
                for (int e = 0; e < head_dim; ++e) store_f(dtype, out, oo + e, 0.0);
                continue;
            }
            attend_row(dtype, n_max, hq, hkv, head_dim, scale, q, k_cache, v_cache, ctx_offsets,
                       k_tree, v_tree, anc, n_nodes, b, n, h, o, sc);
            for (int e = 0; e < head_dim; ++e) store_f(dtype, out, oo + e, o[e]);
        }
        free(o);
        free(sc);
    }
}

void oracle_tree_attention_rows(int dtype, int32_t batch, int32_t n_max, int32_t hq, int32_t hkv,
                                int32_t head_dim, double scale, const void *q, const void *k_cache,
                                const void *v_cache, const int32_t *ctx_offsets,
                                const void *k_tree, const void *v_tree, const uint64_t *anc,
                                const int32_t *n_nodes, int64_t n_rows, const int32_t *rows,
                                double *out) {
    int64_t max_ctx = 0;
    for (int b = 0; b < batch; ++b)
        if (ctx_offsets[b + 1] - ctx_offsets[b] > max_ctx) max_ctx = ctx_offsets[b + 1] - ctx_offsets[b];
#pragma omp parallel
    {
        double *sc = (double *)malloc(sizeof(double) * (size_t)(max_ctx + n_max));
#pragma omp for schedule(dynamic, 1)
        for (int64_t i = 0; i < n_rows; ++i) {
            const int b = rows[3 * i], n = rows[3 * i + 1], h = rows[3 * i + 2];
            double *o = out + i * head_dim;
            if (n >= n_nodes[b]) {
                for (int e = 0; e < head_dim; ++e) o[e] = 0.0;
                continue;
            }
            attend_row(dtype, n_max, hq, hkv, head_dim, scale, q, k_cache, v_cache, ctx_offsets,
                       k_tree, v_tree, anc, n_nodes, b, n, h, o, sc);
        }
        free(sc);
    }
}

/* ------------------------------------------------------------------------ */
/* 4. greedy acceptance                                                     */

int oracle_accept(int dtype, const void *target_logits, int32_t vocab, int64_t row_stride,
                  int32_t batch, int32_t n_max, int32_t depth, const int32_t *parent,
                  const int32_t *token, const int32_t *n_nodes, int32_t *accept_len,
                  int32_t *path, int32_t *bonus, int32_t *target_argmax) {
    int nan_rows = 0;
    int32_t *amax = (int32_t *)malloc(sizeof(int32_t) * (size_t)batch * n_max);
    /* the target's greedy prediction after each node: lowest id attaining the max */
#pragma omp parallel for schedule(dynamic, 1) reduction(+ : nan_rows)
    for (int64_t u = 0; u < (int64_t)batch * n_max; ++u) {
        const int b = (int)(u / n_max), n = (int)(u % n_max);
        if (n >= n_nodes[b]) {
            amax[u] = -1;
            continue;
        }
        const int64_t base = u * row_stride;
        float best = load_f(dtype, target_logits, base);
        int32_t bi = 0, saw_nan = isnan(best);
        for (int32_t v = 1; v < vocab; ++v) {
            float z = load_f(dtype, target_logits, base + v);
            if (isnan(z)) saw_nan = 1;
            if (z > best) {
                best = z;
                bi = v;
            }
        }
        amax[u] = bi;
        nan_rows += saw_nan;
    }
    /* walk: from the root, follow the child whose token equals the target's
     * prediction at the current node; stop at the first mismatch */
    for (int b = 0; b < batch; ++b) {
        const int32_t *par = parent + (int64_t)b * n_max, *tok = token + (int64_t)b * n_max;
        const int32_t *a = amax + (int64_t)b * n_max;
        int cur = 0, L = 0;
        path[(int64_t)b * (depth + 1)] = 0;
        for (;;) {
            int next = -1;
            for (int c = 1; c < n_nodes[b]; ++c)
                if (par[c] == cur && tok[c] == a[cur]) {
                    next = c;
                    break;
                }
            if (next < 0) break;
            cur = next;
            ++L;
            path[(int64_t)b * (depth + 1) + L] = cur;
        }
        for (int i = L + 1; i <= depth; ++i) path[(int64_t)b * (depth + 1) + i] = -1;
        accept_len[b] = L;
        bonus[b] = a[cur];
        if (target_argmax)
            for (int n = 0; n < n_max; ++n) target_argmax[(int64_t)b * n_max + n] = a[n];
    }
    free(amax);
    return nan_rows;
}
