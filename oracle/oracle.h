/*
 * CPU oracle for the PRESTO draft-to-verify round -- TEST INFRASTRUCTURE.
 *
 * This library exists to check the HIP path, never to stand in for it.
 * Only the test suite, the smoke check and the bench's CPU-baseline leg
 * may load it.  It shares no code with the HIP library: separate headers,
 * separate sources, separate build.
 *
 * Storage dtypes: ORACLE_BF16 = bf16 bit patterns (uint16), ORACLE_F32 = fp32.
 */
#ifndef PRESTO_ORACLE_H
#define PRESTO_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { ORACLE_BF16 = 0, ORACLE_F32 = 1 };
enum { ORACLE_BEST_FIRST = 0, ORACLE_BEST_FIRST_ALG2 = 1, ORACLE_BEAM = 2 };

void oracle_set_threads(int n);
int oracle_get_threads(void);

/* Per-row log-softmax normaliser and top-k (Sec. 4.1 / Appendix C stage II).
 * Returns the number of rows holding a NaN (their outputs are unspecified). */
int oracle_topk(int dtype, const void *logits, int64_t rows, int32_t vocab, int64_t row_stride,
                int32_t k, int32_t *ids, float *logprob, float *lse);

/* Softmax entropy H_d of each row (Appendix F), fp64; 0 for a row of only -inf. */
void oracle_entropy(int dtype, const void *logits, int64_t rows, int32_t vocab, int64_t row_stride,
                    double *entropy);

/* Entropy-adaptive weight beta * H / (H + C) (Appendix F), fp64. */
void oracle_entropy_lambda(int64_t rows, const double *entropy, double beta, double c,
                           double *lambda);

/* Prefix-aligned scoring (Eq. 9) and best-first tree construction (Sec. 4.2).
 * lambda is [depth], or [batch, depth] when lambda_per_seq is nonzero.
 * Returns 0, or -1 on an argument the oracle cannot represent. */
int oracle_build_tree(int mode, int32_t batch, int32_t depth, int32_t k, int32_t branch,
                      int32_t budget, int32_t beam_width, const int32_t *ids, const float *logprob,
                      const float *log_rho, const float *lambda, int32_t lambda_per_seq,
                      const int32_t *root_token,
                      int32_t *n_nodes, int32_t *parent, int32_t *token, int32_t *depth_out,
                      int32_t *rank, float *score, uint64_t *anc);

/* Tree-masked attention over [cached prefix ; ancestor tree nodes] (Appendix C stage I). */
void oracle_tree_attention(int dtype, int32_t batch, int32_t n_max, int32_t hq, int32_t hkv,
                           int32_t head_dim, double scale, const void *q, const void *k_cache,
                           const void *v_cache, const int32_t *ctx_offsets, const void *k_tree,
                           const void *v_tree, const uint64_t *anc, const int32_t *n_nodes,
                           void *out);

/* Same attention for a list of (b, n, h) rows only, exact fp64 output [n_rows, head_dim]. */
void oracle_tree_attention_rows(int dtype, int32_t batch, int32_t n_max, int32_t hq, int32_t hkv,
                                int32_t head_dim, double scale, const void *q, const void *k_cache,
                                const void *v_cache, const int32_t *ctx_offsets,
                                const void *k_tree, const void *v_tree, const uint64_t *anc,
                                const int32_t *n_nodes, int64_t n_rows, const int32_t *rows,
                                double *out);

/* Greedy verification (Eq. 1 at temperature 0) and the bonus token (Appendix C stage I).
 * Returns the number of live node rows holding a NaN. */
int oracle_accept(int dtype, const void *target_logits, int32_t vocab, int64_t row_stride,
                  int32_t batch, int32_t n_max, int32_t depth, const int32_t *parent,
                  const int32_t *token, const int32_t *n_nodes, int32_t *accept_len,
                  int32_t *path, int32_t *bonus, int32_t *target_argmax);

#ifdef __cplusplus
}
#endif
#endif
