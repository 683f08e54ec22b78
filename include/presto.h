/*
 * presto.h -- C ABI of libpresto, the MI355X (gfx950) hot path of one
 * PRESTO draft-to-verify round ("PRESTO: Prefix-Aligned Tree Drafting for
 * Diffusion Speculative Decoding").
 *
 * A round is four calls, enqueued in order on one HIP stream:
 *
 *   presto_topk            per-position log-softmax normaliser and top-k
 *                          candidates of the drafter's block marginals
 *   presto_build_tree      prefix-aligned scoring and best-first tree
 *                          construction under a node budget, flattened
 *                          with its ancestor (tree-attention) mask
 *   presto_tree_attention  tree-masked verification attention of one
 *                          target layer over [cached prefix ; tree nodes]
 *   presto_accept          target argmax per node and the longest
 *                          accepted root-to-node path plus bonus token
 *
 * Conventions shared by every entry point:
 *
 * - Every tensor argument is a DEVICE pointer owned by the caller, row
 *   major with a contiguous innermost dimension.  Strides are in elements.
 *   The library allocates no device memory: scratch space comes from a
 *   caller-provided device workspace of at least *_workspace() bytes
 *   (a null workspace is allowed when that size is 0).  Its contents on
 *   entry are ignored; two calls in flight at the same time (on different
 *   streams) need distinct workspaces.  The one exception,
 *   presto_topk_noalloc, uses a fixed static device array of the library
 *   instead of a workspace.
 * - Every call is asynchronous on `stream` (0 = the null stream).  All
 *   argument checks happen on the host before anything is launched; on an
 *   error return nothing was enqueued.
 * - Storage dtype PRESTO_DT_BF16 means bfloat16 values (raw 16-bit
 *   patterns), PRESTO_DT_F32 means IEEE float32.
 * - Data errors found on the device never fault: the kernels OR bits into
 *   the optional caller word `flags` (device int32, may be NULL), which the
 *   caller reads after synchronising.  A call never clears `flags`.
 * - The only host state is a thread-local last-error string.
 * - Results are deterministic: the same inputs give bit-identical outputs.
 */
#ifndef PRESTO_H
#define PRESTO_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    PRESTO_OK = 0,
    PRESTO_ERR_INVALID_ARG = -1, /* rejected on the host; nothing launched          */
    PRESTO_ERR_UNSUPPORTED = -2, /* valid request the library does not implement   */
    PRESTO_ERR_WORKSPACE = -3,   /* workspace missing or smaller than *_workspace() */
    PRESTO_ERR_HIP = -4,         /* HIP runtime error; see presto_last_error()      */
    PRESTO_STATUS_MAX_ENUM_ = 0x7fffffff /* not a status: keeps the type 32 bits wide */
} presto_status;

/* Any other non-negative value is rejected with PRESTO_ERR_INVALID_ARG (the
 * last enumerator only keeps the type 32 bits wide). */
typedef enum { PRESTO_DT_BF16 = 0, PRESTO_DT_F32 = 1, PRESTO_DT_MAX_ENUM_ = 0x7fffffff } presto_dtype;

typedef enum {
    PRESTO_TREE_BEST_FIRST = 0,      /* commit on pop: exactly the B best prefixes by S        */
    PRESTO_TREE_BEST_FIRST_ALG2 = 1, /* Alg. 2 as printed: add children on expand, then TopB  */
    PRESTO_TREE_BEAM = 2             /* Alg. 1 beam search with global retention              */
} presto_tree_mode;

/* Bits ORed into the optional `flags` word. */
enum {
    PRESTO_FLAG_NAN_DRAFTER = 1, /* a drafter logit row held a NaN (or +inf)   */
    PRESTO_FLAG_NAN_TARGET = 2,  /* a live target logit row held a NaN         */
    PRESTO_FLAG_NGRAM_BAD = 4,   /* an n-gram entry was invalid and skipped    */
    PRESTO_FLAG_NGRAM_FULL = 8,  /* an n-gram entry found no free table slot   */
    PRESTO_FLAG_BAD_INDEX = 16,  /* presto_topk_rows: a row index outside the logits */
    PRESTO_FLAG_KV_COMMIT = 32   /* round bookkeeping: a sequence's slot, length or
                                    path was invalid; that sequence was skipped */
};

/* ------------------------------------------------------------------------ */
/* Stage 1: log-softmax normaliser and top-k candidates per drafter position.
 *
 * Defined by the diffusion marginal q_d = softmax(z_d) of each block
 * position d (Sec. 2.3, Eq. 6) and the per-position top-k candidate
 * extraction of Sec. 5.1 / Appendix C stage II.
 *
 * logits     [rows, row_stride] of dtype dt; row r = (sequence, position),
 *            only the first `vocab` entries of a row are read.
 * ids        [rows, k] int32 out: the k largest logits of the row, larger
 *            value first, lower id first among equal values (-0.0 == +0.0).
 * logprob    [rows, k] fp32 out: log q(id) = z_id - LSE.
 * lse        [rows] fp32 out, may be NULL: LSE = log sum_v exp(z_v), fp32.
 *            A row of only -inf gives LSE = -inf and logprob = -inf.
 * entropy    [rows] fp32 out, may be NULL: H = -sum_v q(v) log q(v) of the
 *            row's softmax (Appendix F), terms with q(v) = 0 taken as 0; it
 *            comes out of the same pass over the row as LSE.  A row of only
 *            -inf gives H = 0.
 * flags      optional: PRESTO_FLAG_NAN_DRAFTER when a row holds NaN or
 *            +inf; that row's outputs are then unspecified.
 * Diagnostic: once the call has completed, the first 4 bytes of the
 * workspace hold (uint32) the number of wave-sized chunks of the rows whose
 * candidates did not fit the fast path (more than 256 values in groups that
 * reach the chunk's k-th lane maximum: heavy ties) and were selected by the
 * slower exact pass.  The results are the same either way.
 * Limits: 1 <= k <= 16, k <= vocab, row_stride >= vocab, rows >= 0
 * (rows == 0 is a no-op).
 */
size_t presto_topk_workspace(int64_t rows, int32_t vocab, int32_t k);
presto_status presto_topk(presto_dtype dt, const void *logits, int64_t rows, int32_t vocab,
                          int64_t row_stride, int32_t k, int32_t *ids, float *logprob, float *lse,
                          float *entropy, int32_t *flags, void *ws, size_t ws_bytes,
                          hipStream_t stream);

/* presto_topk for callers that cannot allocate: code under HIP graph
 * capture, serving loops and harnesses that forbid device allocation.  Same
 * arguments, results and limits as presto_topk, without the workspace: the
 * partials live in a static device array of
 * PRESTO_TOPK_NOALLOC_SCRATCH_BYTES per GPU (held from the first call on
 * that GPU until the process ends).  A request whose
 * presto_topk_workspace(rows, vocab, k) exceeds it returns
 * PRESTO_ERR_WORKSPACE with nothing launched (at vocab 151936 that is more
 * than about 2500 rows at k = 4, 800 at k = 16).  Every call on one GPU
 * shares the array: calls that overlap on one GPU (on different streams)
 * race; calls ordered on one stream do not.  The workspace diagnostic of
 * presto_topk is not available here.
 */
#define PRESTO_TOPK_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)
presto_status presto_topk_noalloc(presto_dtype dt, const void *logits, int64_t rows,
                                  int32_t vocab, int64_t row_stride, int32_t k, int32_t *ids,
                                  float *logprob, float *lse, float *entropy, int32_t *flags,
                                  hipStream_t stream);

/* The same on gathered rows: output row r reads logits row row_index[r]
 * (int64 device, [rows]) of logits [logits_rows, row_stride].  An index
 * outside [0, logits_rows) reads as a row of only -inf and raises
 * PRESTO_FLAG_BAD_INDEX.  Used with presto_select_slots to read the next
 * round's drafter rows in place from a slot-logit matrix.  Same limits and
 * workspace as presto_topk (presto_topk_workspace(rows, vocab, k)).
 */
presto_status presto_topk_rows(presto_dtype dt, const void *logits, int64_t logits_rows,
                               const int64_t *row_index, int64_t rows, int32_t vocab,
                               int64_t row_stride, int32_t k, int32_t *ids, float *logprob,
                               float *lse, float *entropy, int32_t *flags, void *ws,
                               size_t ws_bytes, hipStream_t stream);

/* Entropy-adaptive prefix weight (Appendix F):
 *   lambda[r] = beta * H[r] / (H[r] + C), fp32, H from presto_topk's
 * entropy output ([batch, depth] rows give a [batch, depth] lambda for
 * presto_build_tree with lambda_per_seq = 1).  Low-entropy (confident)
 * positions get a weight near 0, high-entropy ones approach beta.
 * entropy, lambda [rows] fp32 device; entropy must be finite and >= 0.
 * Limits: beta > 0 and C > 0, finite; rows >= 0 (0 is a no-op).
 */
presto_status presto_entropy_lambda(int64_t rows, const float *entropy, float beta, float c,
                                    float *lambda, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Prefix-aligned signal from a trigram model (Sec. 5.1: rho is an n-gram
 * model with n = 3).  The table is built once (off the per-round path) and
 * each round gathers the lattice log_rho[b, d, r2, r1, r] that
 * presto_build_tree reads, so the tree search itself never probes it.
 *
 * Table: caller device memory of presto_ngram_table_bytes(capacity) bytes,
 * 8-byte aligned, capacity a power of two in 64 .. 2^32 (an open-addressing
 * hash table; keep it at most about half full for short probes).  Tokens
 * must lie in [0, 2^21).
 *
 * presto_ngram_clear   empties the table (must precede the first insert).
 * presto_ngram_insert  adds n entries log rho(t[i] | t2[i], t1[i]) (device
 *   arrays, t2 the older context token).  log rho must be finite and <= 0;
 *   -0.0 is stored as +0.0.  A key inserted more than once keeps its
 *   largest value, in any order of insertion.  Invalid entries are skipped
 *   with PRESTO_FLAG_NGRAM_BAD, entries finding no free slot with
 *   PRESTO_FLAG_NGRAM_FULL (flags may be NULL).  Calls may be repeated to
 *   add more entries; concurrent inserts and gathers on one table race.
 * presto_ngram_gather  fills log_rho [batch, depth, k, k, k] fp32 from
 *   ids [batch, depth, k] (presto_topk's candidates), prev_token [batch]
 *   (the committed token before the root, or -1 if none) and root_token
 *   [batch]: entry (b, d, r2, r1, r) is log rho(t | t2, t1) with
 *     t  = ids[b, d, r],
 *     t1 = ids[b, d-1, r1] for d >= 1, else the root token,
 *     t2 = ids[b, d-2, r2] for d >= 2, the root token for d = 1, else
 *          prev_token[b],
 *   or floor_log_rho (finite, <= 0) when that trigram is absent or a token
 *   lies outside [0, 2^21).  This is the rank-slot convention of
 *   presto_build_tree (slot 0 for a token outside the block); slots a depth
 *   does not read repeat slot 0.  Limits: depth 1 .. 32, k 1 .. 16.
 */
size_t presto_ngram_table_bytes(int64_t capacity); /* 0 for an invalid capacity */
presto_status presto_ngram_clear(void *table, int64_t capacity, hipStream_t stream);
presto_status presto_ngram_insert(void *table, int64_t capacity, int64_t n, const int32_t *t2,
                                  const int32_t *t1, const int32_t *t, const float *log_rho,
                                  int32_t *flags, hipStream_t stream);
presto_status presto_ngram_gather(const void *table, int64_t capacity, float floor_log_rho,
                                  int32_t batch, int32_t depth, int32_t k, const int32_t *ids,
                                  const int32_t *prev_token, const int32_t *root_token,
                                  float *log_rho, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Stage 2: prefix-aligned scoring and best-first tree construction.
 *
 * Token score (Sec. 4.1, Eq. 9): s = fl(log q_d(t) + fl(lambda_d * log rho_d)),
 * path score S(root) = 0, S(child) = fl(S(parent) + s), fp32, no fused
 * multiply-add.  rho is a trigram over the two preceding tokens, given as
 * the lattice log_rho[b, d, r2, r1, r] over candidate ranks, where r1 is the
 * rank of the parent token and r2 of the grandparent; rank slot 0 stands
 * for a token outside the block (the root and the committed context).
 * A child at depth d+1 reads drafter row d (d = 0 .. depth-1).
 *
 * Expanding a node yields its top-`branch` candidates by s (larger s first,
 * lower rank on ties) if its depth is below `depth`, else nothing.
 * Nodes are ranked by the total order: larger S first, then the rank path
 * compared lexicographically with a proper prefix before its extensions.
 *
 * PRESTO_TREE_BEST_FIRST (Sec. 4.2, Alg. 2 with commit on pop): the tree
 *   is exactly the `budget` best non-root prefixes of the candidate tree
 *   (the closed form of Sec. 4.2 via Eq. 3), or the whole candidate tree
 *   when it has fewer nodes.  This relies on the input bounds below
 *   (logprob <= 0, log_rho <= 0, lambda >= 0: every s <= 0, so S never
 *   increases along a path); outside them the tree is unspecified.
 * PRESTO_TREE_BEST_FIRST_ALG2: Alg. 2 as printed: every pop adds all its
 *   children to T; stop once T holds `budget` non-root nodes; keep TopB(T).
 * PRESTO_TREE_BEAM (Sec. 4.2, Alg. 1, beam search with global retention):
 *   the beam starts as {root}; at each depth every beam node is expanded
 *   (its top-`branch` children join T), and the `beam_width` best of them
 *   in the total order form the next beam.  Depths are taken while T holds
 *   fewer than `budget` non-root nodes (checked before each depth), at most
 *   `depth` of them.  The tree is TopB(T): the `budget` best nodes of T.
 *   Limits: 1 <= beam_width <= 64, beam_width * k <= 256.
 *
 * The budget counts draft (non-root) nodes: the output has N = budget + 1
 * rows, row 0 being the root (the last committed token, root_token[b]).
 */
typedef struct {
    int32_t batch;
    int32_t depth;  /* block length D = maximal tree depth, 1 .. 32 (24 if k=16) */
    int32_t k;      /* candidates per position, 1 .. 16                        */
    int32_t branch; /* children per expansion, 1 .. k                          */
    int32_t budget; /* B, draft nodes excluding the root, 1 .. 1023           */
    int32_t mode;   /* presto_tree_mode                                        */
    int32_t beam_width; /* W, PRESTO_TREE_BEAM only (ignored otherwise)        */
    int32_t lambda_per_seq; /* 0: lambda is [depth]; 1: lambda is [batch, depth] */
} presto_tree_desc;

/* ids, logprob [batch, depth, k] from presto_topk (logprob <= 0);
 * log_rho [batch, depth, k, k, k] fp32, finite and <= 0, or NULL for s = log q;
 * lambda [depth] fp32, finite and >= 0 (device), or [batch, depth] when
 *   desc->lambda_per_seq is 1 (e.g. from presto_entropy_lambda);
 * root_token [batch] int32.
 * Outputs, N = budget + 1 rows per sequence, rows in the total order above
 * (every parent precedes its children):
 *   n_nodes [batch]             live rows, 1 .. N
 *   parent, token, depth_out, rank [batch, N] int32   (root: -1, root_token, 0, -1)
 *   score   [batch, N] fp32     S of the node
 *   anc     [batch, N, ceil(N/64)] uint64   bit m of row n set iff node m is n
 *                                           or an ancestor of n
 * Rows n >= n_nodes: parent/token/depth/rank = -1, score = -inf, anc = 0.
 */
size_t presto_build_tree_workspace(const presto_tree_desc *desc);
presto_status presto_build_tree(const presto_tree_desc *desc, const int32_t *ids,
                                const float *logprob, const float *log_rho, const float *lambda,
                                const int32_t *root_token, int32_t *n_nodes, int32_t *parent,
                                int32_t *token, int32_t *depth_out, int32_t *rank, float *score,
                                uint64_t *anc, void *ws, size_t ws_bytes, hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Stage 3: tree-masked verification attention, one layer.
 *
 * Appendix C stage I: each draft token attends to the committed prefix
 * (its exact KV cache) and to its ancestors in the draft tree (and itself).
 * For sequence b, node n < n_nodes[b], query head h, KV head g = h / (hq/hkv):
 *   O[b,n,h] = softmax_j(scale * q[b,n,h] . k_j) v_j
 * over j in {cache positions of b} U {tree nodes m : anc bit m of row n}.
 * Rows n >= n_nodes[b] are written as zeros.
 *
 * q        [batch, n_max, hq, head_dim]
 * k_cache, v_cache [cache_rows, hkv, head_dim]
 * ctx_offsets, by desc->ctx_layout:
 *   PRESTO_CTX_PACKED: [batch + 1] int32 device, non-decreasing,
 *          ctx_offsets[0] = 0; sequence b owns cache rows
 *          ctx_offsets[b] .. ctx_offsets[b+1]-1 (ctx_b = their count)
 *   PRESTO_CTX_SLOTS: [batch, 2] int32 device (start_b, ctx_b); sequence b
 *          owns rows start_b .. start_b + ctx_b - 1, with room after them
 *          for presto_commit_kv to append to
 *   every ctx_b <= max_ctx (ctx_b = 0 is allowed)
 * k_tree, v_tree [batch, n_max, hkv, head_dim]: K/V of the tree nodes
 * anc      [batch, n_max, ceil(n_max/64)] from presto_build_tree
 * n_nodes  [batch] int32 device, 1 .. n_max
 * out      [batch, n_max, hq, head_dim], dtype dt
 * Arithmetic: bf16 inputs use bf16 matrix cores with fp32 accumulation and
 * fp32 softmax; fp32 inputs use fp32 throughout.
 * Limits: head_dim in {64, 128}; hq % hkv == 0; n_max <= 1024.
 */
typedef enum { PRESTO_CTX_PACKED = 0, PRESTO_CTX_SLOTS = 1 } presto_ctx_layout;

typedef struct {
    int32_t batch, n_max, hq, hkv, head_dim, max_ctx;
    float scale; /* usually 1/sqrt(head_dim) */
    presto_dtype dt;
    int32_t ctx_layout; /* presto_ctx_layout */
    /* Sum of ctx_b over the batch, or 0 when the caller does not know it.
     * A scheduling hint only: the result is the same for any value.  With
     * ragged contexts it lets the context be split by the actual total, and
     * the workgroups be dealt over the splits each sequence really has,
     * instead of assuming batch x max_ctx. */
    int64_t total_ctx;
} presto_attn_desc;

size_t presto_tree_attention_workspace(const presto_attn_desc *desc);
presto_status presto_tree_attention(const presto_attn_desc *desc, const void *q,
                                    const void *k_cache, const void *v_cache,
                                    const int32_t *ctx_offsets, const void *k_tree,
                                    const void *v_tree, const uint64_t *anc,
                                    const int32_t *n_nodes, void *out, void *ws, size_t ws_bytes,
                                    hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Stage 4: greedy verification of the tree (Eq. 1 at temperature 0) and the
 * bonus token (Appendix C stage I: the position after the last accepted
 * token takes the model's own prediction).
 *
 * target_logits [batch * n_max, row_stride], dtype dt: row (b, n) is the
 *          target's next-token logits after node n; rows n >= n_nodes[b]
 *          are not read.
 * a[n] = lowest id attaining the row maximum.  From the root, repeatedly
 * move to the child whose token equals a[current]; stop when none does.
 * accept_len [batch] int32 out: accepted draft tokens, 0 .. depth
 * path       [batch, depth + 1] int32 out: node rows root .. last accepted,
 *            then -1
 * bonus      [batch] int32 out: a[last accepted node]
 * target_argmax [batch, n_max] int32 out, may be NULL: a[n], -1 for
 *            padding rows
 * flags      optional: PRESTO_FLAG_NAN_TARGET when a live row holds a NaN;
 *            that row's argmax is then unspecified.
 * parent, token, n_nodes as produced by presto_build_tree (sibling tokens
 * distinct).  Limits: n_max <= 1024, depth >= 1.
 */
size_t presto_accept_workspace(int32_t batch, int32_t n_max, int32_t vocab);
presto_status presto_accept(presto_dtype dt, const void *target_logits, int32_t vocab,
                            int64_t row_stride, int32_t batch, int32_t n_max, int32_t depth,
                            const int32_t *parent, const int32_t *token, const int32_t *n_nodes,
                            int32_t *accept_len, int32_t *path, int32_t *bonus,
                            int32_t *target_argmax, int32_t *flags, void *ws, size_t ws_bytes,
                            hipStream_t stream);

/* ------------------------------------------------------------------------ */
/* Bookkeeping between rounds.
 *
 * presto_commit_kv (Appendix C stage I: the accepted tokens join the
 * committed prefix for the next round): for every sequence b, the tree K/V
 * rows of path[b, 0 .. accept_len[b]] (the root, then the accepted draft
 * nodes, as written by presto_accept) are appended in that order to the
 * cache after its ctx_b rows, and ctx_b grows by accept_len[b] + 1.
 *   k_tree, v_tree [batch, n_max, hkv, head_dim] (dtype dt), as given to
 *                  presto_tree_attention
 *   path, accept_len from presto_accept ([batch, depth + 1], [batch])
 *   k_cache, v_cache [cache_rows, hkv, head_dim] in PRESTO_CTX_SLOTS layout
 *   ctx [batch, 2] int32 device (start_b, ctx_b), updated in place
 *   ctx_cap [batch] int32 device: sequence b owns rows start_b ..
 *                  start_b + ctx_cap[b] - 1
 * A sequence whose slot lies outside the cache, would overflow its
 * capacity, or whose path is invalid is left unchanged and raises
 * PRESTO_FLAG_KV_COMMIT.  16-byte aligned tensors.  The tree rows of the
 * next round's root (the bonus token) are the caller's: its K/V come from
 * the next verification forward.
 */
typedef struct {
    int32_t batch, n_max, hkv, head_dim, depth;
    presto_dtype dt;
} presto_commit_desc;

presto_status presto_commit_kv(const presto_commit_desc *desc, const void *k_tree,
                               const void *v_tree, const int32_t *path, const int32_t *accept_len,
                               void *k_cache, void *v_cache, int64_t cache_rows, int32_t *ctx,
                               const int32_t *ctx_cap, int32_t *flags, hipStream_t stream);

/* Quadratic self-speculation (Appendix C).  The verification forward also
 * denoises `slots` mask positions after every tree node; slot j (1-based)
 * of node n stands for the position j places after n.  Their logits form
 * the matrix [batch, n_max, slots, V] (row (b, n, j - 1)).
 *
 * presto_select_slots (Appendix C stage II): only the block of the last accepted
 * node a = path[b, accept_len[b]] feeds the next round.  Writes row_index
 * [batch, slots - first_slot] int64: next drafter row d of sequence b reads
 * slot first_slot + d + 1 of a, i.e. matrix row
 * (b * n_max + a) * slots + first_slot + d.  With first_slot = 1 the first
 * slot, whose position the bonus token (the next root) fills, is skipped.
 * An invalid path raises PRESTO_FLAG_KV_COMMIT and reads the root's block.
 * Limits: 0 <= first_slot < slots <= 64.
 *
 * presto_flatten_slots (Appendix C stage IV): the next forward's input puts a
 * block of `slots` mask slots after every tree node: composite row
 * r = n * (1 + slots) + j is node n (j = 0) or its slot j.  Writes
 *   pos_out [batch, R] int32, R = n_max * (1 + slots): root_pos[b] +
 *          depth(n) + j for live rows, -1 for rows of nodes n >= n_nodes
 *   anc_out [batch, R, ceil(R / 64)] uint64: a node row sees the node rows of
 *          its root path (itself included); a slot row sees the same node
 *          rows and every slot of its own block; dead rows see nothing
 *   n_rows  [batch] int32: n_nodes[b] * (1 + slots), the live prefix
 * from depth, anc [batch, n_max, ceil(n_max / 64)], n_nodes of
 * presto_build_tree and root_pos [batch] (the position of the root).  The
 * result is a valid presto_tree_attention mask when R <= 1024.
 * Limits: 1 <= slots <= 64, R <= 65536.
 */
presto_status presto_select_slots(int32_t batch, int32_t n_max, int32_t depth, int32_t slots,
                                  int32_t first_slot, const int32_t *path,
                                  const int32_t *accept_len, int64_t *row_index, int32_t *flags,
                                  hipStream_t stream);
presto_status presto_flatten_slots(int32_t batch, int32_t n_max, int32_t slots,
                                   const int32_t *depth, const uint64_t *anc,
                                   const int32_t *n_nodes, const int32_t *root_pos,
                                   int32_t *pos_out, uint64_t *anc_out, int32_t *n_rows,
                                   hipStream_t stream);

/* ------------------------------------------------------------------------ */
const char *presto_status_string(presto_status s);
const char *presto_last_error(void); /* thread-local text of the last failure ("" if none) */
const char *presto_version(void);

#ifdef __cplusplus
}
#endif
#endif /* PRESTO_H */
