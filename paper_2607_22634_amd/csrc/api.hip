// Host side of libpresto: argument validation, workspace sizing, error
// reporting and dispatch to the stage launchers.  Nothing here touches the
// GPU before every check has passed.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include "common.hpp"

namespace presto_host {

size_t topk_workspace_bytes(int64_t rows, int32_t vocab, int32_t k);
presto_status launch_topk_noalloc(bool bf16, const void* logits, int64_t rows, int32_t vocab,
                                  int64_t row_stride, int32_t k, int32_t* ids, float* logprob,
                                  float* lse, float* entropy, int32_t* flags, hipStream_t stream);
presto_status launch_entropy_lambda(int64_t rows, const float* entropy, float beta, float c,
                                    float* lambda, hipStream_t stream);
presto_status launch_topk(bool bf16, const void* logits, const int64_t* row_index,
                          int64_t logits_rows, int64_t rows, int32_t vocab, int64_t row_stride,
                          int32_t k, int32_t* ids, float* logprob, float* lse, float* entropy,
                          int32_t* flags, void* ws, hipStream_t stream);
presto_status launch_commit_kv(const presto_commit_desc* d, const void* k_tree, const void* v_tree,
                               const int32_t* path, const int32_t* accept_len, void* k_cache,
                               void* v_cache, int64_t cache_rows, int32_t* ctx,
                               const int32_t* ctx_cap, int32_t* flags, hipStream_t stream);
presto_status launch_select_slots(int32_t batch, int32_t n_max, int32_t depth, int32_t slots,
                                  int32_t first_slot, const int32_t* path,
                                  const int32_t* accept_len, int64_t* row_index, int32_t* flags,
                                  hipStream_t stream);
presto_status launch_flatten_slots(int32_t batch, int32_t n_max, int32_t slots,
                                   const int32_t* depth, const uint64_t* anc,
                                   const int32_t* n_nodes, const int32_t* root_pos,
                                   int32_t* pos_out, uint64_t* anc_out, int32_t* n_rows,
                                   hipStream_t stream);
bool tree_build_fits(int D, int k, int branch, int N, int beam_width, bool alg2);
int tree_max_depth(int k);
presto_status launch_build_tree(const presto_tree_desc* desc, const int32_t* ids,
                                const float* logprob, const float* log_rho, const float* lambda,
                                const int32_t* root_token, int32_t* n_nodes, int32_t* parent,
                                int32_t* token, int32_t* depth, int32_t* rank, float* score,
                                uint64_t* anc, hipStream_t stream);
size_t attn_workspace_bytes(const presto_attn_desc* d);
presto_status launch_tree_attention(const presto_attn_desc* d, const void* q, const void* k_cache,
                                    const void* v_cache, const int32_t* ctx_offsets,
                                    const void* k_tree, const void* v_tree, const uint64_t* anc,
                                    const int32_t* n_nodes, void* out, void* ws,
                                    hipStream_t stream);
presto_status launch_ngram_clear(void* table, int64_t capacity, hipStream_t stream);
presto_status launch_ngram_insert(void* table, int64_t capacity, int64_t n, const int32_t* t2,
                                  const int32_t* t1, const int32_t* t, const float* log_rho,
                                  int32_t* flags, hipStream_t stream);
presto_status launch_ngram_gather(const void* table, int64_t capacity, float floor_v,
                                  int32_t batch, int32_t D, int32_t k, const int32_t* ids,
                                  const int32_t* prev_token, const int32_t* root_token,
                                  float* log_rho, hipStream_t stream);
size_t accept_workspace_bytes(int32_t batch, int32_t n_max, int32_t vocab);
presto_status launch_accept(bool bf16, const void* logits, int32_t vocab, int64_t row_stride,
                            int32_t batch, int32_t n_max, int32_t depth, const int32_t* parent,
                            const int32_t* token, const int32_t* n_nodes, int32_t* accept_len,
                            int32_t* path, int32_t* bonus, int32_t* target_argmax, int32_t* flags,
                            void* ws, hipStream_t stream);

static thread_local char g_err[512] = "";

presto_status set_error(presto_status s, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return s;
}

presto_status check_launch(const char* what) {
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return set_error(PRESTO_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
    return PRESTO_OK;
}

}  // namespace presto_host

using namespace presto_host;

#define REQUIRE(cond, ...)                                        \
    do {                                                          \
        if (!(cond)) return set_error(PRESTO_ERR_INVALID_ARG, __VA_ARGS__); \
    } while (0)

static bool valid_dtype(presto_dtype dt) { return dt == PRESTO_DT_BF16 || dt == PRESTO_DT_F32; }

// rows x (1024-entry chunks of the vocabulary) stays below 2^31 (the
// kernels' wave index); checked by division, so that no product overflows
static bool rows_fit(int64_t rows, int32_t vocab) {
    return rows >= 0 && vocab >= 1 && rows < (((int64_t)1 << 31) - 1) / ((vocab + 1023) / 1024);
}

static presto_status check_ws(void* ws, size_t have, size_t need) {
    if (need > 0 && (ws == nullptr || have < need))
        return set_error(PRESTO_ERR_WORKSPACE, "workspace of %zu bytes needed, %zu given", need,
                         ws ? have : (size_t)0);
    return PRESTO_OK;
}

extern "C" {

size_t presto_topk_workspace(int64_t rows, int32_t vocab, int32_t k) {
    if (rows <= 0 || vocab <= 0 || k <= 0 || k > 16 || !rows_fit(rows, vocab)) return 0;
    return topk_workspace_bytes(rows, vocab, k);
}

presto_status presto_topk(presto_dtype dt, const void* logits, int64_t rows, int32_t vocab,
                          int64_t row_stride, int32_t k, int32_t* ids, float* logprob, float* lse,
                          float* entropy, int32_t* flags, void* ws, size_t ws_bytes,
                          hipStream_t stream) {
    g_err[0] = 0;
    REQUIRE(valid_dtype(dt), "presto_topk: unknown dtype %d", (int)dt);
    REQUIRE(rows >= 0, "presto_topk: rows < 0");
    REQUIRE(vocab >= 1, "presto_topk: vocab < 1");
    REQUIRE(k >= 1 && k <= vocab, "presto_topk: k=%d outside 1..vocab", k);
    REQUIRE(row_stride >= vocab, "presto_topk: row_stride < vocab");
    if (k > 16) return set_error(PRESTO_ERR_UNSUPPORTED, "presto_topk: k=%d > 16", k);
    if (rows == 0) return PRESTO_OK;
    REQUIRE(logits && ids && logprob, "presto_topk: null pointer");
    REQUIRE(rows_fit(rows, vocab),
            "presto_topk: too many rows");
    presto_status st = check_ws(ws, ws_bytes, presto_topk_workspace(rows, vocab, k));
    if (st != PRESTO_OK) return st;
    return launch_topk(dt == PRESTO_DT_BF16, logits, nullptr, rows, rows, vocab, row_stride, k, ids,
                       logprob, lse, entropy, flags, ws, stream);
}

presto_status presto_topk_noalloc(presto_dtype dt, const void* logits, int64_t rows,
                                  int32_t vocab, int64_t row_stride, int32_t k, int32_t* ids,
                                  float* logprob, float* lse, float* entropy, int32_t* flags,
                                  hipStream_t stream) {
    g_err[0] = 0;
    REQUIRE(valid_dtype(dt), "presto_topk_noalloc: unknown dtype %d", (int)dt);
    REQUIRE(rows >= 0, "presto_topk_noalloc: rows < 0");
    REQUIRE(vocab >= 1, "presto_topk_noalloc: vocab < 1");
    REQUIRE(k >= 1 && k <= vocab, "presto_topk_noalloc: k=%d outside 1..vocab", k);
    REQUIRE(row_stride >= vocab, "presto_topk_noalloc: row_stride < vocab");
    if (k > 16) return set_error(PRESTO_ERR_UNSUPPORTED, "presto_topk_noalloc: k=%d > 16", k);
    if (rows == 0) return PRESTO_OK;
    REQUIRE(logits && ids && logprob, "presto_topk_noalloc: null pointer");
    REQUIRE(rows_fit(rows, vocab),
            "presto_topk_noalloc: too many rows");
    return launch_topk_noalloc(dt == PRESTO_DT_BF16, logits, rows, vocab, row_stride, k, ids,
                               logprob, lse, entropy, flags, stream);
}

presto_status presto_topk_rows(presto_dtype dt, const void* logits, int64_t logits_rows,
                               const int64_t* row_index, int64_t rows, int32_t vocab,
                               int64_t row_stride, int32_t k, int32_t* ids, float* logprob,
                               float* lse, float* entropy, int32_t* flags, void* ws,
                               size_t ws_bytes, hipStream_t stream) {
    g_err[0] = 0;
    REQUIRE(valid_dtype(dt), "presto_topk_rows: unknown dtype %d", (int)dt);
    REQUIRE(rows >= 0 && logits_rows >= 0, "presto_topk_rows: negative row count");
    REQUIRE(vocab >= 1, "presto_topk_rows: vocab < 1");
    REQUIRE(k >= 1 && k <= vocab, "presto_topk_rows: k=%d outside 1..vocab", k);
    REQUIRE(row_stride >= vocab, "presto_topk_rows: row_stride < vocab");
    if (k > 16) return set_error(PRESTO_ERR_UNSUPPORTED, "presto_topk_rows: k=%d > 16", k);
    if (rows == 0) return PRESTO_OK;
    REQUIRE(logits && row_index && ids && logprob, "presto_topk_rows: null pointer");
    REQUIRE(logits_rows >= 1, "presto_topk_rows: no logits rows");
    REQUIRE(rows_fit(rows, vocab),
            "presto_topk_rows: too many rows");
    presto_status st = check_ws(ws, ws_bytes, presto_topk_workspace(rows, vocab, k));
    if (st != PRESTO_OK) return st;
    return launch_topk(dt == PRESTO_DT_BF16, logits, row_index, logits_rows, rows, vocab,
                       row_stride, k, ids, logprob, lse, entropy, flags, ws, stream);
}

presto_status presto_entropy_lambda(int64_t rows, const float* entropy, float beta, float c,
                                    float* lambda, hipStream_t stream) {
    g_err[0] = 0;
    REQUIRE(rows >= 0, "presto_entropy_lambda: rows < 0");
    REQUIRE(isfinite(beta) && beta > 0.f, "presto_entropy_lambda: beta must be positive");
    REQUIRE(isfinite(c) && c > 0.f, "presto_entropy_lambda: C must be positive");
    if (rows == 0) return PRESTO_OK;
    REQUIRE(entropy && lambda, "presto_entropy_lambda: null pointer");
    return launch_entropy_lambda(rows, entropy, beta, c, lambda, stream);
}

static bool ngram_capacity_ok(int64_t capacity) {
    return capacity >= 64 && capacity <= ((int64_t)1 << 32) && (capacity & (capacity - 1)) == 0;
}

size_t presto_ngram_table_bytes(int64_t capacity) {
    if (!ngram_capacity_ok(capacity)) return 0;
    return (size_t)capacity * (sizeof(uint64_t) + sizeof(uint32_t));
}

presto_status presto_ngram_clear(void* table, int64_t capacity, hipStream_t stream) {
    g_err[0] = 0;
    REQUIRE(ngram_capacity_ok(capacity),
            "presto_ngram_clear: capacity %lld is not a power of two in 64 .. 2^32",
            (long long)capacity);
    REQUIRE(table, "presto_ngram_clear: null table");
    REQUIRE((uintptr_t)table % 8 == 0, "presto_ngram_clear: table not 8-byte aligned");
    return launch_ngram_clear(table, capacity, stream);
}

presto_status presto_ngram_insert(void* table, int64_t capacity, int64_t n, const int32_t* t2,
                                  const int32_t* t1, const int32_t* t, const float* log_rho,
                                  int32_t* flags, hipStream_t stream) {
    g_err[0] = 0;
    REQUIRE(ngram_capacity_ok(capacity),
            "presto_ngram_insert: capacity %lld is not a power of two in 64 .. 2^32",
            (long long)capacity);
    REQUIRE(n >= 0 && n <= ((int64_t)1 << 32), "presto_ngram_insert: n outside 0 .. 2^32");
    if (n == 0) return PRESTO_OK;
    REQUIRE(table && t2 && t1 && t && log_rho, "presto_ngram_insert: null pointer");
    REQUIRE((uintptr_t)table % 8 == 0, "presto_ngram_insert: table not 8-byte aligned");
    return launch_ngram_insert(table, capacity, n, t2, t1, t, log_rho, flags, stream);
}

presto_status presto_ngram_gather(const void* table, int64_t capacity, float floor_log_rho,
                                  int32_t batch, int32_t depth, int32_t k, const int32_t* ids,
                                  const int32_t* prev_token, const int32_t* root_token,
                                  float* log_rho, hipStream_t stream) {
    g_err[0] = 0;
    REQUIRE(ngram_capacity_ok(capacity),
            "presto_ngram_gather: capacity %lld is not a power of two in 64 .. 2^32",
            (long long)capacity);
    REQUIRE(isfinite(floor_log_rho) && floor_log_rho <= 0.f,
            "presto_ngram_gather: floor must be finite and <= 0");
    REQUIRE(batch >= 0, "presto_ngram_gather: batch < 0");
    REQUIRE(depth >= 1 && depth <= 32, "presto_ngram_gather: depth=%d outside 1..32", depth);
    REQUIRE(k >= 1 && k <= 16, "presto_ngram_gather: k=%d outside 1..16", k);
    if (batch == 0) return PRESTO_OK;
    REQUIRE(table && ids && prev_token && root_token && log_rho,
            "presto_ngram_gather: null pointer");
    REQUIRE((uintptr_t)table % 8 == 0, "presto_ngram_gather: table not 8-byte aligned");
    return launch_ngram_gather(table, capacity, floor_log_rho, batch, depth, k, ids, prev_token,
                               root_token, log_rho, stream);
}

size_t presto_build_tree_workspace(const presto_tree_desc* desc) {
    (void)desc;
    return 0;
}

presto_status presto_build_tree(const presto_tree_desc* desc, const int32_t* ids,
                                const float* logprob, const float* log_rho, const float* lambda,
                                const int32_t* root_token, int32_t* n_nodes, int32_t* parent,
                                int32_t* token, int32_t* depth_out, int32_t* rank, float* score,
                                uint64_t* anc, void* ws, size_t ws_bytes, hipStream_t stream) {
    g_err[0] = 0;
    (void)ws;
    (void)ws_bytes;
    REQUIRE(desc, "presto_build_tree: null descriptor");
    const presto_tree_desc d = *desc;
    REQUIRE(d.batch >= 0, "presto_build_tree: batch < 0");
    REQUIRE(d.depth >= 1 && d.depth <= 32, "presto_build_tree: depth=%d outside 1..32", d.depth);
    REQUIRE(d.k >= 1 && d.k <= 16, "presto_build_tree: k=%d outside 1..16", d.k);
    REQUIRE(d.branch >= 1 && d.branch <= d.k, "presto_build_tree: branch=%d outside 1..k",
            d.branch);
    REQUIRE(d.budget >= 1 && d.budget <= 1023, "presto_build_tree: budget=%d outside 1..1023",
            d.budget);
    REQUIRE(d.depth <= tree_max_depth(d.k),
            "presto_build_tree: depth %d exceeds the rank-path key (at most %d for k=%d)", d.depth,
            tree_max_depth(d.k), d.k);
    REQUIRE(d.mode == PRESTO_TREE_BEST_FIRST || d.mode == PRESTO_TREE_BEST_FIRST_ALG2 ||
                d.mode == PRESTO_TREE_BEAM,
            "presto_build_tree: unknown mode %d", d.mode);
    const int beam_width = d.mode == PRESTO_TREE_BEAM ? d.beam_width : 0;
    if (d.mode == PRESTO_TREE_BEAM) {
        REQUIRE(d.beam_width >= 1 && d.beam_width <= 64,
                "presto_build_tree: beam_width=%d outside 1..64", d.beam_width);
        REQUIRE(d.beam_width * d.k <= 256, "presto_build_tree: beam_width * k = %d exceeds 256",
                d.beam_width * d.k);
    }
    if (!tree_build_fits(d.depth, d.k, d.branch, d.budget + 1, beam_width,
                         d.mode == PRESTO_TREE_BEST_FIRST_ALG2))
        return set_error(PRESTO_ERR_UNSUPPORTED, "presto_build_tree: tables exceed 160 KiB of LDS");
    if (d.batch == 0) return PRESTO_OK;
    REQUIRE(ids && logprob && lambda && root_token && n_nodes && parent && token && depth_out &&
                rank && score && anc,
            "presto_build_tree: null pointer");
    return launch_build_tree(&d, ids, logprob, log_rho, lambda, root_token, n_nodes, parent, token,
                             depth_out, rank, score, anc, stream);
}

size_t presto_tree_attention_workspace(const presto_attn_desc* desc) {
    if (!desc || desc->batch <= 0 || desc->n_max <= 0 || desc->hkv <= 0 || desc->hq <= 0 ||
        desc->hq % desc->hkv != 0 || desc->max_ctx < 0 || desc->total_ctx < 0)
        return 0;
    return attn_workspace_bytes(desc);
}

presto_status presto_tree_attention(const presto_attn_desc* desc, const void* q,
                                    const void* k_cache, const void* v_cache,
                                    const int32_t* ctx_offsets, const void* k_tree,
                                    const void* v_tree, const uint64_t* anc,
                                    const int32_t* n_nodes, void* out, void* ws, size_t ws_bytes,
                                    hipStream_t stream) {
    g_err[0] = 0;
    REQUIRE(desc, "presto_tree_attention: null descriptor");
    const presto_attn_desc d = *desc;
    REQUIRE(valid_dtype(d.dt), "presto_tree_attention: unknown dtype %d", (int)d.dt);
    REQUIRE(d.batch >= 0, "presto_tree_attention: batch < 0");
    REQUIRE(d.n_max >= 1 && d.n_max <= 1024, "presto_tree_attention: n_max outside 1..1024");
    REQUIRE(d.hq >= 1 && d.hkv >= 1 && d.hq % d.hkv == 0,
            "presto_tree_attention: hq must be a positive multiple of hkv");
    REQUIRE(d.head_dim == 64 || d.head_dim == 128, "presto_tree_attention: head_dim %d",
            d.head_dim);
    REQUIRE(d.max_ctx >= 0, "presto_tree_attention: max_ctx < 0");
    REQUIRE(d.total_ctx >= 0, "presto_tree_attention: total_ctx < 0");
    REQUIRE(d.ctx_layout == PRESTO_CTX_PACKED || d.ctx_layout == PRESTO_CTX_SLOTS,
            "presto_tree_attention: unknown ctx_layout %d", d.ctx_layout);
    REQUIRE(isfinite(d.scale) && d.scale > 0.f, "presto_tree_attention: scale must be positive");
    REQUIRE((int64_t)d.max_ctx + d.n_max < ((int64_t)1 << 30), "presto_tree_attention: too long");
    if (d.batch == 0) return PRESTO_OK;
    REQUIRE(q && k_tree && v_tree && ctx_offsets && anc && n_nodes && out,
            "presto_tree_attention: null pointer");
    REQUIRE(d.max_ctx == 0 || (k_cache && v_cache), "presto_tree_attention: null cache");
    if (d.dt == PRESTO_DT_BF16) {
        const uintptr_t al = (uintptr_t)q | (uintptr_t)k_tree | (uintptr_t)v_tree |
                             (uintptr_t)out | (uintptr_t)(k_cache ? k_cache : q) |
                             (uintptr_t)(v_cache ? v_cache : q);
        REQUIRE(al % 16 == 0, "presto_tree_attention: bf16 tensors must be 16-byte aligned");
    }
    presto_status st = check_ws(ws, ws_bytes, presto_tree_attention_workspace(&d));
    if (st != PRESTO_OK) return st;
    return launch_tree_attention(&d, q, k_cache, v_cache, ctx_offsets, k_tree, v_tree, anc, n_nodes,
                                 out, ws, stream);
}

size_t presto_accept_workspace(int32_t batch, int32_t n_max, int32_t vocab) {
    if (batch <= 0 || n_max <= 0 || vocab <= 0) return 0;
    return accept_workspace_bytes(batch, n_max, vocab);
}

presto_status presto_accept(presto_dtype dt, const void* target_logits, int32_t vocab,
                            int64_t row_stride, int32_t batch, int32_t n_max, int32_t depth,
                            const int32_t* parent, const int32_t* token, const int32_t* n_nodes,
                            int32_t* accept_len, int32_t* path, int32_t* bonus,
                            int32_t* target_argmax, int32_t* flags, void* ws, size_t ws_bytes,
                            hipStream_t stream) {
    g_err[0] = 0;
    REQUIRE(valid_dtype(dt), "presto_accept: unknown dtype %d", (int)dt);
    REQUIRE(vocab >= 1, "presto_accept: vocab < 1");
    REQUIRE(row_stride >= vocab, "presto_accept: row_stride < vocab");
    REQUIRE(batch >= 0, "presto_accept: batch < 0");
    REQUIRE(n_max >= 1 && n_max <= 1024, "presto_accept: n_max outside 1..1024");
    REQUIRE(depth >= 1 && depth <= 1024, "presto_accept: depth outside 1..1024");
    if (batch == 0) return PRESTO_OK;
    REQUIRE(target_logits && parent && token && n_nodes && accept_len && path && bonus,
            "presto_accept: null pointer");
    REQUIRE((int64_t)batch * n_max * ((vocab + 1023) / 1024) < ((int64_t)1 << 31),
            "presto_accept: too many rows");
    presto_status st = check_ws(ws, ws_bytes, presto_accept_workspace(batch, n_max, vocab));
    if (st != PRESTO_OK) return st;
    return launch_accept(dt == PRESTO_DT_BF16, target_logits, vocab, row_stride, batch, n_max, depth,
                         parent, token, n_nodes, accept_len, path, bonus, target_argmax, flags, ws,
                         stream);
}

presto_status presto_commit_kv(const presto_commit_desc* desc, const void* k_tree,
                               const void* v_tree, const int32_t* path, const int32_t* accept_len,
                               void* k_cache, void* v_cache, int64_t cache_rows, int32_t* ctx,
                               const int32_t* ctx_cap, int32_t* flags, hipStream_t stream) {
    g_err[0] = 0;
    REQUIRE(desc, "presto_commit_kv: null descriptor");
    const presto_commit_desc d = *desc;
    REQUIRE(valid_dtype(d.dt), "presto_commit_kv: unknown dtype %d", (int)d.dt);
    REQUIRE(d.batch >= 0, "presto_commit_kv: batch < 0");
    REQUIRE(d.n_max >= 1 && d.n_max <= 1024, "presto_commit_kv: n_max outside 1..1024");
    REQUIRE(d.depth >= 1 && d.depth <= 1024, "presto_commit_kv: depth outside 1..1024");
    REQUIRE(d.hkv >= 1 && (d.head_dim == 64 || d.head_dim == 128),
            "presto_commit_kv: hkv >= 1 and head_dim in {64, 128}");
    REQUIRE(cache_rows >= 0, "presto_commit_kv: cache_rows < 0");
    if (d.batch == 0) return PRESTO_OK;
    REQUIRE(k_tree && v_tree && path && accept_len && k_cache && v_cache && ctx && ctx_cap,
            "presto_commit_kv: null pointer");
    const uintptr_t al = (uintptr_t)k_tree | (uintptr_t)v_tree | (uintptr_t)k_cache |
                         (uintptr_t)v_cache;
    REQUIRE(al % 16 == 0, "presto_commit_kv: K/V tensors must be 16-byte aligned");
    return launch_commit_kv(&d, k_tree, v_tree, path, accept_len, k_cache, v_cache, cache_rows,
                            ctx, ctx_cap, flags, stream);
}

presto_status presto_select_slots(int32_t batch, int32_t n_max, int32_t depth, int32_t slots,
                                  int32_t first_slot, const int32_t* path,
                                  const int32_t* accept_len, int64_t* row_index, int32_t* flags,
                                  hipStream_t stream) {
    g_err[0] = 0;
    REQUIRE(batch >= 0, "presto_select_slots: batch < 0");
    REQUIRE(n_max >= 1 && n_max <= 1024, "presto_select_slots: n_max outside 1..1024");
    REQUIRE(depth >= 1, "presto_select_slots: depth < 1");
    REQUIRE(slots >= 1 && slots <= 64, "presto_select_slots: slots outside 1..64");
    REQUIRE(first_slot >= 0 && first_slot < slots,
            "presto_select_slots: first_slot outside 0..slots-1");
    if (batch == 0) return PRESTO_OK;
    REQUIRE(path && accept_len && row_index, "presto_select_slots: null pointer");
    return launch_select_slots(batch, n_max, depth, slots, first_slot, path, accept_len, row_index,
                               flags, stream);
}

presto_status presto_flatten_slots(int32_t batch, int32_t n_max, int32_t slots,
                                   const int32_t* depth, const uint64_t* anc,
                                   const int32_t* n_nodes, const int32_t* root_pos,
                                   int32_t* pos_out, uint64_t* anc_out, int32_t* n_rows,
                                   hipStream_t stream) {
    g_err[0] = 0;
    REQUIRE(batch >= 0, "presto_flatten_slots: batch < 0");
    REQUIRE(n_max >= 1 && n_max <= 1024, "presto_flatten_slots: n_max outside 1..1024");
    REQUIRE(slots >= 1 && slots <= 64, "presto_flatten_slots: slots outside 1..64");
    REQUIRE((int64_t)n_max * (1 + slots) <= 65536, "presto_flatten_slots: more than 65536 rows");
    if (batch == 0) return PRESTO_OK;
    REQUIRE(depth && anc && n_nodes && root_pos && pos_out && anc_out && n_rows,
            "presto_flatten_slots: null pointer");
    return launch_flatten_slots(batch, n_max, slots, depth, anc, n_nodes, root_pos, pos_out,
                                anc_out, n_rows, stream);
}

const char* presto_status_string(presto_status s) {
    switch (s) {
        case PRESTO_OK: return "ok";
        case PRESTO_ERR_INVALID_ARG: return "invalid argument";
        case PRESTO_ERR_UNSUPPORTED: return "unsupported";
        case PRESTO_ERR_WORKSPACE: return "workspace too small";
        case PRESTO_ERR_HIP: return "HIP error";
        default: break;
    }
    return "unknown status";
}

const char* presto_last_error(void) { return g_err; }

const char* presto_version(void) { return "presto-mi355x 0.1 (gfx950)"; }

}  // extern "C"
