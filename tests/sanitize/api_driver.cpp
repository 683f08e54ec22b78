// Sanitizer driver for the host side of libpresto: the library's sources are
// compiled for the host only, under AddressSanitizer and
// UndefinedBehaviorSanitizer (no recovery), and this program calls every
// entry point with arguments that the host checks reject (or that launch
// nothing: empty batches), plus the workspace-size queries at their
// extremes.  No GPU is needed and no kernel is launched.  Exit status 0
// means every expected status came back and no sanitizer report fired.
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "presto.h"

static int failures = 0;

static void expect(presto_status got, presto_status want, const char* what) {
    const char* msg = presto_last_error();
    if (got != want || strlen(msg) >= 512) {
        fprintf(stderr, "%s: status %d, expected %d (%s)\n", what, (int)got, (int)want, msg);
        ++failures;
    }
}

int main() {
    void* fake = reinterpret_cast<void*>(0x1000);  // never dereferenced: the checks fail first
    int32_t* fi = static_cast<int32_t*>(fake);
    float* ff = static_cast<float*>(fake);
    const int64_t big = (int64_t)1 << 62;

    // top-k: bad k, dtype, stride, row counts (also far beyond any device)
    expect(presto_topk(PRESTO_DT_BF16, fake, 4, 1024, 1024, 0, fi, ff, 0, 0, 0, fake, 1 << 20, 0),
           PRESTO_ERR_INVALID_ARG, "topk k=0");
    expect(presto_topk((presto_dtype)7, fake, 4, 1024, 1024, 2, fi, ff, 0, 0, 0, fake, 1 << 20, 0),
           PRESTO_ERR_INVALID_ARG, "topk dtype");
    expect(presto_topk(PRESTO_DT_BF16, fake, big, 151936, 151936, 4, fi, ff, 0, 0, 0, fake, 8, 0),
           PRESTO_ERR_INVALID_ARG, "topk 2^62 rows");
    expect(presto_topk(PRESTO_DT_F32, fake, 4, 1024, 1024, 2, fi, ff, 0, 0, 0, fake, 8, 0),
           PRESTO_ERR_WORKSPACE, "topk workspace");
    expect(presto_topk_noalloc(PRESTO_DT_BF16, fake, big, 151936, 151936, 4, fi, ff, 0, 0, 0, 0),
           PRESTO_ERR_INVALID_ARG, "topk_noalloc 2^62 rows");
    expect(presto_topk_noalloc(PRESTO_DT_BF16, fake, 4096, 151936, 151936, 16, fi, ff, 0, 0, 0, 0),
           PRESTO_ERR_WORKSPACE, "topk_noalloc beyond the scratch");
    expect(presto_topk_rows(PRESTO_DT_BF16, fake, 0, (const int64_t*)fake, 3, 64, 64, 2, fi, ff, 0,
                            0, 0, fake, 1 << 20, 0),
           PRESTO_ERR_INVALID_ARG, "topk_rows no logits rows");
    if (presto_topk_workspace(big, 151936, 16) != 0 || presto_topk_workspace(4, 151936, 4) == 0) {
        fprintf(stderr, "topk workspace sizes\n");
        ++failures;
    }
    presto_topk_workspace(-5, 151936, 4);
    expect(presto_entropy_lambda(4, ff, 0.f, 1.f, ff, 0), PRESTO_ERR_INVALID_ARG, "lambda beta");

    // n-gram table
    expect(presto_ngram_clear(fake, 100, 0), PRESTO_ERR_INVALID_ARG, "ngram capacity");
    expect(presto_ngram_insert(fake, 1024, big, fi, fi, fi, ff, 0, 0), PRESTO_ERR_INVALID_ARG,
           "ngram n");
    expect(presto_ngram_gather(fake, 1024, -1.f, 1, 33, 4, fi, fi, fi, ff, 0),
           PRESTO_ERR_INVALID_ARG, "ngram depth");
    if (presto_ngram_table_bytes((int64_t)1 << 40) != 0) ++failures;

    // tree build: every descriptor field out of range, the largest valid trees
    presto_tree_desc d = {1, 16, 10, 10, 1023, PRESTO_TREE_BEAM, 10, 0};
    presto_tree_desc bad[] = {d, d, d, d, d, d, d};
    bad[0].depth = 0; bad[1].k = 17; bad[2].branch = 11; bad[3].budget = 1024;
    bad[4].mode = 9; bad[5].beam_width = 65; bad[6].depth = 25; bad[6].k = 16;
    for (auto& b : bad)
        expect(presto_build_tree(&b, fi, ff, ff, ff, fi, fi, fi, fi, fi, fi, ff,
                                 (uint64_t*)fake, 0, 0, 0),
               PRESTO_ERR_INVALID_ARG, "tree descriptor");
    for (int mode = 0; mode < 3; ++mode) {
        presto_tree_desc e = {0, 24, 16, 16, 1023, mode, 16, 0};
        expect(presto_build_tree(&e, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0), PRESTO_OK,
               "tree batch 0");
        presto_build_tree_workspace(&e);
    }
    expect(presto_build_tree(nullptr, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0),
           PRESTO_ERR_INVALID_ARG, "tree null descriptor");

    // attention: descriptor checks and workspace sizes at the extremes
    presto_attn_desc a = {4, 257, 32, 8, 128, 32768, 0.088f, PRESTO_DT_BF16, PRESTO_CTX_PACKED, 0};
    presto_attn_desc ab[] = {a, a, a, a, a, a};
    ab[0].head_dim = 96; ab[1].hkv = 3; ab[2].n_max = 1025; ab[3].max_ctx = -1;
    ab[4].scale = -1.f; ab[5].max_ctx = (1 << 30) - 1;
    for (auto& b : ab)
        expect(presto_tree_attention(&b, fake, fake, fake, fi, fake, fake, (const uint64_t*)fake,
                                     fi, fake, fake, (size_t)1 << 40, 0),
               PRESTO_ERR_INVALID_ARG, "attention descriptor");
    presto_attn_desc huge = {1 << 20, 1024, 64, 8, 128, (1 << 30) - 2048, 0.088f, PRESTO_DT_BF16,
                             PRESTO_CTX_PACKED, (int64_t)1 << 40};
    presto_tree_attention_workspace(&huge);
    presto_tree_attention_workspace(&a);
    a.batch = 0;
    expect(presto_tree_attention(&a, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0), PRESTO_OK,
           "attention batch 0");

    // accept and bookkeeping
    expect(presto_accept(PRESTO_DT_BF16, fake, 151936, 151936, 1, 65, 1025, fi, fi, fi, fi, fi, fi,
                         0, 0, fake, 1 << 30, 0),
           PRESTO_ERR_INVALID_ARG, "accept depth");
    expect(presto_accept(PRESTO_DT_BF16, fake, 151936, 151936, 1 << 30, 1024, 16, fi, fi, fi, fi,
                         fi, fi, 0, 0, fake, 1 << 30, 0),
           PRESTO_ERR_INVALID_ARG, "accept rows");
    presto_accept_workspace(1 << 30, 1024, 151936);
    presto_commit_desc c = {1, 65, 8, 128, 1025, PRESTO_DT_BF16};
    expect(presto_commit_kv(&c, fake, fake, fi, fi, fake, fake, 100, fi, fi, 0, 0),
           PRESTO_ERR_INVALID_ARG, "commit depth");
    expect(presto_select_slots(1, 65, 16, 65, 0, fi, fi, (int64_t*)fake, 0, 0),
           PRESTO_ERR_INVALID_ARG, "select slots");
    expect(presto_flatten_slots(1, 1024, 64, fi, (const uint64_t*)fake, fi, fi, fi,
                                (uint64_t*)fake, fi, 0),
           PRESTO_ERR_INVALID_ARG, "flatten rows");
    for (int s = -5; s <= 0; ++s) presto_status_string((presto_status)s);
    presto_version();

    if (failures) {
        fprintf(stderr, "%d failure(s)\n", failures);
        return 1;
    }
    printf("api driver: ok\n");
    return 0;
}
