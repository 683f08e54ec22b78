"""PRESTO draft-to-verify round on MI355X (gfx950).

The four stages of a round run in the HIP kernels of ``libpresto.so``
(C ABI declared in ``include/presto.h``); this package holds those sources
(``csrc/``), their build (``build.py``) and a thin ctypes binding whose
functions carry the C names.
"""
from ._lib import (  # noqa: F401
    EXPORTS, PRESTO_DT_BF16, PRESTO_DT_F32, PRESTO_ERR_HIP, PRESTO_ERR_INVALID_ARG,
    PRESTO_ERR_UNSUPPORTED, PRESTO_ERR_WORKSPACE, PRESTO_FLAG_NAN_DRAFTER, PRESTO_FLAG_NAN_TARGET,
    PRESTO_FLAG_NGRAM_BAD, PRESTO_FLAG_NGRAM_FULL, PRESTO_FLAG_BAD_INDEX, PRESTO_FLAG_KV_COMMIT,
    PRESTO_CTX_PACKED, PRESTO_CTX_SLOTS, CommitDesc, presto_commit_kv, presto_flatten_slots,
    presto_select_slots, presto_topk_rows,
    PRESTO_OK, PRESTO_TREE_BEAM, PRESTO_TREE_BEST_FIRST, PRESTO_TREE_BEST_FIRST_ALG2, AttnDesc,
    PrestoError, TreeDesc, lib, presto_accept, presto_build_tree, presto_entropy_lambda, presto_ngram_clear,
    presto_ngram_gather, presto_ngram_insert, presto_ngram_table_bytes, presto_topk,
    presto_topk_noalloc,
    presto_tree_attention, topk_fallback_chunks, topk_workspace, version,
)
