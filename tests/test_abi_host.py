"""Host-only checks of the C ABI (no GPU): the library loads, exports every
entry point declared in include/presto.h, sizes workspaces, and rejects bad
arguments before launching anything."""
import ctypes
import os
import re

import pytest

import paper_2607_22634_amd as P

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    text = open(os.path.join(ROOT, "include", "presto.h")).read()
    return sorted(set(re.findall(r"\b(presto_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = P.lib()
    names = _declared()
    assert set(names) == set(P.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings_and_version():
    lib = P.lib()
    assert lib.presto_status_string(0) == b"ok"
    assert lib.presto_status_string(-3) == b"workspace too small"
    assert b"gfx950" in lib.presto_version()


def test_workspace_sizes_are_deterministic_and_monotone():
    lib = P.lib()
    a = lib.presto_topk_workspace(16, 151936, 4)
    assert a > 0 and a == lib.presto_topk_workspace(16, 151936, 4)
    assert lib.presto_topk_workspace(32, 151936, 4) > a
    assert lib.presto_topk_workspace(0, 151936, 4) == 0
    assert lib.presto_accept_workspace(1, 65, 151936) > 0
    d = P.AttnDesc(4, 257, 32, 8, 128, 32768, 0.088, P.PRESTO_DT_BF16)
    assert lib.presto_tree_attention_workspace(ctypes.byref(d)) > 0
    d1 = P.AttnDesc(32, 129, 32, 8, 128, 2048, 0.088, P.PRESTO_DT_BF16)
    assert lib.presto_tree_attention_workspace(ctypes.byref(d1)) == 0  # fills the chip unsplit


def _err(status):
    return status, P.lib().presto_last_error().decode()


def test_topk_rejects_bad_arguments():
    lib = P.lib()
    st, msg = _err(lib.presto_topk(0, None, 4, 1024, 1024, 0, None, None, None, None, None, None, 0, None))
    assert st == P.PRESTO_ERR_INVALID_ARG and "k=0" in msg
    st, _ = _err(lib.presto_topk(0, None, 4, 1024, 1000, 2, None, None, None, None, None, None, 0, None))
    assert st == P.PRESTO_ERR_INVALID_ARG
    st, _ = _err(lib.presto_topk(7, None, 4, 1024, 1024, 2, None, None, None, None, None, None, 0, None))
    assert st == P.PRESTO_ERR_INVALID_ARG
    st, _ = _err(lib.presto_topk(0, None, 4, 1024, 1024, 17, None, None, None, None, None, None, 0, None))
    assert st == P.PRESTO_ERR_UNSUPPORTED
    st, _ = _err(lib.presto_topk(0, None, 4, 1024, 1024, 2, None, None, None, None, None, None, 0, None))
    assert st == P.PRESTO_ERR_INVALID_ARG  # null pointers
    # zero rows is a no-op, even without pointers
    assert lib.presto_topk(0, None, 0, 1024, 1024, 2, None, None, None, None, None, None, 0, None) == 0


def test_entropy_lambda_rejects_bad_arguments():
    lib = P.lib()
    fake = ctypes.c_void_p(0x1000)  # never dereferenced: the checks fail first
    for beta, c in [(0.0, 1.0), (-1.0, 1.0), (1.0, 0.0), (float("nan"), 1.0), (1.0, float("inf"))]:
        st, msg = _err(lib.presto_entropy_lambda(4, fake, beta, c, fake, None))
        assert st == P.PRESTO_ERR_INVALID_ARG and ("beta" in msg or "C" in msg)
    st, _ = _err(lib.presto_entropy_lambda(4, None, 1.0, 1.0, None, None))
    assert st == P.PRESTO_ERR_INVALID_ARG
    st, _ = _err(lib.presto_entropy_lambda(-1, fake, 1.0, 1.0, fake, None))
    assert st == P.PRESTO_ERR_INVALID_ARG
    assert lib.presto_entropy_lambda(0, None, 1.0, 1.0, None, None) == P.PRESTO_OK


def test_topk_rejects_small_workspace():
    lib = P.lib()
    fake = ctypes.c_void_p(0x1000)  # never dereferenced: the check fails first
    st, msg = _err(lib.presto_topk(0, fake, 4, 1024, 1024, 2, fake, fake, None, None, None, fake, 8, None))
    assert st == P.PRESTO_ERR_WORKSPACE and "workspace" in msg


@pytest.mark.parametrize("field,value", [("depth", 0), ("depth", 33), ("k", 0), ("k", 17),
                                         ("branch", 5), ("budget", 0), ("budget", 1024),
                                         ("mode", 9)])
def test_build_tree_rejects_bad_descriptor(field, value):
    d = P.TreeDesc(1, 4, 4, 4, 8, 0)
    setattr(d, field, value)
    st, _ = _err(P.lib().presto_build_tree(ctypes.byref(d), *([None] * 13), 0, None))
    assert st == P.PRESTO_ERR_INVALID_ARG


@pytest.mark.parametrize("mode", [0, 1, 2])
def test_build_tree_accepts_budget_1023(mode):
    # the largest budget (N = 1024 rows) with the paper's k = 10, depth 16 and
    # beam width 10; batch 0: validated, nothing launched
    d = P.TreeDesc(0, 16, 10, 10, 1023, mode, 10)
    st, msg = _err(P.lib().presto_build_tree(ctypes.byref(d), *([None] * 13), 0, None))
    assert st == P.PRESTO_OK, msg
    d = P.TreeDesc(0, 24, 16, 16, 1023, mode, 16)
    st, msg = _err(P.lib().presto_build_tree(ctypes.byref(d), *([None] * 13), 0, None))
    assert st == P.PRESTO_OK, msg


def test_build_tree_accepts_every_mode():
    # batch 0: validated, nothing launched (no device needed)
    for mode in (P.PRESTO_TREE_BEST_FIRST, P.PRESTO_TREE_BEST_FIRST_ALG2, P.PRESTO_TREE_BEAM):
        d = P.TreeDesc(0, 4, 4, 4, 8, mode, 4)
        st, msg = _err(P.lib().presto_build_tree(ctypes.byref(d), *([None] * 13), 0, None))
        assert st == P.PRESTO_OK, msg


@pytest.mark.parametrize("width,k", [(0, 4), (65, 1), (33, 8)])
def test_build_tree_rejects_bad_beam_width(width, k):
    d = P.TreeDesc(1, 4, k, k, 8, P.PRESTO_TREE_BEAM, width)
    st, msg = _err(P.lib().presto_build_tree(ctypes.byref(d), *([None] * 13), 0, None))
    assert st == P.PRESTO_ERR_INVALID_ARG and "beam_width" in msg


def test_build_tree_path_key_limit():
    d = P.TreeDesc(1, 25, 16, 16, 8, 0)  # 5-bit digits: six per 32-bit word, 24 levels
    st, msg = _err(P.lib().presto_build_tree(ctypes.byref(d), *([None] * 13), 0, None))
    assert st == P.PRESTO_ERR_INVALID_ARG and "24" in msg


@pytest.mark.parametrize("field,value", [("head_dim", 96), ("hkv", 3), ("n_max", 0),
                                         ("n_max", 1025), ("max_ctx", -1), ("dt", 5)])
def test_attention_rejects_bad_descriptor(field, value):
    d = P.AttnDesc(1, 9, 2, 1, 64, 128, 0.125, P.PRESTO_DT_F32)
    setattr(d, field, value)
    st, _ = _err(P.lib().presto_tree_attention(ctypes.byref(d), *([None] * 10), 0, None))
    assert st == P.PRESTO_ERR_INVALID_ARG


def test_accept_rejects_bad_arguments():
    lib = P.lib()
    args = [None] * 9
    assert lib.presto_accept(0, None, 1024, 1000, 1, 9, 4, *args, 0, None) == P.PRESTO_ERR_INVALID_ARG
    assert lib.presto_accept(0, None, 1024, 1024, 1, 0, 4, *args, 0, None) == P.PRESTO_ERR_INVALID_ARG
    assert lib.presto_accept(0, None, 1024, 1024, 1, 9, 0, *args, 0, None) == P.PRESTO_ERR_INVALID_ARG
    assert lib.presto_accept(0, None, 1024, 1024, 1, 9, 4, *args, 0, None) == P.PRESTO_ERR_INVALID_ARG
    assert lib.presto_accept(0, None, 1024, 1024, 0, 9, 4, *args, 0, None) == P.PRESTO_OK
    # depth bounds the pointer-jumping rounds and the path rows: at most 1024
    st, msg = _err(lib.presto_accept(0, None, 1024, 1024, 0, 9, 1025, *args, 0, None))
    assert st == P.PRESTO_ERR_INVALID_ARG and "depth" in msg
    assert lib.presto_accept(0, None, 1024, 1024, 0, 9, 1024, *args, 0, None) == P.PRESTO_OK


def test_commit_kv_rejects_bad_descriptor():
    lib = P.lib()
    for field, value in [("depth", 0), ("depth", 1025), ("n_max", 1025), ("head_dim", 96),
                         ("hkv", 0), ("dt", 4)]:
        d = P.CommitDesc(1, 65, 8, 128, 16, P.PRESTO_DT_BF16)
        setattr(d, field, value)
        st, _ = _err(lib.presto_commit_kv(ctypes.byref(d), *([None] * 6), 0, None, None, None,
                                          None))
        assert st == P.PRESTO_ERR_INVALID_ARG, (field, value)
    d = P.CommitDesc(0, 1024, 8, 128, 1024, P.PRESTO_DT_BF16)  # the largest path; batch 0
    assert lib.presto_commit_kv(ctypes.byref(d), *([None] * 6), 0, None, None, None,
                                None) == P.PRESTO_OK


def test_ngram_entry_points_validate_on_the_host():
    lib = P.lib()
    fake = ctypes.c_void_p(0x1000)  # never dereferenced: the checks fail first
    assert lib.presto_ngram_table_bytes(1024) == 1024 * 12
    for bad_cap in (0, 32, 100, 3 << 20):
        assert lib.presto_ngram_table_bytes(bad_cap) == 0
        st, msg = _err(lib.presto_ngram_clear(fake, bad_cap, None))
        assert st == P.PRESTO_ERR_INVALID_ARG and "capacity" in msg
    st, _ = _err(lib.presto_ngram_clear(None, 1024, None))
    assert st == P.PRESTO_ERR_INVALID_ARG
    st, _ = _err(lib.presto_ngram_insert(fake, 1024, -1, fake, fake, fake, fake, None, None))
    assert st == P.PRESTO_ERR_INVALID_ARG
    assert lib.presto_ngram_insert(None, 1024, 0, None, None, None, None, None, None) == P.PRESTO_OK
    g = lib.presto_ngram_gather
    for floor, depth, k in [(0.5, 4, 4), (float("nan"), 4, 4), (-1.0, 0, 4), (-1.0, 33, 4),
                            (-1.0, 4, 0), (-1.0, 4, 17)]:
        st, _ = _err(g(fake, 1024, floor, 1, depth, k, fake, fake, fake, fake, None))
        assert st == P.PRESTO_ERR_INVALID_ARG, (floor, depth, k)
    st, _ = _err(g(ctypes.c_void_p(0x1004), 1024, -1.0, 1, 4, 4, fake, fake, fake, fake, None))
    assert st == P.PRESTO_ERR_INVALID_ARG  # misaligned table
    assert g(None, 1024, -1.0, 0, 4, 4, None, None, None, None, None) == P.PRESTO_OK
