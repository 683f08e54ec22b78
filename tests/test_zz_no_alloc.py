"""presto_topk_noalloc (top-k for callers that cannot allocate: its partials
live in the library's static per-GPU scratch) against presto_topk with a
caller workspace: identical ids, log q and LSE (and entropy), bit for bit,
on two calls in a row, the second with a smaller input; a request larger
than the scratch is refused on the host with nothing launched."""
import ctypes

import numpy as np
import pytest
import torch

import paper_2607_22634_amd as P
import synthetic as sy
from gpu_util import round_data, to_dev

pytestmark = pytest.mark.gpu


def _same(a, b):
    for x, y in zip(a, b):
        assert torch.equal(x.view(torch.int32), y.view(torch.int32))


def test_topk_noalloc_matches_workspace_entry_point():
    w, rin = round_data(5)  # 1024 drafter rows of vocabulary 151936, bf16
    logits = to_dev(rin["drafter_logits"], w.dtype)
    big = P.presto_topk_noalloc(logits, w.k, entropy=True)
    ref = P.presto_topk(logits, w.k, entropy=True)
    torch.cuda.synchronize()
    _same(big, ref)
    # a smaller second call (fewer rows, larger k) reuses the scratch
    small_logits = logits[37:58]
    small = P.presto_topk_noalloc(small_logits, 10)
    ref_small = P.presto_topk(small_logits, 10)
    torch.cuda.synchronize()
    _same(small, ref_small)


def test_topk_noalloc_fp32_and_ragged_rows():
    rng = np.random.default_rng(4)
    x = (rng.standard_normal((7, 4099)) * 3).astype(np.float32)
    x[2, :] = 1.0  # a tie flood: the exact pass
    t = to_dev(sy.cast(x, "f32"))
    _same(P.presto_topk_noalloc(t, 16), P.presto_topk(t, 16))
    torch.cuda.synchronize()


def test_topk_noalloc_refuses_more_than_the_scratch():
    lib = P.lib()
    fake = ctypes.c_void_p(0x1000)  # never dereferenced: the size check fails first
    rows, V, k = 4096, 151936, 16
    assert lib.presto_topk_workspace(rows, V, k) > (16 << 20)
    st = lib.presto_topk_noalloc(P.PRESTO_DT_BF16, fake, rows, V, V, k, fake, fake, None, None,
                                 None, None)
    assert st == P.PRESTO_ERR_WORKSPACE
    assert b"scratch" in lib.presto_last_error()
