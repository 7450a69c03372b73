"""fastrl_token_logprob_noalloc (the allocation-free variant with the library's fixed
scratch) against fastrl_token_logprob (caller workspace), through the C ABI: the results are
the same bit for bit, on two calls in a row, the second smaller than the first; the first
needs several chunks of the fixed scratch at the 7B vocabulary."""
import ctypes

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module")
def fr():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_36932_amd as m
    return m


def _case(seed, T_rows, d, V, dtype):
    g = torch.Generator().manual_seed(seed)
    H = torch.randn(T_rows, d, generator=g).to(dtype)
    W = (0.02 * torch.randn(V, d, generator=g)).to(dtype)
    y = torch.randint(0, V, (T_rows,), generator=g, dtype=torch.int32)
    rows = torch.randperm(T_rows, generator=g)[: (3 * T_rows) // 4].to(torch.int32)
    return H.to(DEV), W.to(DEV), y.to(DEV), rows.to(DEV)


def _both(fr, H, W, y, rows):
    T = rows.numel()
    st = torch.zeros(1, dtype=torch.int32, device=DEV)
    lp_ref, lse_ref = fr.token_logprob(H, W, y, row_index=rows, status=st)
    lp = torch.full((T,), float("nan"), device=DEV)
    lse = torch.full((T,), float("nan"), device=DEV)
    fr.token_logprob_noalloc(H, W, y, lp, lse, row_index=rows, status=st)
    torch.cuda.synchronize()
    assert st.item() == 0, fr.status_names(st.item())
    return lp, lse, lp_ref, lse_ref


def test_noalloc_matches_workspace_entry_point(fr):
    V, d = 152064, 256
    chunk = fr._lib.fastrl_token_logprob_noalloc_max_chunk(V)
    assert 256 <= chunk < 20000
    # first call: more tokens than one chunk of the fixed scratch
    H, W, y, rows = _case(1, 40000, d, V, torch.bfloat16)
    assert rows.numel() > 2 * chunk
    lp, lse, lp_ref, lse_ref = _both(fr, H, W, y, rows)
    assert torch.isfinite(lp).all() and torch.equal(lp, lp_ref) and torch.equal(lse, lse_ref)
    # second call, smaller (another vocabulary, fewer tokens, float32): the scratch keeps the
    # first call's contents, which must not leak into the result
    H, W, y, rows = _case(2, 700, 64, 5000, torch.float32)
    lp, lse, lp_ref, lse_ref = _both(fr, H, W, y, rows)
    assert torch.isfinite(lp).all() and torch.equal(lp, lp_ref) and torch.equal(lse, lse_ref)


def test_noalloc_rejects_and_accepts(fr):
    L = fr._lib
    assert L.fastrl_token_logprob_noalloc_scratch_bytes() == 64 << 20
    # a vocabulary whose partials for 256 tokens exceed the scratch: refused, nothing enqueued
    assert L.fastrl_token_logprob_noalloc(ctypes.c_void_p(256), None, ctypes.c_void_p(256), 1,
                                          10, 64, 9_000_000, ctypes.c_void_p(256),
                                          ctypes.c_void_p(256), None, None, None) == -2
    assert b"fixed scratch" in L.fastrl_last_error()
    # T = 0 succeeds without touching the outputs
    H, W, y, rows = _case(3, 16, 64, 300, torch.bfloat16)
    lp = torch.full((1,), 7.0, device=DEV)
    fr.token_logprob_noalloc(H, W, y, lp, None, row_index=rows, T=0)
    torch.cuda.synchronize()
    assert lp.item() == 7.0
