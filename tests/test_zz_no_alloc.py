"""dls_draft_block_noalloc (the library's per-GPU scratch array instead of a workspace) against
dls_draft_block with a workspace: bit-identical tokens and statistics on two calls in a row, the
second with a smaller input, on the persistent kernel (wide, then narrow) and on the
per-position launches; a call that fails does not affect the next one."""
import numpy as np
import pytest
import torch

from paper_2607_07409_amd import binding as B
from paper_2607_07409_amd import workloads as W

pytestmark = pytest.mark.gpu


def _inputs(name, seed=None, **shape):
    wl = W.WORKLOADS[name]
    if shape:
        wl = wl.with_(**shape)
    hw = W.make_head(wl, "stress", seed=seed)
    head = B.LocalHead.from_weights(hw)
    lt = B.as_tensor(W.make_long_logits(wl))
    last = torch.from_numpy(W.make_last_token(wl)).cuda()
    return wl, head, lt, last


def _both(head, lt, last, alpha=0.5):
    ref_tok, ref_st = B.draft_block(head, lt, last, None, 1.0, alpha, 0.0)
    tok, st = B.draft_block_noalloc(head, lt, last, None, 1.0, alpha, 0.0)
    torch.cuda.synchronize()
    assert B.workspace_error(None) == 0
    assert torch.equal(tok, ref_tok)
    assert torch.equal(st.view(torch.int32), ref_st.view(torch.int32))
    return tok


def test_noalloc_matches_workspace_entry_point():
    # call 1: the batch-16 Qwen3-8B-shaped workload (wide persistent kernel, full vocabulary)
    wl, head, lt, last = _inputs("qwen3-8b-b16")
    head.prepare()
    assert head.path(wl.batch, wl.B, lt.dtype, False) == 1
    t1 = _both(head, lt, last)
    assert bool((t1 >= 0).all().item())
    del head
    # call 2, smaller: batch 3, 7 positions, V = 5003 (narrow persistent kernel)
    wl2, head2, lt2, last2 = _inputs("qwen3-8b-b16", V=5003, d=96, H=128, r=128, B=7, batch=3, dtype="bf16")
    head2.prepare()
    assert head2.path(wl2.batch, wl2.B, lt2.dtype, False) == 1
    _both(head2, lt2, last2, alpha=0.7)
    # the per-position launches (unprepared head) on the same scratch
    _both(head2.twin(), lt2, last2, alpha=0.7)


def test_noalloc_recovers_after_a_failed_call():
    """A call refused by the kernel (a prepared buffer of another head) sets the scratch's error
    word; the next call restores the scratch first and drafts normally."""
    wl, head, lt, last = _inputs("qwen3-8b-b16", V=4099, d=128, H=128, r=128, B=5, batch=37, dtype="bf16")
    head.prepare()
    _, other, _, _ = _inputs("qwen3-8b-b16", seed=991, V=4099, d=128, H=128, r=128, B=5, batch=37, dtype="bf16")
    other.c.prepared = head.prepared.data_ptr()
    other.c.prepared_bytes = head.prepared.numel()
    tok, st = B.draft_block_noalloc(other, lt, last, None, 1.0, 0.5, 0.0)
    torch.cuda.synchronize()
    assert B.workspace_error(None) == B.DLS_DRAFT_ERR_PREPARED
    assert bool((tok == -1).all().item()) and bool(torch.isnan(st).all().item())
    _both(head, lt, last)


def test_noalloc_refuses_oversized_calls():
    """A call whose workspace would exceed the 32 MiB scratch is refused on the host (nothing is
    read from the uninitialised tensors)."""
    V, d, H, r = 1024, 64, 4096, 256
    e = lambda *s: torch.empty(s, dtype=torch.bfloat16, device="cuda")
    head = B.LocalHead(e(V, d), e(3 * H, d), e(3 * H, H), e(r, H), e(V, r))
    with pytest.raises(B.DlsError, match="scratch"):
        B.draft_block_noalloc(head, e(256, 64, V), torch.zeros(256, dtype=torch.int32, device="cuda"))
