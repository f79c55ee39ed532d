"""Failure handling of the persistent drafting kernel through the C ABI, forced from the host so
that every kernel exits normally at its entry check:

* a workspace whose error word is already set (an earlier stalled hand-off) makes a call write
  token -1 everywhere and NaN statistics, and dls_draft_block_error reports the word; a
  zero-filled workspace works again;
* a prepared buffer that belongs to another head (same shapes, other tensors) is refused by
  the kernel (DLS_DRAFT_ERR_PREPARED) with the same sentinels; the error word is sticky.
"""
import numpy as np
import pytest
import torch

from paper_2607_07409_amd import binding as B
from paper_2607_07409_amd import workloads as W

pytestmark = pytest.mark.gpu

SHAPES = [dict(V=5003, d=96, H=128, r=128, B=7, batch=3),      # narrow kernel
          dict(V=4099, d=128, H=128, r=128, B=5, batch=37)]    # wide kernel (three M tiles)


def _setup(i, seed=None):
    wl = W.WORKLOADS["qwen3-8b-b16"].with_(dtype="bf16", **SHAPES[i])
    hw = W.make_head(wl, "stress", seed=seed)
    head = B.LocalHead.from_weights(hw).prepare()
    lt = B.as_tensor(W.make_long_logits(wl))
    last = torch.from_numpy(W.make_last_token(wl)).cuda()
    assert head.path(wl.batch, wl.B, lt.dtype, False) == 1
    return wl, head, lt, last


def _call(head, lt, last, ws):
    tok, st = B.draft_block(head, lt, last, None, 1.0, 0.5, 0.0, workspace=ws, exclusive_device=False)
    torch.cuda.synchronize()
    return tok, st


@pytest.mark.parametrize("i", range(len(SHAPES)))
def test_preset_error_word_gives_sentinels(i):
    wl, head, lt, last = _setup(i)
    ws = B.draft_workspace(head, wl.batch, wl.B)
    good_tok, good_st = _call(head, lt, last, ws)
    assert B.workspace_error(ws) == 0 and int((good_tok >= 0).all().item()) == 1
    ws[4:8].view(torch.int32).fill_(B.DLS_DRAFT_ERR_STALLED)     # as a stalled hand-off leaves it
    tok, st = _call(head, lt, last, ws)
    assert bool((tok == -1).all().item()), tok
    assert bool(torch.isnan(st).all().item())
    assert B.workspace_error(ws) == B.DLS_DRAFT_ERR_STALLED
    ws.zero_()
    tok2, st2 = _call(head, lt, last, ws)
    assert B.workspace_error(ws) == 0
    assert torch.equal(tok2, good_tok) and torch.equal(st2.view(torch.int32), good_st.view(torch.int32))


@pytest.mark.parametrize("i", range(len(SHAPES)))
def test_prepared_buffer_of_another_head_is_refused(i):
    wl, head, lt, last = _setup(i)
    _, other, _, _ = _setup(i, seed=991)
    ws = B.draft_workspace(head, wl.batch, wl.B)
    good_tok, good_st = _call(head, lt, last, ws)
    # other's descriptor pointing at head's prepared buffer: same size, wrong tensors
    other.c.prepared = head.prepared.data_ptr()
    other.c.prepared_bytes = head.prepared.numel()
    ws2 = B.draft_workspace(head, wl.batch, wl.B)
    tok, st = _call(other, lt, last, ws2)
    assert bool((tok == -1).all().item()) and bool(torch.isnan(st).all().item())
    assert B.workspace_error(ws2) == B.DLS_DRAFT_ERR_PREPARED
    # sticky until the workspace is zero-filled
    tok, _ = _call(head, lt, last, ws2)
    assert bool((tok == -1).all().item())
    ws2.zero_()
    tok, st = _call(head, lt, last, ws2)
    assert torch.equal(tok, good_tok) and torch.equal(st.view(torch.int32), good_st.view(torch.int32))
    assert B.workspace_error(ws2) == 0 and B.workspace_error(ws) == 0


def test_error_query_is_stream_ordered():
    """dls_draft_block_error reads the word after the work queued before it on the stream."""
    wl, head, lt, last = _setup(0)
    ws = B.draft_workspace(head, wl.batch, wl.B)
    s = torch.cuda.Stream()
    out = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    with torch.cuda.stream(s):
        ws[4:8].view(torch.int32).fill_(B.DLS_DRAFT_ERR_STALLED)
        B._check(B.lib().dls_draft_block_error(B._ptr(ws), ws.numel(), B._ptr(out), B._stream(s)))
    s.synchronize()
    assert int(out.item()) == B.DLS_DRAFT_ERR_STALLED
