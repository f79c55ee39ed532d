"""Hand-off robustness under injected delays (GPU).

libdels_stress.so is the library with the persistent kernel compiled with DLS_STRESS_DELAYS: before
every cross-workgroup publish (h words, rho words, argmax keys, merged tokens, statistics partials,
the final header) a wave may pause 3 to 10 us, pseudo-randomly per call, workgroup, wave, position
and site.  The pauses reorder the hand-offs but must not change a single bit: each call is compared
with the product library's result on the same inputs, for the narrow and both wide forms (one M
tile, and several with the delegated token merge), the Markov head, sampling, the prior and both
launch modes, several calls in a row on one workspace (every call draws other pauses).  The error word must stay clear; the pauses lie far inside the bounded waits.
"""
import math
import os

import numpy as np
import pytest
import torch

from paper_2607_07409_amd import binding as B
from paper_2607_07409_amd import workloads as W

pytestmark = pytest.mark.gpu

CALLS = 4


def _case(name, markov=False, batch=None):
    wl = W.WORKLOADS[name] if batch is None else W.WORKLOADS[name].with_(batch=batch, seed=batch)
    if markov:
        em, wm = W.make_markov_head(wl.V, wl.r, "bf16", 90, scale=math.sqrt(3.0 / math.sqrt(wl.r)))
        head = B.LocalHead.markov_from_weights(em, wm)
    else:
        head = B.LocalHead.from_weights(W.make_head(wl, "stress"))
    head.prepare()
    L = B.as_tensor(W.make_long_logits(wl))
    last = torch.from_numpy(W.make_last_token(wl)).cuda()
    return wl, head, L, last


def _draft(head, wl, L, last, ws, **kw):
    tok, st = B.draft_block(head, L, last, kw.pop("prior", None), 1.0, 0.5, kw.pop("beta", 0.0), workspace=ws, **kw)
    return tok, st


@pytest.mark.parametrize("name,markov,batch,kw", [
    ("qwen3-4b-b1", False, None, {}),                                   # narrow
    ("qwen3-4b-b1", False, 3, {"first_row_long_only": True}),           # narrow, literal first row
    ("qwen3-8b-b16", False, None, {}),                                  # wide, one M tile
    ("qwen3-8b-b16", False, 37, {}),                                    # wide, three M tiles, ragged
    ("b64-d5120", False, None, {"exclusive_device": True}),             # wide, four M tiles, ordinary dispatch
    ("qwen3-8b-b16", True, None, {}),                                   # Markov head
    ("b64-d5120", True, 37, {}),                                        # Markov head, delegated merge
    ("qwen3-8b-b16", False, None, {"temperature": 1.0, "seed": 77}),    # sampled
    ("qwen3-8b-b16", False, None, {"prior": True, "beta": 0.4}),        # prior
])
def test_delays_change_no_bit(name, markov, batch, kw):
    if not os.path.exists(B.STRESS_LIB_PATH):
        pytest.fail(f"{B.STRESS_LIB_PATH} is missing: build it with __graft_entry__.build()")
    wl, head, L, last = _case(name, markov, batch)
    kw = dict(kw)
    if kw.get("prior"):
        kw["prior"] = torch.from_numpy(W.make_zipf_log_prior(wl.V, wl.seed)).cuda()
    assert head.path(wl.batch, wl.B, L.dtype, kw.get("prior") is not None) == 1
    print(f"stress case {name} batch={wl.batch} markov={markov} {sorted(kw)}", flush=True)
    ws = B.draft_workspace(head, wl.batch, wl.B)
    ref_tok, ref_st = _draft(head, wl, L, last, ws, **kw)
    torch.cuda.synchronize()
    assert B.workspace_error(ws) == 0
    ref_tok, ref_st = ref_tok.clone(), ref_st.clone()
    with B.using(B.STRESS_LIB_PATH):
        sws = B.draft_workspace(head, wl.batch, wl.B)
        for c in range(CALLS):
            tok, st = _draft(head, wl, L, last, sws, **kw)
            torch.cuda.synchronize()
            assert B.workspace_error(sws) == 0, f"call {c}: error word set"
            assert torch.equal(tok, ref_tok), f"call {c}: tokens differ"
            assert torch.equal(st.view(torch.int32), ref_st.view(torch.int32)), f"call {c}: statistics differ"


def test_stress_build_pauses():
    """The test build really pauses: the same block takes longer than with the product library."""
    wl, head, L, last = _case("qwen3-8b-b16")
    ws = B.draft_workspace(head, wl.batch, wl.B)

    def timed(n=6):
        us = []
        for _ in range(n):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            _draft(head, wl, L, last, ws, exclusive_device=True)
            e1.record()
            torch.cuda.synchronize()
            us.append(e0.elapsed_time(e1) * 1e3)
        assert B.workspace_error(ws) == 0
        return float(np.median(us))

    timed(2)
    plain = timed()
    with B.using(B.STRESS_LIB_PATH):
        ws = B.draft_workspace(head, wl.batch, wl.B)
        timed(2)
        stressed = timed()
    print(f"block {plain:.1f} us, with pauses {stressed:.1f} us")
    assert stressed > plain * 1.05
