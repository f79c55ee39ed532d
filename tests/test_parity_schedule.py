"""GPU parity of per-position fusion weights (dls_draft_block_scheduled; Sec. 5.6 learns one
alpha_j and beta_j per draft position) against the oracle, for the RNN and Markov heads, through
the per-position launches and the persistent kernel."""
import math

import numpy as np
import pytest
import torch

from oracle import dels_oracle as O
from paper_2607_07409_amd import binding as B
from paper_2607_07409_amd import workloads as W
from parity_util import check_draft

pytestmark = pytest.mark.gpu

ALPHA = [0.2 + 0.05 * j for j in range(16)]            # rising with the position, like the learned values
BETA = [0.1 + 0.02 * j for j in range(16)]


def _rnn():
    wl = W.WORKLOADS["qwen3-4b-b1"]
    hw = W.make_head(wl, "stress")
    return wl, B.LocalHead.from_weights(hw), O.RnnHead.from_weights(hw)


def _markov():
    wl = W.WORKLOADS["qwen3-4b-b1"].with_(seed=90)
    em, wm = W.make_markov_head(wl.V, wl.r, "bf16", 90, scale=math.sqrt(3.0 / math.sqrt(wl.r)))
    return wl, B.LocalHead.markov_from_weights(em, wm), O.MarkovHead(np.asarray(em, np.float64),
                                                                    np.asarray(wm, np.float64))


def _draft(head, wl, alpha, beta, prior=None, literal=False):
    long_h = W.make_long_logits(wl)
    last = W.make_last_token(wl)
    lt = B.as_tensor(long_h)
    pt = None if prior is None else torch.from_numpy(np.ascontiguousarray(prior, np.float32)).cuda()
    ws = B.draft_workspace(head, wl.batch, wl.B)
    tok, st = B.draft_block(head, lt, torch.from_numpy(last).cuda(), pt, 1.0, alpha, beta,
                            first_row_long_only=literal, workspace=ws)
    torch.cuda.synchronize()
    assert B.workspace_error(ws) == 0
    return tok.cpu().numpy(), st.cpu().numpy(), long_h, last


@pytest.mark.parametrize("prepared", [False, True])
@pytest.mark.parametrize("kind", ["rnn", "markov"])
def test_schedule_matches_oracle(kind, prepared):
    wl, head, oh = _rnn() if kind == "rnn" else _markov()
    if prepared:
        head.prepare()
    prior = W.make_zipf_log_prior(wl.V, wl.seed)
    tok, st, long_h, last = _draft(head, wl, ALPHA, BETA, prior)
    rep = check_draft(tok, st, oh, long_h, last, prior, 1.0, ALPHA, BETA)
    print(f"{kind} prepared={prepared}: near_ties={rep['near_ties']} fusion_active={rep['fusion_active']:.2f} "
          f"errs={rep['errs']}")
    assert rep["fusion_active"] > 0.2
    # literal first row with a schedule (row 0 ignores alpha_0 and beta_0)
    tok, st, long_h, last = _draft(head, wl, ALPHA, BETA, prior, literal=True)
    check_draft(tok, st, oh, long_h, last, prior, 1.0, ALPHA, BETA, literal=True)


@pytest.mark.parametrize("prepared", [False, True])
def test_constant_schedule_is_scalar(prepared):
    wl, head, oh = _rnn()
    if prepared:
        head.prepare()
    t0, s0, _, _ = _draft(head, wl, 0.5, 0.0)
    t1, s1, _, _ = _draft(head, wl, [0.5] * wl.B, [0.0] * wl.B)
    assert np.array_equal(t0, t1) and np.array_equal(s0.view(np.int32), s1.view(np.int32))


def test_zero_alpha_rows_follow_the_long_logits():
    wl, head, oh = _rnn()
    head.prepare()
    al = [0.0 if j % 3 == 0 else 0.6 for j in range(wl.B)]
    tok, st, long_h, last = _draft(head, wl, al, 0.0)
    rows = np.asarray(long_h[0], np.float32)
    for j in range(0, wl.B, 3):
        assert tok[0, j] == int(np.argmax(rows[j]))
    check_draft(tok, st, oh, long_h, last, None, 1.0, al, 0.0)


def test_schedule_rejects_bad_weights():
    wl, head, _ = _rnn()
    lt = B.as_tensor(W.make_long_logits(wl))
    last = torch.from_numpy(W.make_last_token(wl)).cuda()
    with pytest.raises(B.DlsError):
        B.draft_block(head, lt, last, None, 1.0, [0.5] * 15 + [float("nan")], 0.0)
    with pytest.raises(ValueError):
        B.draft_block(head, lt, last, None, 1.0, [0.5] * 3, 0.0)
