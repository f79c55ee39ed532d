"""GPU parity of dls_draft_block with the Markov local head (App. A, Markov variant:
rho_j = E_M[u_j], l_S = W_M rho_j) against the oracle.

* the hand-worked three-position example (V = 3) with its printed tokens, gaps, scores and
  log-probabilities, and its variants (long logits alone, head alone, literal first row, prior);
* random Markov heads at the Qwen3 vocabulary, through the per-position launches and the
  persistent kernel, for narrow (1, 3), wide (16) and multi-tile (37) batches, both first-row
  readings, the prior and float32 long logits;
* repeated calls on one workspace are bit-identical.
"""
import math

import numpy as np
import pytest
import torch

from oracle import dels_oracle as O
from paper_2607_07409_amd import binding as B
from paper_2607_07409_amd import workloads as W
from parity_util import TOL, check_draft

pytestmark = pytest.mark.gpu

LN = math.log
# the worked example: short logits are the row T[prev] of this table (E_M = I_3, W_M = T^T)
T_TABLE = np.array([[0, 0, LN(2)], [LN(5), 0, 0], [0, LN(3), 0]], dtype=np.float32)
LONG3 = np.array([[[LN(2), 0, 0], [0, 0, LN(4)], [0, LN(3), 0]]], dtype=np.float32)


def _h3_head():
    """E_M = I_3 and W_M = T^T, padded to rank 8 with zero columns (the rank must be a multiple of 8)."""
    em = np.zeros((3, 8), np.float32)
    em[:, :3] = np.eye(3)
    wm = np.zeros((3, 8), np.float32)
    wm[:, :3] = T_TABLE.T
    return em, wm


def _run(head, long_h, last, prior=None, wl=1.0, al=1.0, be=0.0, literal=False, expect_path=None):
    lt = B.as_tensor(long_h)
    last_t = None if last is None else torch.as_tensor(np.asarray(last, np.int32)).cuda()
    pt = None if prior is None else torch.from_numpy(np.ascontiguousarray(prior, np.float32)).cuda()
    if expect_path is not None:
        assert head.path(lt.shape[0], lt.shape[1], lt.dtype, prior is not None) == expect_path
    ws = B.draft_workspace(head, lt.shape[0], lt.shape[1])
    tok, st = B.draft_block(head, lt, last_t, pt, wl, al, be, first_row_long_only=literal, workspace=ws)
    torch.cuda.synchronize()
    assert B.workspace_error(ws) == 0
    return tok.cpu().numpy(), st.cpu().numpy()


def test_hand_worked_example():
    em, wm = _h3_head()
    head = B.LocalHead.markov_from_weights(em, wm)
    tok, st = _run(head, LONG3, [2])
    assert tok.tolist() == [[1, 0, 1]]
    np.testing.assert_allclose(st[0, :, 2], [LN(3 / 2), LN(5 / 4), LN(3 / 2)], atol=1e-5)     # gap
    np.testing.assert_allclose(st[0, :, 0], [LN(3 / 20), LN(5 / 42), LN(3 / 20)], atol=1e-5)  # score
    np.testing.assert_allclose(st[0, :, 1], [LN(1 / 2)] * 3, atol=1e-5)                        # logprob
    np.testing.assert_allclose(st[0, :, 3], [LN(4), LN(6), LN(5)], atol=1e-5)                  # lse_long
    np.testing.assert_allclose(st[0, :, 4], [LN(5), LN(7), LN(4)], atol=1e-5)                  # lse_short


def test_hand_worked_variants():
    em, wm = _h3_head()
    head = B.LocalHead.markov_from_weights(em, wm)
    assert _run(head, LONG3, [2], al=0.0)[0].tolist() == [[0, 2, 1]]           # long logits alone
    assert _run(head, LONG3, [2], wl=0.0)[0].tolist() == [[1, 0, 2]]           # head alone
    assert _run(head, LONG3, None, literal=True)[0].tolist() == [[0, 2, 1]]    # literal first row
    P = np.log([0.7, 0.15, 0.15])
    tok, st = _run(head, LONG3, [2], prior=P, be=1.0)
    assert tok.tolist() == [[1, 2, 1]]
    assert abs(st[0, 1, 2] - LN((4 / 42 / 0.15) / (5 / 42 / 0.7))) < 1e-5


def _markov_problem(V, r, batch, Bk, seed, dtype="bf16"):
    """A random Markov head scaled so that the short logits have a standard deviation near 3
    (comparable to the long logits), with the long logits of the Qwen3-shaped workloads."""
    scale = math.sqrt(3.0 / math.sqrt(r))
    em, wm = W.make_markov_head(V, r, dtype, seed, scale=scale)
    wl = W.WORKLOADS["qwen3-8b-b16"].with_(V=V, B=Bk, batch=batch, dtype=dtype, seed=seed)
    return dict(em=em, wm=wm, oracle=O.MarkovHead(np.asarray(em, np.float64), np.asarray(wm, np.float64)),
                long_h=W.make_long_logits(wl), last=W.make_last_token(wl),
                prior=W.make_zipf_log_prior(V, seed))


CASES = [
    dict(V=W.QWEN3_VOCAB, r=256, batch=1, Bk=16, seed=70),
    dict(V=W.QWEN3_VOCAB, r=256, batch=3, Bk=16, seed=71),
    dict(V=W.QWEN3_VOCAB, r=256, batch=16, Bk=16, seed=72),
    dict(V=5003, r=128, batch=37, Bk=5, seed=73),
    dict(V=7001, r=256, batch=2, Bk=9, seed=74),
    dict(V=5003, r=128, batch=100, Bk=4, seed=75),        # prepared: launches of 64 and 36 sequences
]


@pytest.mark.parametrize("prepared", [False, True])
@pytest.mark.parametrize("case", range(len(CASES)))
def test_markov_random(case, prepared):
    c = CASES[case]
    p = _markov_problem(c["V"], c["r"], c["batch"], c["Bk"], c["seed"])
    head = B.LocalHead.markov_from_weights(p["em"], p["wm"])
    if prepared:
        head.prepare()
    tok, st = _run(head, p["long_h"], p["last"], al=0.5, expect_path=1 if prepared else 0)
    seqs = sorted(set([0, c["batch"] // 2, c["batch"] - 1]))
    rep = check_draft(tok, st, p["oracle"], p["long_h"], p["last"], None, 1.0, 0.5, 0.0, sequences=seqs)
    print(f"markov {c}: prepared={prepared} near_ties={rep['near_ties']} "
          f"fusion_active={rep['fusion_active']:.2f} errs={rep['errs']}")
    assert rep["fusion_active"] > 0.2


@pytest.mark.parametrize("prepared", [False, True])
def test_markov_literal_and_prior(prepared):
    c = CASES[1]
    p = _markov_problem(c["V"], c["r"], c["batch"], c["Bk"], c["seed"])
    head = B.LocalHead.markov_from_weights(p["em"], p["wm"])
    if prepared:
        head.prepare()
    tok, st = _run(head, p["long_h"], None, literal=True, al=0.5)
    check_draft(tok, st, p["oracle"], p["long_h"], p["last"], None, 1.0, 0.5, 0.0, literal=True, sequences=[0, 2])
    tok, st = _run(head, p["long_h"], p["last"], prior=p["prior"], al=0.5, be=0.5)
    check_draft(tok, st, p["oracle"], p["long_h"], p["last"], p["prior"], 1.0, 0.5, 0.5, sequences=[1])


def test_markov_f32_long_logits_and_repeat():
    c = CASES[4]
    p = _markov_problem(c["V"], c["r"], c["batch"], c["Bk"], c["seed"])
    head = B.LocalHead.markov_from_weights(p["em"], p["wm"]).prepare()
    lf = np.asarray(p["long_h"], np.float32) + np.float32(1e-3)
    tok, st = _run(head, lf, p["last"], al=0.5, expect_path=1)
    check_draft(tok, st, p["oracle"], lf, p["last"], None, 1.0, 0.5, 0.0)
    # back-to-back calls on one workspace: the same bits every time
    lt = B.as_tensor(p["long_h"])
    last_t = torch.from_numpy(p["last"]).cuda()
    ws = B.draft_workspace(head, lt.shape[0], lt.shape[1])
    outs = []
    for _ in range(4):
        t, s = B.draft_block(head, lt, last_t, None, 1.0, 0.5, 0.0, workspace=ws)
        outs.append((t.clone(), s.clone()))
    torch.cuda.synchronize()
    assert B.workspace_error(ws) == 0
    for t, s in outs[1:]:
        assert torch.equal(t, outs[0][0]) and torch.equal(s.view(torch.int32), outs[0][1].view(torch.int32))
    ref = O.draft_block(p["oracle"], p["long_h"], p["last"], None, 1.0, 0.5, 0.0)
    near = outs[0][0].cpu().numpy() != ref.tokens
    assert np.all(ref.gap[near] < TOL)


@pytest.mark.parametrize("with_prior", [False, True])
def test_markov_b64_full_size(with_prior):
    """The Markov head at the batch-64 serving shape (V = 151,936, r = 256; prepared, four M
    tiles and the delegated token merge), greedy, with and without the Zipf prior, every sequence."""
    wl = W.WORKLOADS["b64-d5120"]
    em, wm = W.make_markov_head(wl.V, wl.r, "bf16", 92, scale=math.sqrt(3.0 / math.sqrt(wl.r)))
    head = B.LocalHead.markov_from_weights(em, wm).prepare()
    oh = O.MarkovHead(np.asarray(em, np.float64), np.asarray(wm, np.float64))
    long_h, last = W.make_long_logits(wl), W.make_last_token(wl)
    prior = W.make_zipf_log_prior(wl.V, wl.seed) if with_prior else None
    be = 0.5 if with_prior else 0.0
    tok, st = _run(head, long_h, last, prior=prior, wl=1.0, al=0.5, be=be, expect_path=1)
    rep = check_draft(tok, st, oh, long_h, last, prior, 1.0, 0.5, be)
    print(f"markov b64 prior={with_prior}: near_ties={rep['near_ties']} errs={rep['errs']}")
