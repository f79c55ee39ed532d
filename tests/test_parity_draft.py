"""GPU parity of dls_draft_block and dls_accept_len against the oracle, on all five
drafting workloads (tiny; Qwen3-4B and -8B shaped at batch 1; batch 16; batch 64),
with baseline and stress-scaled head weights, both first-row readings, the prior term,
a ragged small problem and mixed dtypes.
"""
import functools

import numpy as np
import pytest
import torch

from oracle import dels_oracle as O
from paper_2607_07409_amd import binding as B
from paper_2607_07409_amd import workloads as W
from parity_util import TOL, check_draft

pytestmark = pytest.mark.gpu


@functools.lru_cache(maxsize=2)
def _problem(name, init, V=None, d=None, H=None, r=None, Bk=None, batch=None, dtype=None):
    wl = W.WORKLOADS[name]
    kw = {k: v for k, v in dict(V=V, d=d, H=H, r=r, B=Bk, batch=batch, dtype=dtype).items() if v is not None}
    if kw:
        wl = wl.with_(**kw)
    hw = W.make_head(wl, init)
    return dict(wl=wl, hw=hw, head=B.LocalHead.from_weights(hw), oracle=O.RnnHead.from_weights(hw),
                long_h=W.make_long_logits(wl), last=W.make_last_token(wl),
                prior=W.make_zipf_log_prior(wl.V, wl.seed))


def _draft(p, alpha, beta=0.0, with_prior=False, literal=False, long_h=None):
    long_h = p["long_h"] if long_h is None else long_h
    lt = B.as_tensor(long_h)
    last = torch.from_numpy(p["last"]).cuda()
    prior = torch.from_numpy(p["prior"]).cuda() if with_prior else None
    tok, st = B.draft_block(p["head"], lt, last, prior, 1.0, alpha, beta, first_row_long_only=literal)
    torch.cuda.synchronize()
    return tok.cpu().numpy(), st.cpu().numpy()


def _check(p, alpha, beta=0.0, with_prior=False, literal=False, sequences=None):
    tok, st = _draft(p, alpha, beta, with_prior, literal)
    rep = check_draft(tok, st, p["oracle"], p["long_h"], p["last"], p["prior"] if with_prior else None,
                      1.0, alpha, beta if with_prior else 0.0, literal, sequences)
    print(f"{p['wl'].name}: near_ties={rep['near_ties']} fusion_active={rep['fusion_active']:.2f} "
          f"errs={rep['errs']}")
    return tok, st, rep


@pytest.mark.parametrize("init", ["baseline", "stress"])
@pytest.mark.parametrize("literal", [False, True])
@pytest.mark.parametrize("with_prior", [False, True])
def test_tiny(init, literal, with_prior):
    p = _problem("tiny", init)
    _check(p, 0.5, 0.5, with_prior, literal)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_small_ragged(dtype):
    """V not a multiple of any tile, rows of the long logits misaligned, d/H/r small and odd multiples of 8."""
    p = _problem("qwen3-8b-b16", "stress", V=5003, d=72, H=40, r=24, Bk=7, batch=3, dtype=dtype)
    _, _, rep = _check(p, 1.0)
    assert rep["fusion_active"] > 0.2


def test_mixed_dtypes():
    """fp32 head weights with bf16 long logits and the reverse."""
    p = _problem("qwen3-8b-b16", "stress", V=3001, d=64, H=64, r=32, Bk=5, batch=2, dtype="f32")
    lb = W.Bf16Array.from_f32(np.asarray(p["long_h"], np.float32))
    tok, st = _draft(p, 0.5, long_h=lb)
    check_draft(tok, st, p["oracle"], lb, p["last"], None, 1.0, 0.5, 0.0)


@pytest.mark.parametrize("init", ["baseline", "stress"])
def test_qwen3_4b_b1(init):
    p = _problem("qwen3-4b-b1", init)
    tok, st, rep = _check(p, 0.5)
    if init == "stress":
        assert rep["fusion_active"] > 0.3
    # literal first-row reading on the same inputs
    _check(p, 0.5, literal=True)


@pytest.mark.parametrize("alpha", [0.25, 0.5, 1.0])
def test_qwen3_8b_b1_alpha_sweep(alpha):
    p = _problem("qwen3-8b-b1", "stress")
    _check(p, alpha)


def test_qwen3_8b_b1_alpha_zero_is_dflash():
    p = _problem("qwen3-8b-b1", "stress")
    tok, _ = _draft(p, 0.0)
    assert np.array_equal(tok, np.argmax(np.asarray(p["long_h"], np.float32), axis=2))


@pytest.mark.parametrize("init", ["baseline", "stress"])
def test_serving_b16(init):
    p = _problem("qwen3-8b-b16", init)
    _check(p, 0.5, sequences=[0, 5, 10, 15])


def test_serving_b64():
    p = _problem("b64-d5120", "stress")
    _check(p, 0.5, sequences=[0, 21, 42, 63])


def test_serving_b64_prior():
    """beta = alpha with the Zipf log-prior (the paper's alpha = beta diagonal)."""
    p = _problem("b64-d5120", "stress")
    _check(p, 0.5, 0.5, with_prior=True, sequences=[1, 62])


@pytest.mark.parametrize("name", ["tiny", "qwen3-4b-b1", "qwen3-8b-b16"])
def test_accept_len_on_drafts(name):
    """Targets agree with the oracle draft for a geometric prefix; the GPU acceptance length on its own
    draft equals the oracle's on that draft."""
    p = _problem(name, "stress")
    tok, _ = _draft(p, 0.5)
    seqs = list(range(min(p["wl"].batch, 4)))
    ref = O.draft_block(p["oracle"], p["long_h"], p["last"], None, 1.0, 0.5, 0.0, sequences=seqs)
    targets, k = W.make_targets(ref.tokens, p["wl"])
    acc = B.accept_len(torch.from_numpy(tok).cuda(), torch.from_numpy(targets).cuda())
    torch.cuda.synchronize()
    want = O.accept_len(tok, targets)
    assert np.array_equal(acc.cpu().numpy(), want)
    same = np.array_equal(tok[seqs], ref.tokens[seqs])
    if same:
        assert np.all(want[seqs] >= k[seqs])


def test_accept_len_cases():
    g = np.random.default_rng(3)
    for batch, Bk in [(1, 1), (5, 16), (300, 16), (7, 100), (3, 0), (64, 64), (2, 65)]:
        d = g.integers(0, 50, (batch, Bk)).astype(np.int32)
        t = d.copy()
        for b in range(batch):
            if Bk:
                k = int(g.integers(0, Bk + 1))
                if k < Bk:
                    t[b, k] += 1
        got = B.accept_len(torch.from_numpy(d).cuda(), torch.from_numpy(t).cuda())
        torch.cuda.synchronize()
        assert np.array_equal(got.cpu().numpy(), O.accept_len(d, t)), (batch, Bk)


def test_draft_deterministic():
    p = _problem("qwen3-4b-b1", "stress")
    t0, s0 = _draft(p, 0.5)
    for _ in range(3):
        t1, s1 = _draft(p, 0.5)
        assert np.array_equal(t0, t1) and np.array_equal(s0, s1)
