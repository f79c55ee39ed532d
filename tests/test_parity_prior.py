"""GPU parity of dls_unigram_log_prior (App. A, prior estimation) against the oracle:
counts are exact, the log-prior matches the oracle's float64 value rounded to float32."""
import numpy as np
import pytest
import torch

from oracle import dels_oracle as O
from paper_2607_07409_amd import binding as B
from paper_2607_07409_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("n,V,smoothing,seed", [
    (1_000_000, W.QWEN3_VOCAB, 1.0, 80),     # Zipf-distributed stream at the Qwen3 vocabulary
    (12_345, 5003, 0.5, 81),
    (0, 1000, 1.0, 82),                      # no tokens: the uniform prior
    (777, 1, 1.0, 83),                       # a single-token vocabulary
    (4_000_000, 256, 1.0, 84),               # heavy contention on few counters
    (50_000, 100_000, 0.5, 86),              # three vocabulary slices, fewer chunks than XCDs
    (1_000_000, 400_000, 1.0, 85),           # too many slices: the cached counter
])
def test_unigram_prior(n, V, smoothing, seed):
    g = np.random.default_rng(seed)
    ranks = W.zipf_ranks(V, seed)
    order = np.argsort(ranks)                  # token of rank k+1
    p = 1.0 / np.arange(1, V + 1) ** 1.1
    p /= p.sum()
    toks = order[g.choice(V, size=n, p=p)].astype(np.int32) if n else np.zeros(0, np.int32)
    if n > 10:                                 # out-of-range entries are skipped
        toks[:3] = [-1, V, V + 7]
    t = torch.from_numpy(toks).cuda()
    logp, counts = B.unigram_log_prior(t, V, smoothing)
    torch.cuda.synchronize()
    valid = toks[(toks >= 0) & (toks < V)]
    want_counts = np.bincount(valid, minlength=V)
    got = counts.cpu().numpy()
    assert np.array_equal(got[:V], want_counts)
    assert got[V] == valid.size
    want = O.unigram_log_prior(want_counts, smoothing).astype(np.float32)
    got_p = logp.cpu().numpy()
    # float64 logarithms of two libraries, each rounded once to float32: at most one ulp apart
    ulps = np.abs(got_p.view(np.int32).astype(np.int64) - want.view(np.int32).astype(np.int64))
    assert ulps.max() <= 1, ulps.max()


@pytest.mark.parametrize("kind", ["uniform", "constant", "two_hot"])
def test_unigram_prior_adversarial_streams(kind):
    """Streams that stress the counters: uniform ids over the Qwen3 vocabulary (every counter of
    every slice touched, and every device count flushed by every chunk), one id repeated (every
    increment hits one LDS counter) and two adjacent ids, interleaved."""
    V = W.QWEN3_VOCAB
    g = np.random.default_rng(91)
    if kind == "uniform":
        toks = g.integers(0, V, 6_000_000).astype(np.int32)
    elif kind == "constant":
        toks = np.full(3_000_001, 4242, np.int32)
    else:
        toks = np.where(g.random(2_000_000) < 0.5, 17, 18).astype(np.int32)
    logp, counts = B.unigram_log_prior(torch.from_numpy(toks).cuda(), V, 1.0)
    torch.cuda.synchronize()
    want_counts = np.bincount(toks, minlength=V)
    got = counts.cpu().numpy()
    assert np.array_equal(got[:V], want_counts)
    assert got[V] == toks.size
    want = O.unigram_log_prior(want_counts, 1.0).astype(np.float32)
    ulps = np.abs(logp.cpu().numpy().view(np.int32).astype(np.int64) - want.view(np.int32).astype(np.int64))
    assert ulps.max() <= 1


def test_unigram_prior_feeds_combine():
    """The estimated prior is the prior argument of the fused combine (beta term)."""
    V = 4099
    g = np.random.default_rng(85)
    toks = torch.from_numpy(g.integers(0, 50, 10_000).astype(np.int32)).cuda()   # a few frequent tokens
    logp, _ = B.unigram_log_prior(toks, V, 1.0)
    L = W.make_logit_rows(6, V, "f32", 85, "normal", 1.0, purpose=20)
    S = W.make_logit_rows(6, V, "f32", 85, "normal", 1.0, purpose=21)
    tok, st, _ = B.combine_logits(B.as_tensor(L), B.as_tensor(S), logp, 1.0, 0.5, 1.0)
    torch.cuda.synchronize()
    P = logp.cpu().numpy().astype(np.float64)
    for i in range(6):
        r = O.combine_row(np.asarray(L[i]), np.asarray(S[i]), P, 1.0, 0.5, 1.0)
        assert tok[i].item() == r.token or r.gap < 2e-2
