"""Pins of the oracle's sampling path (temperature T > 0, Gumbel-max over softmax(l / T)):

* Philox4x32-10 against its published known-answer vectors;
* the uniforms lie in (0, 1) and are exact float32 numbers;
* the Gumbel noise has the standard moments (mean: Euler's constant, variance pi^2 / 6);
* the sampled tokens follow softmax(l / T) (chi-square over many independent rows) at
  T = 1 and T = 0.5, and a tiny T gives the greedy token;
* the statistics of a sampled row: logprob = log softmax(l / T) at the token.
"""
import json
import math
import os

import numpy as np

from oracle import dels_oracle as O

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def test_philox_known_answers():
    kat = json.load(open(os.path.join(GOLD, "philox4x32_10_kat.json")))
    for v in kat["vectors"]:
        ctr = np.array([int(x, 16) for x in v["counter"]], dtype=np.uint32)
        key = tuple(int(x, 16) for x in v["key"])
        out = O.philox4x32(ctr, key)
        assert [f"{int(x):08x}" for x in out] == v["output"]


def test_uniforms_exact_and_open():
    u = O.uniforms_row(1234567890123, 3, 7, 100_003)
    assert u.shape == (100_003,)
    assert np.all(u > 0) and np.all(u < 1)
    assert np.array_equal(u.astype(np.float32).astype(np.float64), u)
    # one counter per four entries: entries 4q..4q+3 are the four words of one Philox call
    x = O.philox4x32(np.array([5, 7, 3, 0], np.uint32), (1234567890123 & 0xFFFFFFFF, 1234567890123 >> 32))
    np.testing.assert_array_equal(u[20:24], ((x.astype(np.uint64) >> 9).astype(np.float64) + 0.5) * 2.0 ** -23)
    # different rows and seeds give different noise
    assert not np.array_equal(u, O.uniforms_row(1234567890123, 3, 8, 100_003))
    assert not np.array_equal(u, O.uniforms_row(1234567890124, 3, 7, 100_003))


def test_gumbel_moments():
    g = np.concatenate([O.gumbel_row(99, b, j, 151_936) for b in range(2) for j in range(2)])
    n = g.size
    assert abs(g.mean() - 0.5772156649) < 5 * math.sqrt(math.pi ** 2 / 6 / n)
    assert abs(g.var() - math.pi ** 2 / 6) < 0.02


def _chi2_ok(counts, probs):
    n = counts.sum()
    exp = n * probs
    chi2 = float(np.sum((counts - exp) ** 2 / exp))
    dof = len(probs) - 1
    return chi2 < dof + 6 * math.sqrt(2 * dof), chi2


def test_sampling_follows_softmax():
    V = 6
    logits = np.array([1.0, 0.2, -0.5, 2.0, 0.0, 1.3])
    for T in (1.0, 0.5):
        draws = np.zeros(V, int)
        for j in range(4000):
            r = O.combine_row(logits, None, None, 1.0, 0.0, 0.0, temperature=T, gumbel=O.gumbel_row(7, 0, j, V))
            draws[r.token] += 1
            # the statistics refer to softmax(l / T)
            ref = logits / T - np.log(np.sum(np.exp(logits / T)))
            assert abs(r.logprob - ref[r.token]) < 1e-12
        p = np.exp(logits / T)
        ok, chi2 = _chi2_ok(draws, p / p.sum())
        assert ok, (T, chi2, draws)


def test_small_temperature_is_greedy():
    g = np.random.default_rng(5)
    for j in range(20):
        row = g.normal(0, 1, 1000)
        r = O.combine_row(row, None, None, 1.0, 0.0, 0.0, temperature=1e-6, gumbel=O.gumbel_row(3, 0, j, 1000))
        assert r.token == int(np.argmax(row.astype(np.float32)))


def test_sampled_block_uses_row_noise():
    """A sampled draft block decodes each row from l / T + gumbel_row(seed, b, j, V)."""
    g = np.random.default_rng(6)
    V, Bk = 50, 4
    head = O.MarkovHead(g.normal(0, 1, (V, 8)), g.normal(0, 1, (V, 8)))
    L = g.normal(0, 1, (2, Bk, V))
    res = O.draft_block(head, L, [3, 4], None, 1.0, 0.5, 0.0, temperature=0.8, seed=42)
    for b, last in enumerate([3, 4]):
        u = last
        for j in range(Bk):
            _, s = head.step(None, u)
            f = L[b, j] + 0.5 * s
            want = int(np.argmax((f / 0.8 + O.gumbel_row(42, b, j, V)).astype(np.float32)))
            assert res.tokens[b, j] == want
            u = want
