"""Pins of the oracle's adaptive fusion (Sec. 7: weights adjusted by the entropy or the
confidence of the long logits) against values fixed by the mathematics: the uniform and
one-hot limits, scipy's entropy of the same distribution, exact rational distributions on
tiny vocabularies, the binary entropy, and reductions of the gated draft to the
ungated one and to the long logits' own argmax.  CPU only.
"""
import math
from fractions import Fraction

import numpy as np
import pytest
import scipy.stats

import oracle as O

RNG = np.random.default_rng(2607)


@pytest.mark.parametrize("V", [2, 3, 7, 1000, 151936])
def test_uniform_row_has_entropy_log_v(V):
    row = np.full(V, -3.25)
    assert O.long_entropy(row) == pytest.approx(math.log(V), rel=1e-12)
    assert O.long_max_prob(row) == pytest.approx(1.0 / V, rel=1e-12)
    assert O.uncertainty(row, O.UNC_ENTROPY) == pytest.approx(1.0, rel=1e-12)
    assert O.uncertainty(row, O.UNC_MAXPROB) == pytest.approx(1.0, rel=1e-12)


@pytest.mark.parametrize("V,hot", [(1, 0), (2, 1), (9, 4), (5003, 17)])
def test_one_hot_row_is_certain(V, hot):
    row = np.full(V, -np.inf)
    row[hot] = 12.5
    assert O.long_entropy(row) == 0.0
    assert O.long_max_prob(row) == 1.0
    assert O.uncertainty(row, O.UNC_ENTROPY) == 0.0
    assert O.uncertainty(row, O.UNC_MAXPROB) == 0.0


def test_entropy_matches_scipy_on_random_distributions():
    for V in (2, 5, 64, 4096):
        for _ in range(5):
            p = RNG.dirichlet(np.full(V, 0.3))
            p = np.maximum(p, 1e-300)
            shift = RNG.normal() * 40
            row = np.log(p) + shift
            assert O.long_entropy(row) == pytest.approx(scipy.stats.entropy(p), rel=1e-9, abs=1e-12)
            assert O.long_max_prob(row) == pytest.approx(p.max() / p.sum(), rel=1e-9)


@pytest.mark.parametrize("counts", [(1, 1), (1, 3), (2, 1, 1), (5, 0, 3, 1), (1, 2, 3, 4, 5, 6), (7, 7, 1, 0, 0, 1)])
def test_exact_rational_distributions(counts):
    # p_v = k_v / K exactly; l_v = log k_v (a zero count is a masked entry).  H = log K - sum k log k / K,
    # max p = k_max / K as a fraction; both written out independently of the oracle's route.
    k = np.asarray(counts, dtype=np.float64)
    K = int(sum(counts))
    V = len(counts)
    row = np.where(k > 0, np.log(np.where(k > 0, k, 1.0)), -np.inf)
    h_exact = math.log(K) - sum(c * math.log(c) for c in counts if c > 0) / K
    assert O.long_entropy(row) == pytest.approx(h_exact, rel=1e-13, abs=1e-15)
    pmax = Fraction(max(counts), K)
    assert O.long_max_prob(row) == pytest.approx(float(pmax), rel=1e-14)
    u_max = (1 - pmax) / (1 - Fraction(1, V))
    assert O.uncertainty(row, O.UNC_MAXPROB) == pytest.approx(float(u_max), rel=1e-13, abs=1e-15)
    assert O.uncertainty(row, O.UNC_ENTROPY) == pytest.approx(h_exact / math.log(V), rel=1e-13, abs=1e-15)


def test_row_without_a_finite_entry_is_fully_uncertain():
    row = np.full(12, -np.inf)
    assert math.isnan(O.long_entropy(row)) and math.isnan(O.long_max_prob(row))
    assert O.uncertainty(row, O.UNC_ENTROPY) == 1.0 and O.uncertainty(row, O.UNC_MAXPROB) == 1.0
    assert O.adaptive_gates(row[None, None], O.UNC_MAXPROB, 0.2, 0.6)[0, 0] == 1.0


@pytest.mark.parametrize("q", [0.5, 0.1, 0.999, 1e-6])
def test_binary_entropy_closed_form(q):
    row = np.array([math.log(q), math.log1p(-q)]) + 3.0
    hb = -q * math.log(q) - (1 - q) * math.log1p(-q)
    assert O.long_entropy(row) == pytest.approx(hb, rel=1e-10)
    assert O.uncertainty(row, O.UNC_ENTROPY) == pytest.approx(hb / math.log(2), rel=1e-10)


def test_masked_entries_change_only_the_normalisation():
    row = RNG.normal(size=40) * 3
    masked = np.concatenate([row, np.full(60, -np.inf)])
    assert O.long_entropy(masked) == pytest.approx(O.long_entropy(row), rel=1e-13)
    assert O.long_max_prob(masked) == pytest.approx(O.long_max_prob(row), rel=1e-13)
    assert O.uncertainty(masked, O.UNC_ENTROPY) == pytest.approx(O.long_entropy(row) / math.log(100), rel=1e-13)


def test_sharper_rows_are_less_uncertain():
    row = RNG.normal(size=500)
    us = [O.uncertainty(row * t, m) for m in (O.UNC_ENTROPY, O.UNC_MAXPROB) for t in (0.0, 0.5, 1, 2, 8)]
    for m in range(2):
        seq = us[5 * m:5 * m + 5]
        assert all(a > b for a, b in zip(seq, seq[1:])), seq
        assert seq[0] == pytest.approx(1.0)


def test_gate_piecewise_linear():
    assert O.gate(0.2, 0.2, 0.6) == 0.0
    assert O.gate(0.6, 0.2, 0.6) == 1.0
    assert O.gate(0.4, 0.2, 0.6) == pytest.approx(0.5)
    assert O.gate(0.3, 0.2, 0.6) == pytest.approx(0.25)
    assert O.gate(0.0, 0.2, 0.6) == 0.0
    assert O.gate(1.0, 0.2, 0.6) == 1.0
    assert O.gate(0.0, -0.5, 0.5) == pytest.approx(0.5)     # a floor at u = 0
    with pytest.raises(ValueError):
        O.gate(0.5, 0.5, 0.5)
    with pytest.raises(ValueError):
        O.gate(0.5, 0.6, 0.2)


def _tiny_head(V, d=6, H=5, r=4, seed=1):
    rng = np.random.default_rng(seed)
    return O.RnnHead(emb=rng.normal(size=(V, d)) * 0.5, w_ih=rng.normal(size=(3 * H, d)) * 0.4,
                     w_hh=rng.normal(size=(3 * H, H)) * 0.4, w_rank=rng.normal(size=(r, H)) * 0.5,
                     w_vocab=rng.normal(size=(V, r)) * 0.8)


def test_unit_gates_are_the_plain_draft():
    V, B, batch = 23, 5, 3
    head = _tiny_head(V)
    long = RNG.normal(size=(batch, B, V))
    prior = np.log(RNG.dirichlet(np.ones(V)))
    ref = O.draft_block(head, long, [1, 2, 3], prior, 1.0, 0.3, 0.3)
    got = O.draft_block(head, long, [1, 2, 3], prior, 1.0, 0.3, 0.3, gates=np.ones((batch, B)))
    assert np.array_equal(ref.tokens, got.tokens)
    assert np.array_equal(ref.score, got.score)
    assert np.array_equal(ref.lse_fused, got.lse_fused)


def test_zero_gates_decode_the_long_logits_alone():
    V, B, batch = 31, 6, 2
    head = _tiny_head(V, seed=3)
    long = RNG.normal(size=(batch, B, V)) * 2
    long[0, 2, 5] = -np.inf
    prior = np.log(RNG.dirichlet(np.ones(V)))
    prior[7] = -np.inf
    got = O.draft_block(head, long, [4, 9], prior, 1.0, 0.7, 0.4, gates=np.zeros((batch, B)))
    assert np.array_equal(got.tokens, np.argmax(long.astype(np.float32), axis=2))
    assert np.allclose(got.lse_fused, got.lse_long)


def test_gates_of_one_sequence_are_a_position_schedule():
    # with one sequence a per-row gate is a per-position weight: alpha_j * g_j
    V, B = 17, 7
    head = _tiny_head(V, seed=5)
    long = RNG.normal(size=(1, B, V))
    prior = np.log(RNG.dirichlet(np.ones(V)))
    g = RNG.uniform(size=(1, B))
    g[0, 3] = 0.0
    alpha, beta = RNG.uniform(0.1, 1.0, B), RNG.uniform(0.1, 1.0, B)
    got = O.draft_block(head, long, [6], prior, 1.0, alpha, beta, gates=g)
    ref = O.draft_block(head, long, [6], prior, 1.0, alpha * g[0], beta * g[0])
    assert np.array_equal(got.tokens, ref.tokens)
    assert np.allclose(got.score, ref.score, rtol=1e-14, atol=1e-14)


def test_gates_follow_their_sequence():
    # row (b, j) of a batch uses gates[b, j]: the same as drafting sequence b alone with the
    # position schedule alpha * gates[b]
    V, B, batch = 19, 5, 4
    head = _tiny_head(V, seed=8)
    long = RNG.normal(size=(batch, B, V)) * 1.5
    g = RNG.uniform(size=(batch, B))
    g[2] = 0.0
    last = [3, 1, 4, 1]
    got = O.draft_block(head, long, last, None, 1.0, 0.9, 0.0, gates=g)
    for b in range(batch):
        ref = O.draft_block(head, long[b:b + 1], [last[b]], None, 1.0, 0.9 * g[b], np.zeros(B))
        assert np.array_equal(got.tokens[b], ref.tokens[0])
        assert np.allclose(got.score[b], ref.score[0], rtol=1e-14, atol=1e-14)


def test_adaptive_gates_of_a_block():
    long = RNG.normal(size=(2, 3, 50))
    long[1, 2] = -np.inf
    long[1, 2, 9] = 0.0                      # one-hot row: u = 0
    long[0, 1] = 1.5                         # uniform row: u = 1
    g = O.adaptive_gates(long, O.UNC_ENTROPY, 0.1, 0.9)
    assert g[1, 2] == 0.0 and g[0, 1] == 1.0
    for b in range(2):
        for j in range(3):
            u = O.long_entropy(long[b, j]) / math.log(50)
            assert g[b, j] == pytest.approx(min(1, max(0, (u - 0.1) / 0.8)), rel=1e-12, abs=1e-15)
