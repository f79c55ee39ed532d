"""Pins of the oracle's fusion and greedy decoding against values fixed by mathematics.

* exact rational brute force: with logits = ln(positive rationals) every softmax is
  rational, so the fused distribution p_L^w p_S^a / p_P^b (Sec. 4.3 fusion equation,
  token-independent factors absorbed as in Sec. 4.1) is rational for integer exponents
  and its argmax, ties, gap and log-probabilities are known exactly;
* half-integer alpha with perfect-square short weights (still rational);
* shift invariance of log-softmax (Sec. 4.1: token-independent factors drop out);
* the limits alpha = beta = 0 (DFlash alone, Sec. 5.6, Table 4) and the
  all-zero head;
* a hand-worked three-position example through the Markov head of App. A.
"""
import itertools
import math
from fractions import Fraction

import numpy as np
import pytest

from oracle import dels_oracle as O


def _exact_row(qL, qS, qP, w, a, b):
    """Exact fused quantities for integer exponents w, a, b in {0, 1}."""
    sL, sS, sP = sum(qL), sum(qS), sum(qP)
    pL = [Fraction(q, sL) for q in qL]
    pS = [Fraction(q, sS) for q in qS]
    pP = [Fraction(q, sP) for q in qP]
    F = [pL[v] ** w * pS[v] ** a / pP[v] ** b for v in range(len(qL))]
    best = max(F)
    tok = F.index(best)                           # lowest index among ties
    rest = sorted(F, reverse=True)
    gap = math.log(rest[0] / rest[1]) if len(F) > 1 else math.inf
    tot = sum(F)
    # the fused logits themselves are w ln qL + a ln qS - b ln pP (unnormalised long/short)
    G = [Fraction(qL[v]) ** w * Fraction(qS[v]) ** a / pP[v] ** b for v in range(len(qL))]
    return dict(token=tok, gap=gap, score=math.log(F[tok]), logprob=math.log(F[tok] / tot),
                lse_long=math.log(sL), lse_short=math.log(sS), lse_fused=math.log(sum(G)),
                scores=[math.log(f) for f in F])


def _random_cases(n, seed):
    g = np.random.default_rng(seed)
    for _ in range(n):
        V = int(g.integers(1, 7))
        qL = [int(x) for x in g.integers(1, 10, size=V)]
        qS = [int(x) for x in g.integers(1, 10, size=V)]
        qP = [int(x) for x in g.integers(1, 10, size=V)]
        yield qL, qS, qP


def _tie_cases():
    # exact ties that the lowest-index rule must resolve
    yield [2, 3, 3], [1, 1, 1], [1, 1, 1]
    yield [2, 3], [3, 2], [1, 1]
    yield [1, 1, 1, 1], [1, 1, 1, 1], [1, 1, 1, 1]
    yield [4, 1, 2], [1, 4, 2], [1, 1, 1]      # 4*1 == 1*4 > 2*2 tie between 0 and 1
    yield [6, 2, 3], [1, 3, 2], [2, 1, 1]      # prior breaks the tie of the product


@pytest.mark.parametrize("w,a,b", list(itertools.product([0, 1], repeat=3)))
def test_brute_force_exact(w, a, b):
    cases = list(_random_cases(200, 1000 + 4 * w + 2 * a + b)) + list(_tie_cases())
    for qL, qS, qP in cases:
        ex = _exact_row(qL, qS, qP, w, a, b)
        long_row = np.log(np.array(qL, dtype=np.float64))
        short_row = np.log(np.array(qS, dtype=np.float64))
        prior = np.log(np.array(qP, dtype=np.float64) / sum(qP))
        res = O.combine_row(long_row, short_row, prior, float(w), float(a), float(b),
                            want_scores=True)
        assert res.token == ex["token"], (qL, qS, qP, w, a, b)
        if math.isinf(ex["gap"]):
            assert math.isinf(res.gap)
        else:
            assert abs(res.gap - ex["gap"]) < 1e-12
        for k in ("score", "logprob", "lse_long", "lse_short", "lse_fused"):
            assert abs(getattr(res, k) - ex[k]) < 1e-12, k
        np.testing.assert_allclose(res.scores, ex["scores"], atol=1e-12)


def test_brute_force_half_alpha():
    """alpha = 1/2 with short weights that are perfect squares: p_S^(1/2) is rational up to
    the token-independent factor (sum s^2)^(-1/2)."""
    g = np.random.default_rng(7)
    for _ in range(300):
        V = int(g.integers(2, 7))
        qL = [int(x) for x in g.integers(1, 10, size=V)]
        s = [int(x) for x in g.integers(1, 6, size=V)]
        qS = [x * x for x in s]
        F = [Fraction(qL[v], 1) * s[v] for v in range(V)]
        best = max(F)
        tok = F.index(best)
        res = O.combine_row(np.log(np.array(qL, float)), np.log(np.array(qS, float)), None,
                            1.0, 0.5, 0.0)
        assert res.token == tok
        # c_tok = log p_L(tok) + 1/2 log p_S(tok)
        exp_score = math.log(Fraction(qL[tok], sum(qL))) + 0.5 * math.log(Fraction(qS[tok], sum(qS)))
        assert abs(res.score - exp_score) < 1e-12
        exp_lp = math.log(F[tok] / sum(F))
        assert abs(res.logprob - exp_lp) < 1e-12


def test_shift_invariance():
    g = np.random.default_rng(3)
    V = 257
    for _ in range(50):
        L = g.normal(0, 3, V)
        S = g.normal(0, 2, V)
        P = np.log(g.dirichlet(np.ones(V)))
        w, a, b = 1.0, float(g.uniform(0, 1.5)), float(g.uniform(0, 1))
        base = O.combine_row(L, S, P, w, a, b, want_scores=True)
        sh = O.combine_row(L + g.normal(0, 50), S + g.normal(0, 50), P, w, a, b, want_scores=True)
        if base.gap > 1e-6:
            assert sh.token == base.token
        for k in ("score", "logprob", "gap"):
            assert abs(getattr(sh, k) - getattr(base, k)) < 1e-9 * max(1.0, abs(getattr(base, k)))
        np.testing.assert_allclose(sh.scores, base.scores, atol=1e-9)
        # the fused log-softmax is also invariant to a shift of the prior
        sp = O.combine_row(L, S, P + 5.0, w, a, b)
        assert sp.token == base.token and abs(sp.logprob - base.logprob) < 1e-9


def _rnn_head(seed, V=97, d=24, H=16, r=8, scale=1.0):
    g = np.random.default_rng(seed)
    return O.RnnHead(g.normal(0, 1, (V, d)), g.normal(0, scale / math.sqrt(d), (3 * H, d)),
                     g.normal(0, scale / math.sqrt(H), (3 * H, H)),
                     g.normal(0, 1 / math.sqrt(H), (r, H)), g.normal(0, 3 / math.sqrt(r), (V, r)))


def test_alpha_zero_is_dflash():
    """alpha = beta = 0: the draft is the row-wise argmax of the long logits (the DFlash baseline)."""
    g = np.random.default_rng(11)
    head = _rnn_head(1)
    L = g.normal(0, 3, (3, 6, 97)).astype(np.float32)
    last = g.integers(0, 97, 3)
    res = O.draft_block(head, L, last, None, 1.0, 0.0, 0.0)
    np.testing.assert_array_equal(res.tokens, np.argmax(L, axis=2))
    # same with the literal first-row reading
    res2 = O.draft_block(head, L, last, None, 1.0, 0.0, 0.0, first_row_long_only=True)
    np.testing.assert_array_equal(res2.tokens, np.argmax(L, axis=2))


def test_alpha_zero_with_prior():
    """alpha = 0, beta > 0: argmax of l_L - beta * l_P, row by row."""
    g = np.random.default_rng(12)
    head = _rnn_head(2)
    L = g.normal(0, 3, (2, 5, 97))
    P = np.log(g.dirichlet(np.ones(97)))
    res = O.draft_block(head, L, [3, 4], P, 1.0, 0.0, 0.7)
    np.testing.assert_array_equal(res.tokens, np.argmax((L - 0.7 * P).astype(np.float32), axis=2))


def test_zero_head_equals_dflash():
    """All-zero head weights give zero short logits, so fusion leaves the long argmax."""
    g = np.random.default_rng(13)
    V, d, H, r = 50, 8, 6, 4
    head = O.RnnHead(np.zeros((V, d)), np.zeros((3 * H, d)), np.zeros((3 * H, H)),
                     np.zeros((r, H)), np.zeros((V, r)))
    L = g.normal(0, 3, (2, 7, V))
    res = O.draft_block(head, L, [1, 2], None, 1.0, 0.5, 0.0)
    np.testing.assert_array_equal(res.tokens, np.argmax(L.astype(np.float32), axis=2))
    # lse_short of an all-zero row is log V
    assert np.allclose(res.lse_short, math.log(V))


# ---------------------------------------------------------------------------------------
# hand-worked example: V = 3, B = 3, last token 2, w_long = 1, alpha = 1, beta = 0.
# Short logits come from a Markov head with E_M = I_3 and W_M = T^T, i.e. row T[prev].
#   T[0] = [0, 0, ln 2], T[1] = [ln 5, 0, 0], T[2] = [0, ln 3, 0]
#   long rows: [ln 2, 0, 0], [0, 0, ln 4], [0, ln 3, 0]
# Row 0 (prev 2): p_L = [1/2, 1/4, 1/4], p_S = [1/5, 3/5, 1/5], p_L p_S = [1/10, 3/20, 1/20] -> 1
# Row 1 (prev 1): p_L = [1/6, 1/6, 2/3], p_S = [5/7, 1/7, 1/7], product [5/42, 1/42, 4/42] -> 0
# Row 2 (prev 0): p_L = [1/5, 3/5, 1/5], p_S = [1/4, 1/4, 1/2], product [1/20, 3/20, 1/10] -> 1
# ---------------------------------------------------------------------------------------
LN = math.log
T_TABLE = np.array([[0, 0, LN(2)], [LN(5), 0, 0], [0, LN(3), 0]])
LONG3 = np.array([[[LN(2), 0, 0], [0, 0, LN(4)], [0, LN(3), 0]]])


def _markov_h3():
    return O.MarkovHead(np.eye(3), T_TABLE.T.copy())


def test_hand_worked_example():
    res = O.draft_block(_markov_h3(), LONG3, [2], None, 1.0, 1.0, 0.0)
    assert res.tokens.tolist() == [[1, 0, 1]]
    np.testing.assert_allclose(res.gap[0], [LN(3 / 2), LN(5 / 4), LN(3 / 2)], atol=1e-12)
    np.testing.assert_allclose(res.score[0], [LN(3 / 20), LN(5 / 42), LN(3 / 20)], atol=1e-12)
    np.testing.assert_allclose(res.logprob[0], [LN(1 / 2), LN(1 / 2), LN(1 / 2)], atol=1e-12)
    np.testing.assert_allclose(res.lse_long[0], [LN(4), LN(6), LN(5)], atol=1e-12)
    np.testing.assert_allclose(res.lse_short[0], [LN(5), LN(7), LN(4)], atol=1e-12)
    # full score rows c_v = log(p_L p_S)
    r0 = O.combine_row(LONG3[0, 0], T_TABLE[2], None, 1.0, 1.0, 0.0, want_scores=True)
    np.testing.assert_allclose(r0.scores, [LN(1 / 10), LN(3 / 20), LN(1 / 20)], atol=1e-12)


def test_hand_worked_variants():
    h = _markov_h3()
    # long logits alone (alpha = 0): [0, 2, 1]
    assert O.draft_block(h, LONG3, [2], None, 1.0, 0.0, 0.0).tokens.tolist() == [[0, 2, 1]]
    # head alone (w_long = 0): [1, 0, 2]
    assert O.draft_block(h, LONG3, [2], None, 0.0, 1.0, 0.0).tokens.tolist() == [[1, 0, 2]]
    # literal first-row reading: row 0 from the long logits, head starts from d_0 = 0
    assert O.draft_block(h, LONG3, [2], None, 1.0, 1.0, 0.0,
                         first_row_long_only=True).tokens.tolist() == [[0, 2, 1]]
    # with a prior P = ln[0.7, 0.15, 0.15], beta = 1: row 1 becomes token 2,
    # p_L p_S / p_P = [5/42/0.7, 1/42/0.15, 4/42/0.15]
    P = np.log([0.7, 0.15, 0.15])
    res = O.draft_block(h, LONG3, [2], P, 1.0, 1.0, 1.0)
    assert res.tokens.tolist() == [[1, 2, 1]]
    assert abs(res.gap[0, 1] - LN((4 / 42 / 0.15) / (5 / 42 / 0.7))) < 1e-12


def test_literal_first_row_random():
    """With the literal first-row reading, row 0 ignores the head and the last token, and the
    head state after row 0 starts from d_0 (checked against a direct replay)."""
    g = np.random.default_rng(21)
    head = _rnn_head(5, scale=2.0)
    L = g.normal(0, 1, (2, 5, 97))
    r1 = O.draft_block(head, L, [10, 20], None, 1.0, 1.0, 0.0, first_row_long_only=True)
    r2 = O.draft_block(head, L, [30, 40], None, 1.0, 1.0, 0.0, first_row_long_only=True)
    np.testing.assert_array_equal(r1.tokens, r2.tokens)           # last token unused
    np.testing.assert_array_equal(r1.tokens[:, 0], np.argmax(L[:, 0].astype(np.float32), 1))
    assert np.all(np.isnan(r1.lse_short[:, 0]))
    # rows 1.. equal the default reading started from d_0 on rows 1..
    r3 = O.draft_block(head, L[:, 1:], r1.tokens[:, 0], None, 1.0, 1.0, 0.0)
    np.testing.assert_array_equal(r3.tokens, r1.tokens[:, 1:])


def test_force_replay():
    """A forced token replaces the decoded one and feeds the head; statistics refer to it."""
    g = np.random.default_rng(22)
    head = _rnn_head(6, scale=2.0)
    L = g.normal(0, 1, (1, 6, 97))
    free = O.draft_block(head, L, [3], None, 1.0, 1.0, 0.0)
    force = free.tokens.copy()
    force[0, 2] = (force[0, 2] + 1) % 97
    fr = O.draft_block(head, L, [3], None, 1.0, 1.0, 0.0, force=force)
    np.testing.assert_array_equal(fr.tokens, force)
    np.testing.assert_array_equal(fr.tokens[0, :2], free.tokens[0, :2])
    assert fr.logprob[0, 2] < free.logprob[0, 2]


def test_decision_precision_float32():
    """Two fused values that differ only below float32 resolution are a tie: lowest index wins."""
    L = np.array([1.0, 1.0 + 1e-12, 0.0])
    assert O.combine_row(L, np.zeros(3), None, 1.0, 0.0, 0.0).token == 0
    L2 = np.array([1.0, 1.0 + 1e-5, 0.0])
    assert O.combine_row(L2, np.zeros(3), None, 1.0, 0.0, 0.0).token == 1


def test_per_position_weights():
    """Per-position alpha_j / beta_j (Sec. 5.6): a constant schedule is the scalar run; a schedule
    is the same as drafting each row with its own scalars, fed the same previous tokens; alpha_j = 0
    at a row gives that row the long logits' argmax (minus the prior term)."""
    g = np.random.default_rng(23)
    head = _rnn_head(5, scale=2.0)
    L = g.normal(0, 1, (2, 6, 97))
    P = np.log(g.dirichlet(np.ones(97)))
    sc = O.draft_block(head, L, [4, 9], P, 1.0, 0.4, 0.2)
    cs = O.draft_block(head, L, [4, 9], P, 1.0, [0.4] * 6, [0.2] * 6)
    np.testing.assert_array_equal(sc.tokens, cs.tokens)
    np.testing.assert_array_equal(sc.score, cs.score)
    al = [0.0, 0.3, 1.0, 0.0, 2.0, 0.5]
    be = [0.1, 0.0, 0.7, 0.3, 0.0, 1.0]
    res = O.draft_block(head, L, [4, 9], P, 1.0, al, be)
    for b, last in enumerate([4, 9]):
        state, u = head.init_state(), last
        for j in range(6):
            state, s = head.step(state, u)
            r = O.combine_row(L[b, j], s, P, 1.0, al[j], be[j])
            assert res.tokens[b, j] == r.token and abs(res.score[b, j] - r.score) < 1e-12
            if al[j] == 0.0:
                fused = (L[b, j] - be[j] * P).astype(np.float32)
                assert res.tokens[b, j] == int(np.argmax(fused))
            u = r.token


def _exact_masked(qL, qS, w, a):
    """Exact fused quantities when some long probabilities are 0 (a -inf long logit, a masked
    token).  With integer exponents the fused weight is p_L^w p_S^a, and 0^0 = 1: a zero long
    weight leaves a masked token in play, a positive one removes it."""
    sL, sS = sum(qL), sum(qS)
    F = [Fraction(qL[v], sL) ** w * Fraction(qS[v], sS) ** a for v in range(len(qL))]
    best = max(F)
    tok = F.index(best)
    rest = sorted(F, reverse=True)
    if len(F) < 2:
        gap = math.inf
    elif rest[1] == 0:
        gap = math.inf
    else:
        gap = math.log(rest[0] / rest[1])
    G = [Fraction(qL[v]) ** w * Fraction(qS[v]) ** a for v in range(len(qL))]
    return dict(token=tok, gap=gap, score=math.log(F[tok]), logprob=math.log(F[tok] / sum(F)),
                lse_long=math.log(sL), lse_short=math.log(sS), lse_fused=math.log(sum(G)),
                scores=[math.log(f) if f > 0 else -math.inf for f in F])


@pytest.mark.parametrize("w,a", [(0, 1), (1, 0), (1, 1)])
def test_brute_force_masked_long(w, a):
    """Masked long logits (-inf): with w_long = 1 a masked token can never be drafted unless
    every token is masked; with w_long = 0 the mask is absent with the rest of the long term
    (the fusion's exponent form, p^0 = 1)."""
    g = np.random.default_rng(4242 + 2 * w + a)
    for _ in range(400):
        V = int(g.integers(1, 7))
        qL = [int(x) for x in g.integers(0, 6, size=V)]
        if sum(qL) == 0:
            qL[int(g.integers(0, V))] = 1          # at least one unmasked token
        qS = [int(x) for x in g.integers(1, 10, size=V)]
        with np.errstate(divide="ignore"):
            long_row = np.log(np.array(qL, dtype=np.float64))
        short_row = np.log(np.array(qS, dtype=np.float64))
        ex = _exact_masked(qL, qS, w, a)
        res = O.combine_row(long_row, short_row, None, float(w), float(a), 0.0, want_scores=True)
        assert res.token == ex["token"], (qL, qS, w, a)
        if w == 1:
            assert qL[res.token] > 0
        if math.isinf(ex["gap"]):
            assert math.isinf(res.gap) and res.gap > 0, (qL, qS, w, a, res.gap)
        else:
            assert abs(res.gap - ex["gap"]) < 1e-12
        for k in ("score", "logprob", "lse_long", "lse_short", "lse_fused"):
            assert abs(getattr(res, k) - ex[k]) < 1e-12, (k, qL, qS, w, a)
        np.testing.assert_allclose(res.scores, ex["scores"], atol=1e-12)


def test_zero_prior_weight_ignores_unseen_tokens():
    """beta = 0 removes the prior term even where an unsmoothed prior is -inf (an unseen
    token): the fused row equals the row without a prior."""
    g = np.random.default_rng(11)
    for _ in range(50):
        V = int(g.integers(2, 40))
        L = g.normal(0, 3, V)
        S = g.normal(0, 2, V)
        P = np.log(g.dirichlet(np.ones(V)))
        P[g.integers(0, V, size=3)] = -np.inf
        a = O.combine_row(L, S, P, 1.0, 0.5, 0.0, want_scores=True)
        b = O.combine_row(L, S, None, 1.0, 0.5, 0.0, want_scores=True)
        assert a.token == b.token and a.gap == b.gap and a.logprob == b.logprob
        np.testing.assert_array_equal(a.scores, b.scores)
