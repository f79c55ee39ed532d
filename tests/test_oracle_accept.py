"""Pins of the verification statistics: acceptance length, tau, rate_i, the tau gain ratio
and the add-smoothing unigram prior.

* closed forms of the acceptance length on constructed targets;
* E[tau] = sum_i rate_i (tail-sum formula) on any sample;
* the paper's printed Table 3 gain ratios (Sec. 5.5) and Table 8 rate curves (App. D);
* the prior of App. A on small hand-checked counts.
"""
import json
import os

import numpy as np
import pytest

from oracle import dels_oracle as O

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def test_accept_len_closed_forms():
    g = np.random.default_rng(0)
    B = 16
    d = g.integers(0, 1000, (40, B))
    for k in range(B + 1):
        t = d.copy()
        if k < B:
            t[:, k] = (t[:, k] + 1) % 1000          # first mismatch exactly at k
            t[:, k + 1:] = g.integers(0, 1000, (40, B - k - 1))
        assert (O.accept_len(d, t) == k).all()
    # mismatch at position 0 with everything after equal still gives 0
    t = d.copy()
    t[:, 0] += 1
    assert (O.accept_len(d, t) == 0).all()


def test_accept_len_edge_shapes():
    assert O.accept_len(np.zeros((0, 5), int), np.zeros((0, 5), int)).shape == (0,)
    assert (O.accept_len(np.zeros((3, 0), int), np.zeros((3, 0), int)) == 0).all()
    assert O.accept_len(np.array([[4]]), np.array([[4]]))[0] == 1


def test_tau_tail_sum():
    g = np.random.default_rng(1)
    B = 16
    acc = g.integers(0, B + 1, 1000)
    rate = O.rate_curve(acc, B)
    assert rate[0] == 1.0
    assert np.all(np.diff(rate) <= 0)
    assert abs(rate.sum() - O.tau(acc).mean()) < 1e-12


def test_table8_rate_curve():
    """A population whose acceptance-length frequencies are read off the paper's Table 8
    reproduces the printed rate_i through rate_curve, and the printed differences agree."""
    gold = json.load(open(os.path.join(GOLD, "table8_rate_curve.json")))
    for col in ("dflash_percent", "dels_percent"):
        surv = np.array(gold[col]) / 100.0
        n = 100000
        counts = np.round(np.append(surv[:-1] - surv[1:], surv[-1]) * n).astype(int)
        acc = np.repeat(np.arange(16), counts)        # tau = acc + 1 in 1..16
        rate = O.rate_curve(acc, 16)[:16]
        np.testing.assert_allclose(rate * 100, gold[col], atol=2e-3)
        # the paper's tau of that column is the tail sum of its rates
        assert abs(O.tau(acc).mean() - surv.sum()) < 1e-3
    diff = np.array(gold["dels_percent"]) - np.array(gold["dflash_percent"])
    np.testing.assert_allclose(diff, gold["diff_percent"], atol=0.011)


def test_table3_gain_ratio():
    gold = json.load(open(os.path.join(GOLD, "table3_tau_gain_ratio.json")))
    for i, name in enumerate(gold["benchmarks"]):
        ratio = O.tau_gain_ratio(gold["tau_dels_rnn"][i], gold["tau_dflash"][i],
                                 gold["tau_domino_ft"][i])
        assert abs(100 * ratio - gold["gain_ratio_percent"][i]) < 0.006, name
    # the average ratio: (0.3075 / 0.40625) from the unrounded means
    m = {k: float(np.mean(gold[k])) for k in ("tau_dels_rnn", "tau_dflash", "tau_domino_ft")}
    r = O.tau_gain_ratio(m["tau_dels_rnn"], m["tau_dflash"], m["tau_domino_ft"])
    assert abs(100 * r - gold["avg"]["gain_ratio_percent"]) < 0.006
    for k in ("tau_dels_rnn", "tau_dflash", "tau_domino_ft"):
        assert abs(m[k] - gold["avg"][k]) < 0.0051


def test_unigram_prior_closed_form():
    # counts (3, 0, 1) with smoothing 1: (4, 1, 2) / 7
    np.testing.assert_allclose(O.unigram_log_prior([3, 0, 1]), np.log([4 / 7, 1 / 7, 2 / 7]),
                               rtol=1e-14)
    # no counts at all: uniform
    np.testing.assert_allclose(O.unigram_log_prior(np.zeros(8)), np.full(8, -np.log(8)), rtol=1e-14)
    # smoothing 0.5
    np.testing.assert_allclose(O.unigram_log_prior([1, 1], 0.5), np.log([0.5, 0.5]), rtol=1e-14)
    p = O.unigram_log_prior(np.random.default_rng(0).integers(0, 100, 1000))
    assert abs(np.exp(p).sum() - 1) < 1e-12
