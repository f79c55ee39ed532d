"""GPU parity of adaptive fusion (Sec. 7's proposal: local-head and prior weights driven by the
entropy or confidence of the long logits) against the oracle.

dls_long_uncertainty is compared row by row with the oracle's entropy, maximum probability,
measure and gate, over ragged vocabularies, both dtypes, split and unsplit rows and the
degenerate rows (uniform, one-hot, masked, without a finite entry).  dls_draft_block_adaptive
is compared with the oracle's gated draft on both heads, both paths (per-position launches and
the persistent kernel, narrow and wide), both measures, with a prior, sampled at T = 1 and on
masked long logits; the gates the oracle uses are its own.  Rules whose gate is 1 everywhere
reproduce dls_draft_block bit for bit; rules whose gate is 0 everywhere decode the long logits
alone.
"""
import math

import numpy as np
import pytest
import torch

from oracle import dels_oracle as O
from paper_2607_07409_amd import binding as B
from paper_2607_07409_amd import workloads as W
from parity_util import check_draft

pytestmark = pytest.mark.gpu

RULES = {"qwen3-4b-b1": {O.UNC_ENTROPY: (0.55, 0.65), O.UNC_MAXPROB: (0.85, 0.97)},
         "qwen3-8b-b16": {O.UNC_ENTROPY: (0.40, 0.80), O.UNC_MAXPROB: (0.80, 0.99)},
         # the 25th and 75th to 80th percentiles of u over the batch-64 rows
         "b64-d5120": {O.UNC_ENTROPY: (0.35, 0.50), O.UNC_MAXPROB: (0.67, 0.90)}}


def _oracle_unc(rows, measure, lo, hi):
    out = []
    for x in rows:
        x = np.asarray(x, np.float64)
        u = O.uncertainty(x, measure)
        out.append((O.long_entropy(x), O.long_max_prob(x), u, O.gate(u, lo, hi)))
    return np.asarray(out)


def _check_unc(gpu, ref, lo, hi):
    gpu = np.asarray(gpu, np.float64).reshape(-1, 4)
    assert np.array_equal(np.isnan(gpu[:, :2]), np.isnan(ref[:, :2]))
    ok = ~np.isnan(ref[:, 0])
    err_h = np.abs(gpu[ok, 0] - ref[ok, 0])
    assert np.all(err_h <= 2e-5 + 2e-5 * np.abs(ref[ok, 0])), err_h.max()
    assert np.max(np.abs(gpu[ok, 1] - ref[ok, 1]), initial=0.0) <= 2e-6
    assert np.max(np.abs(gpu[:, 2] - ref[:, 2])) <= 1e-5
    assert np.max(np.abs(gpu[:, 3] - ref[:, 3])) <= 1e-5 / (hi - lo) + 1e-6


def _special_rows(V, rng):
    rows = [rng.normal(size=V) * 3.0, np.full(V, 0.75)]
    hot = np.full(V, -np.inf)
    hot[rng.integers(V)] = 4.0
    rows.append(hot)
    if V > 1:
        half = rng.normal(size=V) * 2.0
        half[rng.permutation(V)[: V // 2]] = -np.inf
        rows.append(half)
        rows.append(np.full(V, -np.inf))            # no finite entry
        big = rng.normal(size=V) * 40.0 + 1.0e4    # large magnitudes, sharp distribution
        rows.append(big)
    return np.stack(rows)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("V", [1, 2, 7, 1003, 5003, 151936])
@pytest.mark.parametrize("measure", [O.UNC_ENTROPY, O.UNC_MAXPROB])
def test_uncertainty_matches_oracle(V, dtype, measure):
    rng = np.random.default_rng(V + 17 * measure)
    rows = _special_rows(V, rng)
    t = torch.from_numpy(rows.astype(np.float32)).to(dtype).cuda()
    lo, hi = (0.2, 0.7) if measure == O.UNC_ENTROPY else (-0.3, 0.9)
    print(f"V={V} dtype={dtype} measure={measure} rows={rows.shape[0]}", flush=True)
    gpu = B.long_uncertainty(t, measure, lo, hi)
    torch.cuda.synchronize()
    ref = _oracle_unc(t.float().cpu().numpy(), measure, lo, hi)
    _check_unc(gpu.cpu().numpy(), ref, lo, hi)


@pytest.mark.parametrize("rows,V", [(3, 151936), (37, 30011), (2048, 5003), (4096, 1000)])
def test_uncertainty_split_and_unsplit_rows(rows, V):
    # few rows are split into ranges merged by a second kernel; many rows are one workgroup each
    rng = np.random.default_rng(rows * 7 + V)
    x = (rng.normal(size=(rows, V)) * rng.uniform(0.5, 6.0, size=(rows, 1))).astype(np.float32)
    x[0, : V // 3] = -np.inf
    t = torch.from_numpy(x).to(torch.bfloat16).cuda()
    print(f"rows={rows} V={V} parts-workspace={B.long_uncertainty_workspace_size(rows, V)}", flush=True)
    gpu = B.long_uncertainty(t, O.UNC_ENTROPY, 0.1, 0.9)
    torch.cuda.synchronize()
    xs = t.float().cpu().numpy()
    pick = sorted(set([0, 1, rows - 1] + list(np.random.default_rng(1).integers(0, rows, 60))))
    ref = _oracle_unc(xs[pick], O.UNC_ENTROPY, 0.1, 0.9)
    _check_unc(gpu.cpu().numpy()[pick], ref, 0.1, 0.9)


def test_uncertainty_is_deterministic_and_stream_ordered():
    x = torch.randn(5, 151936, device="cuda", dtype=torch.float32) * 2
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        a = B.long_uncertainty(x, O.UNC_ENTROPY, 0.0, 1.0, stream=s)
        b = B.long_uncertainty(x, O.UNC_ENTROPY, 0.0, 1.0, stream=s)
    s.synchronize()
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))


def _rnn(name):
    wl = W.WORKLOADS[name]
    hw = W.make_head(wl, "stress")
    return wl, B.LocalHead.from_weights(hw), O.RnnHead.from_weights(hw)


def _markov(name):
    wl = W.WORKLOADS[name].with_(seed=90)
    em, wm = W.make_markov_head(wl.V, wl.r, "bf16", 90, scale=math.sqrt(3.0 / math.sqrt(wl.r)))
    return wl, B.LocalHead.markov_from_weights(em, wm), O.MarkovHead(np.asarray(em, np.float64),
                                                                    np.asarray(wm, np.float64))


def _run(head, wl, measure, lo, hi, alpha=0.6, beta=0.3, prior=None, long_h=None, temperature=0.0, seed=0,
         literal=False):
    long_h = W.make_long_logits(wl) if long_h is None else long_h
    last = W.make_last_token(wl)
    lt = B.as_tensor(long_h)
    pt = None if prior is None else torch.from_numpy(np.ascontiguousarray(prior, np.float32)).cuda()
    ws = B.draft_workspace(head, wl.batch, wl.B)
    print(f"adaptive draft {wl.name} batch={wl.batch} path={head.path(wl.batch, wl.B, lt.dtype, prior is not None)} "
          f"measure={measure} rule=({lo}, {hi}) T={temperature}", flush=True)
    tok, st, unc = B.draft_block(head, lt, torch.from_numpy(last).cuda(), pt, 1.0, alpha, beta, workspace=ws,
                                 adaptive=(measure, lo, hi), temperature=temperature, seed=seed,
                                 first_row_long_only=literal)
    torch.cuda.synchronize()
    assert B.workspace_error(ws) == 0
    return tok.cpu().numpy(), st.cpu().numpy(), unc.cpu().numpy(), long_h, last


def _gates(long_h, measure, lo, hi):
    return O.adaptive_gates([np.asarray(long_h[b], np.float64) for b in range(len(long_h))], measure, lo, hi)


@pytest.mark.parametrize("prepared", [False, True])
@pytest.mark.parametrize("kind", ["rnn", "markov"])
@pytest.mark.parametrize("measure", [O.UNC_ENTROPY, O.UNC_MAXPROB])
def test_adaptive_draft_matches_oracle(kind, prepared, measure):
    wl, head, oh = _rnn("qwen3-4b-b1") if kind == "rnn" else _markov("qwen3-4b-b1")
    if prepared:
        head.prepare()
    lo, hi = RULES["qwen3-4b-b1"][measure]
    prior = W.make_zipf_log_prior(wl.V, wl.seed)
    tok, st, unc, long_h, last = _run(head, wl, measure, lo, hi, prior=prior)
    g = _gates(long_h, measure, lo, hi)
    assert (g == 0).any() and (g == 1).any() and ((g > 0) & (g < 1)).any(), g
    assert np.max(np.abs(unc[..., 3] - g)) <= 1e-5 / (hi - lo) + 1e-6
    rep = check_draft(tok, st, oh, long_h, last, prior, 1.0, 0.6, 0.3, gates=g)
    print(f"  near_ties={rep['near_ties']} fusion_active={rep['fusion_active']:.2f} errs={rep['errs']}")


@pytest.mark.parametrize("measure", [O.UNC_ENTROPY, O.UNC_MAXPROB])
def test_adaptive_draft_wide_batch(measure):
    # 16 sequences: the wide form of the persistent kernel, every sequence compared
    wl, head, oh = _rnn("qwen3-8b-b16")
    head.prepare()
    lo, hi = RULES["qwen3-8b-b16"][measure]
    tok, st, unc, long_h, last = _run(head, wl, measure, lo, hi, alpha=0.5, beta=0.0)
    g = _gates(long_h, measure, lo, hi)
    assert ((g > 0) & (g < 1)).mean() > 0.2
    rep = check_draft(tok, st, oh, long_h, last, None, 1.0, 0.5, 0.0, gates=g)
    print(f"  near_ties={rep['near_ties']} fusion_active={rep['fusion_active']:.2f}")


@pytest.mark.parametrize("batch", [5, 7])
def test_adaptive_draft_ragged_batch(batch):
    # batches past the narrow form with a partial M tile, and rows past V % 16 on the tail tile
    wl = W.WORKLOADS["qwen3-8b-b16"].with_(batch=batch, V=30011, seed=batch)
    hw = W.make_head(wl, "stress")
    head, oh = B.LocalHead.from_weights(hw).prepare(), O.RnnHead.from_weights(hw)
    u = [O.uncertainty(np.asarray(r, np.float64), O.UNC_ENTROPY) for r in np.asarray(W.make_long_logits(wl)).reshape(-1, wl.V)[:40]]
    lo, hi = float(np.percentile(u, 25)), float(np.percentile(u, 75))
    prior = W.make_zipf_log_prior(wl.V, wl.seed)
    tok, st, unc, long_h, last = _run(head, wl, O.UNC_ENTROPY, lo, hi, prior=prior)
    g = _gates(long_h, O.UNC_ENTROPY, lo, hi)
    check_draft(tok, st, oh, long_h, last, prior, 1.0, 0.6, 0.3, gates=g)


@pytest.mark.parametrize("prepared", [False, True])
def test_adaptive_sampled_matches_oracle(prepared):
    wl, head, oh = _rnn("qwen3-4b-b1")
    if prepared:
        head.prepare()
    lo, hi = RULES["qwen3-4b-b1"][O.UNC_MAXPROB]
    tok, st, unc, long_h, last = _run(head, wl, O.UNC_MAXPROB, lo, hi, temperature=1.0, seed=2607)
    g = _gates(long_h, O.UNC_MAXPROB, lo, hi)
    check_draft(tok, st, oh, long_h, last, None, 1.0, 0.6, 0.3, temperature=1.0, seed=2607, gates=g)


@pytest.mark.parametrize("prepared", [False, True])
def test_adaptive_masked_long_logits(prepared):
    wl, head, oh = _rnn("qwen3-4b-b1")
    if prepared:
        head.prepare()
    masked, _ = W.mask_long_logits(W.make_long_logits(wl), 0.5, 11, single=((0, 3),))
    lo, hi = 0.3, 0.7
    tok, st, unc, long_h, last = _run(head, wl, O.UNC_ENTROPY, lo, hi, long_h=masked, literal=True)
    g = _gates(masked, O.UNC_ENTROPY, lo, hi)
    assert g[0, 3] == 0.0        # one finite entry: certain
    check_draft(tok, st, oh, masked, last, None, 1.0, 0.6, 0.3, gates=g, literal=True)


@pytest.mark.parametrize("prepared", [False, True])
def test_full_gate_is_the_plain_draft(prepared):
    wl, head, _ = _rnn("qwen3-4b-b1")
    if prepared:
        head.prepare()
    prior = W.make_zipf_log_prior(wl.V, wl.seed)
    lt = B.as_tensor(W.make_long_logits(wl))
    last = torch.from_numpy(W.make_last_token(wl)).cuda()
    pt = torch.from_numpy(prior.astype(np.float32)).cuda()
    t0, s0 = B.draft_block(head, lt, last, pt, 1.0, 0.6, 0.3)
    t1, s1, unc = B.draft_block(head, lt, last, pt, 1.0, 0.6, 0.3, adaptive=(O.UNC_ENTROPY, -2.0, -1.0))
    torch.cuda.synchronize()
    assert torch.all(unc[..., 3] == 1.0)
    assert torch.equal(t0, t1) and torch.equal(s0.view(torch.int32), s1.view(torch.int32))


@pytest.mark.parametrize("prepared", [False, True])
@pytest.mark.parametrize("kind", ["rnn", "markov"])
def test_zero_gate_decodes_the_long_logits(kind, prepared):
    wl, head, _ = _rnn("qwen3-4b-b1") if kind == "rnn" else _markov("qwen3-4b-b1")
    if prepared:
        head.prepare()
    long_h = W.make_long_logits(wl)
    tok, st, unc, _, _ = _run(head, wl, O.UNC_MAXPROB, 1.5, 2.0, long_h=long_h,
                              prior=W.make_zipf_log_prior(wl.V, wl.seed))
    assert np.all(unc[..., 3] == 0.0)
    assert np.array_equal(tok, np.argmax(np.asarray(long_h, np.float32), axis=2))


def test_adaptive_split_launches():
    """80 sequences run as persistent launches of 64 and 16: each launch reads the gates of its own
    rows; the first and last sequence of both launches are compared with the oracle's gated draft."""
    wl = W.WORKLOADS["qwen3-8b-b16"].with_(batch=80, V=2053, d=64, H=128, r=128, B=4, seed=80)
    hw = W.make_head(wl, "stress")
    head, oh = B.LocalHead.from_weights(hw).prepare(), O.RnnHead.from_weights(hw)
    long_h = W.make_long_logits(wl)
    u = [O.uncertainty(np.asarray(r, np.float64), O.UNC_ENTROPY) for r in np.asarray(long_h).reshape(-1, wl.V)[:60]]
    lo, hi = float(np.percentile(u, 25)), float(np.percentile(u, 75))
    tok, st, unc, long_h, last = _run(head, wl, O.UNC_ENTROPY, lo, hi, long_h=long_h)
    g = _gates(long_h, O.UNC_ENTROPY, lo, hi)
    assert np.max(np.abs(unc[..., 3] - g)) <= 1e-5 / (hi - lo) + 1e-6
    check_draft(tok, st, oh, long_h, last, None, 1.0, 0.6, 0.3, sequences=[0, 63, 64, 79], gates=g)


@pytest.mark.parametrize("measure", [O.UNC_ENTROPY, O.UNC_MAXPROB])
@pytest.mark.parametrize("kind", ["rnn", "markov"])
def test_adaptive_b64_full_size(kind, measure):
    """Adaptive fusion at the batch-64 serving shape the bench times (prepared head, four M tiles
    and the delegated token merge), every sequence against the oracle with its own gates."""
    wl, head, oh = _rnn("b64-d5120") if kind == "rnn" else _markov("b64-d5120")
    head.prepare()
    assert head.path(wl.batch, wl.B, torch.bfloat16, False) == 1
    lo, hi = RULES["b64-d5120"][measure]
    tok, st, unc, long_h, last = _run(head, wl, measure, lo, hi, alpha=0.5, beta=0.0)
    g = _gates(long_h, measure, lo, hi)
    assert ((g > 0) & (g < 1)).mean() > 0.2
    assert np.max(np.abs(unc[..., 3] - g)) <= 1e-5 / (hi - lo) + 1e-6
    rep = check_draft(tok, st, oh, long_h, last, None, 1.0, 0.5, 0.0, gates=g)
    print(f"  near_ties={rep['near_ties']} fusion_active={rep['fusion_active']:.2f} errs={rep['errs']}")
