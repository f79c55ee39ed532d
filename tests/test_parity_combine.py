"""GPU parity of dls_combine_logits (fused combine + greedy argmax) against the oracle.

Shapes: the tiny workload's rows, the 16-row rows of the batch-1 Qwen3 workloads, the
256- and 1024-row serving shapes at V = 151,936, plus ragged/misaligned vocabularies,
V = 1, masked (-inf) long logits, exact ties and the prior term.
"""
import math

import numpy as np
import pytest
import torch

from oracle import dels_oracle as O
from paper_2607_07409_amd import binding as B
from paper_2607_07409_amd import workloads as W
from parity_util import TOL, check_rows

pytestmark = pytest.mark.gpu

QV = W.QWEN3_VOCAB


def _run(long_h, short_h, prior, wl, al, be, want_scores=False):
    lt = B.as_tensor(long_h)
    st = B.as_tensor(short_h)
    pt = None if prior is None else torch.from_numpy(np.ascontiguousarray(prior, dtype=np.float32)).cuda()
    tok, stats, scores = B.combine_logits(lt, st, pt, wl, al, be, want_stats=True, want_scores=want_scores)
    torch.cuda.synchronize()
    return (tok.cpu().numpy(), stats.cpu().numpy(),
            None if scores is None else scores.cpu().numpy())


def _check(long_h, short_h, prior, wl, al, be, row_ids=None, want_scores=False):
    tok, stats, scores = _run(long_h, short_h, prior, wl, al, be, want_scores)
    near, errs, rows = check_rows(tok, stats, long_h, short_h, prior, wl, al, be, row_ids=row_ids)
    if want_scores:
        for i, r in zip(row_ids if row_ids is not None else range(len(rows)), rows):
            ref = O.combine_row(long_h[i], short_h[i], prior, wl, al, be, want_scores=True).scores
            err = np.nanmax(np.abs(scores[i] - ref))
            assert err <= TOL, f"score row {i}: {err:.3e}"
            errs["scores_row"] = max(errs.get("scores_row", 0.0), float(err))
    print(f"rows={len(rows)} near_ties={near} errs={errs}")
    return tok, stats, near, errs


@pytest.mark.parametrize("rows,V,dtype,seed", [
    (4, 1024, "f32", 0),          # tiny workload rows
    (16, QV, "bf16", 1),          # batch-1 Qwen3 rows (B = 16)
    (7, 4099, "bf16", 2),         # ragged, rows start misaligned
    (5, 4099, "f32", 3),
    (3, 1, "bf16", 4),            # a single-token vocabulary
    (6, 3, "f32", 5),
    (33, 8191, "bf16", 6),
    (300, 5003, "bf16", 7),       # one 1024-thread workgroup per row (256 to 1023 rows)
    (257, 4099, "f32", 8),
])
def test_combine_shapes(rows, V, dtype, seed):
    L = W.make_logit_rows(rows, V, dtype, seed, "onehot", 3.0, purpose=20)
    S = W.make_logit_rows(rows, V, dtype, seed, "normal", 2.0, purpose=21)
    _check(L, S, None, 1.0, 0.5, 0.0, want_scores=V <= 8191)


@pytest.mark.parametrize("rows", [256, 1024])
def test_combine_serving_shapes(rows):
    L = W.make_logit_rows(rows, QV, "bf16", 10 + rows, "onehot", 3.0, purpose=20)
    S = W.make_logit_rows(rows, QV, "bf16", 10 + rows, "normal", 2.0, purpose=21)
    _check(L, S, None, 1.0, 0.5, 0.0)        # every row against the oracle


@pytest.mark.parametrize("wl,al,be", [(1.0, 0.0, 0.0), (0.0, 1.0, 0.0), (1.0, 0.3, 0.3), (1.0, 1.0, 1.0),
                                      (0.7, 0.25, 0.5)])
def test_combine_weights_and_prior(wl, al, be):
    rows, V = 9, 20011
    L = W.make_logit_rows(rows, V, "bf16", 30, "onehot", 3.0, purpose=20)
    S = W.make_logit_rows(rows, V, "bf16", 30, "normal", 3.0, purpose=21)
    P = W.make_zipf_log_prior(V, 30)
    tok, _, _, _ = _check(L, S, P, wl, al, be, want_scores=True)
    if al == 0.0:
        want = np.argmax(np.asarray(L, np.float32) * np.float32(wl) - np.float32(be) * P[None], axis=1)
        assert np.array_equal(tok, want)


@pytest.mark.parametrize("rows,dtype", [(8, "f32"), (1024, "f32"), (1024, "bf16")])
def test_combine_leaders_anywhere(rows, dtype):
    """The row's two largest fused values at the start, at the end, in ascending and descending
    rows: the 256-thread kernel skips the top-two pushes of iterations below its wave threshold,
    and must still keep both leaders (and the gap between them) wherever they lie."""
    V = 40000
    g = np.random.default_rng(50 + rows)
    L = g.normal(0, 1, (rows, V)).astype(np.float32)
    S = g.normal(0, 1, (rows, V)).astype(np.float32)
    for i in range(rows):
        k = i % 5
        if k == 0:
            L[i] = np.sort(L[i])               # ascending: the threshold rises to the very end
        elif k == 1:
            L[i] = np.sort(L[i])[::-1]         # descending: leaders first, nearly all skipped after
        elif k == 2:
            L[i, -2:] = [7.0, 6.5]             # both leaders in the last chunk
        elif k == 3:
            L[i, :2] = [7.0, 6.5]              # both leaders in the first chunk
        else:
            L[i, [3, V - 3]] = [7.0, 7.0]      # equal long leaders far apart: the short logits decide
    if dtype == "bf16":
        L, S = W.Bf16Array.from_f32(L), W.Bf16Array.from_f32(S)
    _check(L, S, None, 1.0, 0.5, 0.0)


@pytest.mark.parametrize("rows,V", [(8, 40000 + 8 * 37), (1024, 30000 + 8 * 13), (5, 1000)])
def test_combine_all_negative_rows(rows, V):
    """Rows whose fused values are all far below zero, at lengths that leave a ragged last
    iteration: the top-two threshold of a wave must come only from its own lanes' values (a
    threshold of 0 from anywhere else would skip every entry of such a row)."""
    g = np.random.default_rng(60 + rows)
    L = (g.normal(0, 1, (rows, V)) - 200.0).astype(np.float32)
    S = (g.normal(0, 1, (rows, V)) - 100.0).astype(np.float32)
    _check(L, S, None, 1.0, 0.5, 0.0)
    _check(W.Bf16Array.from_f32(L), W.Bf16Array.from_f32(S), None, 1.0, 0.5, 0.0)


def test_combine_exact_ties_lowest_index():
    """Equal fused values: the lowest index wins, bit-exactly (alpha = 0 keeps l = l_L exact)."""
    rows, V = 12, 30000
    g = np.random.default_rng(40)
    L = g.normal(0, 1, (rows, V)).astype(np.float32)
    for i in range(rows):
        pos = np.sort(g.choice(V, size=1 + i % 4, replace=False))
        L[i, pos] = 9.0                               # several copies of the maximum
    S = g.normal(0, 1, (rows, V)).astype(np.float32)
    tok, stats, _ = _run(L, S, None, 1.0, 0.0, 0.0)
    assert np.array_equal(tok, np.argmax(L, axis=1))
    assert np.all(stats[:, 2][[i for i in range(rows) if i % 4]] == 0.0)     # gap 0 on real ties
    Lb = W.Bf16Array.from_f32(L)
    Sb = W.Bf16Array.from_f32(S)
    tok2, _, _ = _run(Lb, Sb, None, 1.0, 0.0, 0.0)
    assert np.array_equal(tok2, np.argmax(np.asarray(Lb, np.float32), axis=1))


def test_combine_masked_long_logits():
    """-inf entries in the long logits (masked tokens) take no probability mass."""
    rows, V = 8, 5000
    g = np.random.default_rng(41)
    L = g.normal(0, 3, (rows, V)).astype(np.float32)
    L[g.random((rows, V)) < 0.3] = -np.inf
    S = g.normal(0, 2, (rows, V)).astype(np.float32)
    for arr in (L, W.Bf16Array.from_f32(L)):
        tok, stats, _ = _run(arr, W.Bf16Array.from_f32(S) if isinstance(arr, W.Bf16Array) else S,
                             None, 1.0, 0.5, 0.0)
        Lv = np.asarray(arr, np.float32)
        assert np.all(np.isfinite(Lv[np.arange(rows), tok]))
        for i in range(rows):
            r = O.combine_row(Lv[i], np.asarray(S[i], np.float32) if not isinstance(arr, W.Bf16Array)
                              else np.asarray(W.Bf16Array.from_f32(S)[i], np.float32), None, 1.0, 0.5, 0.0)
            assert tok[i] == r.token or r.gap < TOL
            assert abs(stats[i, 3] - r.lse_long) <= TOL
            assert abs(stats[i, 5] - r.lse_fused) <= TOL


def test_combine_empty_rows():
    lt = torch.empty((0, 100), dtype=torch.bfloat16, device="cuda")
    tok, st, _ = B.combine_logits(lt, lt, None, 1.0, 0.5, 0.0)
    torch.cuda.synchronize()
    assert tok.numel() == 0


def test_combine_deterministic():
    rows, V = 16, QV
    L = B.as_tensor(W.make_logit_rows(rows, V, "bf16", 50, "onehot", 3.0, purpose=20))
    S = B.as_tensor(W.make_logit_rows(rows, V, "bf16", 50, "normal", 2.0, purpose=21))
    t0, s0, _ = B.combine_logits(L, S, None, 1.0, 0.5, 0.0)
    for _ in range(5):
        t1, s1, _ = B.combine_logits(L, S, None, 1.0, 0.5, 0.0)
        torch.cuda.synchronize()
        assert torch.equal(t0, t1) and torch.equal(s0, s1)


@pytest.mark.parametrize("rows,V,dtype,seed,prior", [
    (16, QV, "bf16", 60, False),
    (256, QV, "bf16", 61, True),
    (7, 4099, "bf16", 62, False),
    (5, 4099, "f32", 63, True),
    (3, 1, "bf16", 64, False),
])
def test_combine_tokens_only_matches(rows, V, dtype, seed, prior):
    """Without statistics the kernel keeps only the running maximum: the tokens must be the
    same bits as with statistics, and agree with the oracle up to near-ties."""
    L = W.make_logit_rows(rows, V, dtype, seed, "onehot", 3.0, purpose=20)
    S = W.make_logit_rows(rows, V, dtype, seed, "normal", 2.0, purpose=21)
    P = W.make_zipf_log_prior(V, seed) if prior else None
    be = 0.5 if prior else 0.0
    lt, st = B.as_tensor(L), B.as_tensor(S)
    pt = None if P is None else torch.from_numpy(np.ascontiguousarray(P, dtype=np.float32)).cuda()
    t_stats, _, _ = B.combine_logits(lt, st, pt, 1.0, 0.5, be, want_stats=True)
    t_only, s_only, _ = B.combine_logits(lt, st, pt, 1.0, 0.5, be, want_stats=False)
    torch.cuda.synchronize()
    assert s_only is None
    assert torch.equal(t_stats, t_only)
    tok = t_only.cpu().numpy()
    for i in range(rows):
        r = O.combine_row(np.asarray(L[i], np.float32), np.asarray(S[i], np.float32), P, 1.0, 0.5, be)
        assert tok[i] == r.token or r.gap < TOL, (i, tok[i], r.token, r.gap)


def test_combine_tokens_only_ties_and_masks():
    rows, V = 12, 30000
    g = np.random.default_rng(65)
    L = g.normal(0, 1, (rows, V)).astype(np.float32)
    for i in range(rows):
        L[i, np.sort(g.choice(V, size=1 + i % 4, replace=False))] = 9.0
    L[g.random((rows, V)) < 0.2] = -np.inf
    S = g.normal(0, 1, (rows, V)).astype(np.float32)
    t, _, _ = B.combine_logits(B.as_tensor(L), B.as_tensor(S), None, 1.0, 0.0, 0.0, want_stats=False)
    torch.cuda.synchronize()
    Lm = np.where(np.isneginf(L), -np.inf, L)
    assert np.array_equal(t.cpu().numpy(), np.argmax(Lm, axis=1))
