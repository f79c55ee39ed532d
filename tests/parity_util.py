"""Comparison protocol between the HIP path and the CPU oracle.

Tokens must be identical, except at a position where the oracle's top-2 fused gap is
below TOL; there the GPU token must still be a valid near-argmax (its oracle fused value
within TOL of the maximum).  Such positions are counted.  The oracle is always replayed
on the GPU's own tokens (force=...), so after a tolerated near-tie both sides keep
conditioning on the same history.  Scores, log-probabilities and log-sum-exps must agree
within TOL absolute (float32 accumulation against float64).
"""
import numpy as np

from oracle import dels_oracle as O

TOL = 2e-2
STAT_KEYS = ("score", "logprob", "gap", "lse_long", "lse_short", "lse_fused")


def _stat(stats, k):
    return np.asarray(stats)[..., STAT_KEYS.index(k)].astype(np.float64)


def compare_stats(gpu_stats, ref, keys=("score", "logprob", "lse_long", "lse_short", "lse_fused"), idx=None):
    """Max abs error per statistic; NaN must match NaN (rows without short logits)."""
    errs = {}
    for k in keys:
        g = _stat(gpu_stats, k)
        r = np.asarray(getattr(ref, k) if not isinstance(ref, dict) else ref[k], dtype=np.float64)
        if idx is not None:
            g, r = g[idx], r[idx]
        nan_r = np.isnan(r)
        assert np.array_equal(np.isnan(g), nan_r), f"NaN pattern differs for {k}"
        d = np.abs(g[~nan_r] - r[~nan_r])
        errs[k] = float(d.max()) if d.size else 0.0
        assert errs[k] <= TOL, f"{k}: max abs error {errs[k]:.3e} > {TOL}"
    return errs


def check_rows(gpu_tok, gpu_stats, long_rows, short_rows, prior, w_long, alpha, beta, row_ids=None):
    """Oracle rows replayed on the GPU tokens (force_token), then the protocol.
    Returns (near_tie_count, errs, oracle rows)."""
    near = 0
    gt = np.asarray(gpu_tok)
    ids = range(gt.shape[0]) if row_ids is None else row_ids
    rows = []
    for i in ids:
        r = O.combine_row(long_rows[i], short_rows[i], prior, w_long, alpha, beta, force_token=int(gt[i]))
        if r.argmax != gt[i]:
            assert r.gap < TOL and r.margin < TOL, (
                f"row {i}: GPU token {gt[i]} vs oracle {r.argmax}, gap {r.gap:.3e}, margin {r.margin:.3e}")
            near += 1
        rows.append(r)
    if gpu_stats is None:
        return near, {}, rows
    ref = {k: np.array([getattr(r, k) for r in rows]) for k in STAT_KEYS}
    errs = compare_stats(np.asarray(gpu_stats)[list(ids)], ref)
    return near, errs, rows


def check_draft(gpu_tok, gpu_stats, head, long_logits, last_token, prior, w_long, alpha, beta,
                literal=False, sequences=None, temperature=0.0, seed=0, gates=None):
    """Replay the oracle on the GPU's tokens and apply the comparison protocol.  With
    temperature > 0 the oracle draws the same Gumbel noise (seed) and the gaps and margins
    are those of the perturbed values l / T + g, so a near-tie there is tolerated likewise.
    gates: the oracle's own adaptive-fusion gates [batch, B] (never the GPU's).

    Returns a report dict (near-tie count, max errors, fusion-active fraction, the oracle result)."""
    gt = np.asarray(gpu_tok)
    batch, B = gt.shape
    seqs = list(range(batch)) if sequences is None else list(sequences)
    ref = O.draft_block(head, long_logits, last_token, prior, w_long, alpha, beta,
                        first_row_long_only=literal, force=gt, sequences=seqs, temperature=temperature, seed=seed,
                        gates=gates)
    near = 0
    active = 0
    for b in seqs:
        rows = np.asarray(long_logits[b], dtype=np.float32)
        long_arg = np.argmax(rows, axis=1)
        for j in range(B):
            if ref.argmax[b, j] != gt[b, j]:
                assert ref.gap[b, j] < TOL and ref.margin[b, j] < TOL, (
                    f"seq {b} pos {j}: GPU token {gt[b, j]} vs oracle {ref.argmax[b, j]}, "
                    f"gap {ref.gap[b, j]:.3e}, margin {ref.margin[b, j]:.3e}")
                near += 1
            active += int(ref.argmax[b, j] != long_arg[j])
    errs = {}
    if gpu_stats is not None:
        idx = np.ix_(seqs, range(B))
        errs = compare_stats(np.asarray(gpu_stats), ref, idx=idx)
    return dict(near_ties=near, errs=errs, fusion_active=active / (len(seqs) * B), ref=ref)
