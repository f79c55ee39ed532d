"""Plain CPU oracle for the DeLS-Spec block-drafting path.

TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only the tests, the smoke check of the
package entry point and the CPU-baseline leg of the benchmark may import this
module.  It shares no code with the HIP library and imports nothing from it.

Everything is computed in float64 with numpy, in the order the paper states:

* fusion of long, short and prior logits        -- Sec. 4.3, fusion equation
* DeLS-Spec inference over one draft block       -- Sec. 4.3, Algorithm 1
* RNN local head (bias-free one-layer GRU on the frozen target embedding,
  SiLU low-rank projection, vocabulary head)     -- App. A, RNN-head equation
* Markov local head                               -- App. A, Markov-head equation
* add-smoothing unigram log-prior                 -- App. A, prior estimation
* acceptance length, tau and rate_i               -- Sec. 5.1; App. D

Readings where the paper is silent (each is also listed in the design notes):

* GRU gates follow the common (r, z, n) convention with the reset gate applied
  to the recurrent part of the candidate, h' = (1 - z) * n + z * h, h_0 = 0.
* Greedy decoding: the argmax takes the lowest index among equal values.  The
  decision is taken on the fused logits rounded to float32 (the precision the
  GPU path decides in); every reported value is float64.
* The short-logit weight is the paper's alpha; a long-logit weight w_long
  (1 in the paper) is kept so that w_long = 0 gives the local head alone.
* A term whose weight is zero is absent, also where its logit is -inf (a
  masked token): 0 * (-inf) reads as 0, the exponent form p^0 = 1 of the
  fusion.  So w_long = 0 ignores a mask in the long logits, and beta = 0 an
  unsmoothed prior's -inf.
* Row j of the long logits is draft position j.  By default the head is seeded
  with the last accepted token and every row is fused.  With
  first_row_long_only=True row 0 is decoded from the long logits alone and the
  head only sees drafted tokens (the literal form of Algorithm 1).
* The acceptance length counts leading positions where draft == target
  (0..B); the paper's tau adds the bonus token, tau = accepted + 1.
* Per-position fusion weights alpha_j, beta_j (Sec. 5.6) are indexed by the
  row j of the block; a row decoded from the long logits alone ignores them.
* The Markov head's state at row j is E_M of the token before it: the last
  accepted token for row 0, the drafted token d_{j-1} afterwards.
* Adaptive fusion (Sec. 7 proposes it as future work without a rule): row (b, j)
  fuses with alpha_j * g and beta_j * g, g = clamp((u - h_lo) / (h_hi - h_lo), 0, 1)
  of that row's uncertainty u, either the entropy of p_L over log V or
  (1 - max p_L) / (1 - 1/V); u = 0 when V = 1 and u = 1 for a row without a
  finite entry.
* Sampling at temperature T > 0 (the paper reports T = 0 and T = 1 but not how
  it draws) is the Gumbel-max rule on l / T.  The noise of entry v of row
  (sequence b, position j) comes from Philox4x32-10 keyed by the seed at
  counter (v // 4, j, b, 0), word v % 4, u = ((x >> 9) + 1/2) / 2^23 and
  g = -log(-log u), so that a draw depends on (seed, b, j, v) only.

Parity pins (tests/test_oracle_*.py): exact-rational brute force on tiny
vocabularies, the alpha = 0 / w_long = 0 limits, shift invariance, a
hand-worked three-position example, torch.nn.GRU equivalence, closed forms
for the acceptance length, brute-force counting for the prior, the published
Philox4x32-10 known-answer vectors, the Gumbel moments and chi-square tests
of the sampled distribution.
"""
from __future__ import annotations

import dataclasses
from typing import Callable, Optional, Sequence

import numpy as np

F64 = np.float64


# ----------------------------------------------------------------------------------------
# elementary functions
# ----------------------------------------------------------------------------------------
def logsumexp(x: np.ndarray) -> float:
    """log sum_v exp(x_v), by subtracting the maximum first."""
    x = np.asarray(x, dtype=F64)
    m = np.max(x)
    if not np.isfinite(m):
        return float(m)
    return float(m + np.log(np.sum(np.exp(x - m))))


def sigmoid(x):
    return 1.0 / (1.0 + np.exp(-np.asarray(x, dtype=F64)))


def silu(x):
    x = np.asarray(x, dtype=F64)
    return x * sigmoid(x)


# ----------------------------------------------------------------------------------------
# Sec. 4.3: logit fusion and greedy decoding of one row
# ----------------------------------------------------------------------------------------
@dataclasses.dataclass
class RowResult:
    token: int
    score: float      # c_tok: w_long*log softmax(long) + alpha*log softmax(short) - beta*prior
    logprob: float    # q_tok: log softmax(fused)
    gap: float        # top-1 minus top-2 of the fused logits (inf if V == 1)
    lse_long: float
    lse_short: float  # nan when the row has no short logits
    lse_fused: float
    argmax: int = -1  # the oracle's own decision (differs from token only when forced)
    margin: float = 0.0   # fused[argmax] - fused[token] (0 unless forced)
    scores: Optional[np.ndarray] = None   # c_v for every v, when requested


def weighted(w: float, x) -> np.ndarray:
    """w * x, except that a zero weight gives 0 even where x = -inf: a term weighted by 0 is
    absent from the fusion (p^0 = 1 for every p, a masked p = 0 included), so w_long = 0
    ignores the long logits and beta = 0 the prior, masked entries and all."""
    x = np.asarray(x, dtype=F64)
    if w == 0:
        return np.zeros_like(x)
    return F64(w) * x


def fuse(long_row, short_row, prior, w_long: float, alpha: float, beta: float) -> np.ndarray:
    """l = w_long * l_L + alpha * l_S - beta * l_P  (Sec. 4.3; w_long = 1 in the paper)."""
    f = weighted(w_long, long_row)
    if short_row is not None:
        f = f + weighted(alpha, short_row)
    if prior is not None:
        f = f - weighted(beta, prior)
    return f


def greedy_token(fused: np.ndarray) -> int:
    """argmax over the vocabulary, decided in float32, lowest index on ties."""
    return int(np.argmax(np.asarray(fused, dtype=np.float32)))


def top2_gap(fused: np.ndarray) -> float:
    if fused.shape[0] < 2:
        return float("inf")
    top = np.partition(fused, -2)[-2:]
    return float(top[1] - top[0])


def combine_row(long_row, short_row, prior, w_long: float, alpha: float, beta: float,
                force_token: Optional[int] = None, want_scores: bool = False,
                temperature: float = 0.0, gumbel: Optional[np.ndarray] = None) -> RowResult:
    """Fuse one row of long and short logits, decode and report its statistics.

    With short_row = None the row is decoded from the long logits alone (no prior
    either), as for the first position of Algorithm 1.

    temperature = 0 decodes greedily.  temperature T > 0 samples from softmax(l / T) (the
    Decode step of Algorithm 1 at T; the paper reports T = 0 and T = 1) by the Gumbel-max
    rule: the token is the argmax of l / T + g for the given standard Gumbel noise g [V].
    The statistics then refer to softmax(l / T): lse_fused = log sum exp(l / T),
    logprob = l_tok / T - lse_fused, and the gap and margin are those of l / T + g.
    """
    long_row = np.asarray(long_row, dtype=F64)
    if short_row is None:
        fused = weighted(w_long, long_row)
        lse_s = float("nan")
        a_eff = 0.0
    else:
        fused = fuse(long_row, short_row, prior, w_long, alpha, beta)
        lse_s = logsumexp(short_row)
        a_eff = alpha
    lse_l = logsumexp(long_row)
    if temperature > 0:
        scaled = fused / F64(temperature)
        decide = scaled + np.asarray(gumbel, dtype=F64)     # Gumbel-max
    else:
        scaled = fused
        decide = fused
    lse_f = logsumexp(scaled)
    best = greedy_token(decide)
    tok = best if force_token is None else int(force_token)
    norm = float(weighted(w_long, lse_l)) + (float(weighted(a_eff, lse_s)) if short_row is not None else 0.0)
    res = RowResult(token=tok, score=float(fused[tok] - norm), logprob=float(scaled[tok] - lse_f),
                    gap=top2_gap(decide), lse_long=lse_l, lse_short=lse_s, lse_fused=lse_f,
                    argmax=best, margin=float(decide[best] - decide[tok]))
    if want_scores:
        res.scores = fused - norm
    return res


def combine_rows(long_rows, short_rows, prior, w_long, alpha, beta, want_scores=False):
    """combine_row over every row of [rows, V] inputs."""
    long_rows = np.asarray(long_rows, dtype=F64)
    short_rows = np.asarray(short_rows, dtype=F64)
    return [combine_row(long_rows[i], short_rows[i], prior, w_long, alpha, beta,
                        want_scores=want_scores) for i in range(long_rows.shape[0])]


# ----------------------------------------------------------------------------------------
# adaptive fusion: the local-head and prior weights of a row scaled by a gate that grows with
# the uncertainty of that row's long logits (Sec. 7 proposes weights adjusted by the
# token-level entropy or confidence of the long-context logits; the measures and the gate
# below are this library's reading of that proposal)
# ----------------------------------------------------------------------------------------
UNC_ENTROPY, UNC_MAXPROB = 0, 1


def long_entropy(long_row) -> float:
    """H(p_L) = -sum_v p_v log p_v in nats, p = softmax(l_L); a masked entry (p_v = 0) adds
    nothing (p log p -> 0).  NaN for a row without a finite entry (no distribution)."""
    x = np.asarray(long_row, dtype=F64)
    if not np.isfinite(x).any():
        return float("nan")
    logp = x - logsumexp(x)
    p = np.exp(logp)
    keep = p > 0
    return float(-np.sum(p[keep] * logp[keep]))


def long_max_prob(long_row) -> float:
    """max_v p_v, p = softmax(l_L): the confidence of the long logits in their own argmax.
    NaN for a row without a finite entry."""
    x = np.asarray(long_row, dtype=F64)
    if not np.isfinite(x).any():
        return float("nan")
    return float(np.exp(np.max(x) - logsumexp(x)))


def uncertainty(long_row, measure: int) -> float:
    """u in [0, 1]: 0 when p_L is one-hot, 1 when it is uniform over the whole vocabulary.
    UNC_ENTROPY: H(p_L) / log V.  UNC_MAXPROB: (1 - max p_L) / (1 - 1/V).  V = 1: u = 0.
    A row without a finite entry carries no information: u = 1."""
    V = np.asarray(long_row).shape[0]
    if not np.isfinite(np.asarray(long_row, dtype=F64)).any():
        return 1.0
    if V == 1:
        return 0.0
    if measure == UNC_ENTROPY:
        return long_entropy(long_row) / np.log(F64(V))
    if measure == UNC_MAXPROB:
        return (1.0 - long_max_prob(long_row)) / (1.0 - 1.0 / F64(V))
    raise ValueError(f"unknown uncertainty measure {measure}")


def gate(u: float, h_lo: float, h_hi: float) -> float:
    """g(u) = min(1, max(0, (u - h_lo) / (h_hi - h_lo))), h_lo < h_hi: no local terms while the
    long logits are confident (u <= h_lo), full weights once they are uncertain (u >= h_hi),
    linear between; h_lo < 0 keeps a floor of -h_lo / (h_hi - h_lo) at u = 0."""
    if not h_lo < h_hi:
        raise ValueError("the gate needs h_lo < h_hi")
    return float(min(1.0, max(0.0, (F64(u) - h_lo) / (F64(h_hi) - h_lo))))


def adaptive_gates(long_logits, measure: int, h_lo: float, h_hi: float) -> np.ndarray:
    """The gate of every row (sequence b, position j) of long logits [batch, B, V]."""
    batch = len(long_logits)
    B = np.asarray(long_logits[0]).shape[0]
    g = np.zeros((batch, B), dtype=F64)
    for b in range(batch):
        rows = np.asarray(long_logits[b], dtype=F64)
        for j in range(B):
            g[b, j] = gate(uncertainty(rows[j], measure), h_lo, h_hi)
    return g


# ----------------------------------------------------------------------------------------
# sampling noise: Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as
# easy as 1, 2, 3", SC 2011) keyed by the seed, one counter per 4 vocabulary entries of a row
# ----------------------------------------------------------------------------------------
PHILOX_M0, PHILOX_M1 = 0xD2511F53, 0xCD9E8D57      # round multipliers
PHILOX_W0, PHILOX_W1 = 0x9E3779B9, 0xBB67AE85      # key increments (Weyl sequence)
MASK32 = 0xFFFFFFFF


def philox4x32(counter, key, rounds: int = 10) -> np.ndarray:
    """Philox4x32 over counters [..., 4] (uint32) with key (k0, k1): each round multiplies
    words 0 and 2 by the round constants (64-bit products), and mixes the high halves with
    the other words and the key; the key advances by the Weyl constants between rounds."""
    c = [np.asarray(counter, dtype=np.uint64)[..., i] for i in range(4)]
    k0, k1 = np.uint64(key[0] & MASK32), np.uint64(key[1] & MASK32)
    m = np.uint64(MASK32)
    for r in range(rounds):
        if r > 0:
            k0 = (k0 + np.uint64(PHILOX_W0)) & m
            k1 = (k1 + np.uint64(PHILOX_W1)) & m
        p0 = np.uint64(PHILOX_M0) * c[0]
        p1 = np.uint64(PHILOX_M1) * c[2]
        c = [(p1 >> np.uint64(32)) ^ c[1] ^ k0, p1 & m, (p0 >> np.uint64(32)) ^ c[3] ^ k1, p0 & m]
    return np.stack(c, axis=-1).astype(np.uint32)


def uniforms_row(seed: int, b: int, j: int, V: int) -> np.ndarray:
    """The uniform of vocabulary entry v of row (sequence b, position j): word v % 4 of
    Philox4x32-10 at counter (v // 4, j, b, 0) with key (seed low, seed high), as
    ((x >> 9) + 1/2) / 2^23, which lies in (0, 1) and is exact in float32."""
    q = np.arange((V + 3) // 4, dtype=np.uint64)
    ctr = np.stack([q, np.full_like(q, j), np.full_like(q, b), np.zeros_like(q)], axis=-1)
    x = philox4x32(ctr, (seed & MASK32, (seed >> 32) & MASK32)).reshape(-1)[:V].astype(np.uint64)
    return ((x >> np.uint64(9)).astype(F64) + 0.5) * 2.0 ** -23


def gumbel_row(seed: int, b: int, j: int, V: int) -> np.ndarray:
    """Standard Gumbel noise g = -log(-log u) of a row."""
    return -np.log(-np.log(uniforms_row(seed, b, j, V)))


# ----------------------------------------------------------------------------------------
# App. A: local heads
# ----------------------------------------------------------------------------------------
def gru_cell(x, h, w_ih, w_hh):
    """One step of a bias-free GRU; gate rows of w_ih [3H, d] and w_hh [3H, H] are (r, z, n)."""
    x = np.asarray(x, dtype=F64)
    h = np.asarray(h, dtype=F64)
    H = h.shape[0]
    gi = np.asarray(w_ih, dtype=F64) @ x
    gh = np.asarray(w_hh, dtype=F64) @ h
    r = sigmoid(gi[:H] + gh[:H])
    z = sigmoid(gi[H:2 * H] + gh[H:2 * H])
    n = np.tanh(gi[2 * H:] + r * gh[2 * H:])
    return (1.0 - z) * n + z * h


class RnnHead:
    """r_i = SiLU(W_rank GRU(E_tgt(z_i))),  l_S = W_vocab r_i  (App. A)."""

    def __init__(self, emb, w_ih, w_hh, w_rank, w_vocab):
        self.emb = emb                                # indexed by token; rows become float64
        self.w_ih = np.asarray(w_ih, dtype=F64)
        self.w_hh = np.asarray(w_hh, dtype=F64)
        self.w_rank = np.asarray(w_rank, dtype=F64)
        self.w_vocab = np.asarray(w_vocab, dtype=F64)
        self.H = self.w_hh.shape[1]

    @classmethod
    def from_weights(cls, hw) -> "RnnHead":
        return cls(hw.emb, hw.w_ih, hw.w_hh, hw.w_rank, hw.w_vocab)

    def init_state(self):
        return np.zeros(self.H, dtype=F64)

    def step(self, h, token: int):
        x = np.asarray(self.emb[int(token)], dtype=F64)
        h = gru_cell(x, h, self.w_ih, self.w_hh)
        rho = silu(self.w_rank @ h)
        return h, self.w_vocab @ rho

    def rho(self, h):
        return silu(self.w_rank @ h)


class MarkovHead:
    """r_i = E_M(x_{i-1}),  l_S = r_i W_M^T  with E_M, W_M in R^{V x d_r}  (App. A)."""

    def __init__(self, e_m, w_m):
        self.e_m = e_m
        self.w_m = np.asarray(w_m, dtype=F64)

    def init_state(self):
        return None

    def step(self, state, token: int):
        r = np.asarray(self.e_m[int(token)], dtype=F64)
        return state, self.w_m @ r


# ----------------------------------------------------------------------------------------
# Algorithm 1: one draft block
# ----------------------------------------------------------------------------------------
@dataclasses.dataclass
class DraftResult:
    tokens: np.ndarray          # [batch, B] int32
    score: np.ndarray           # [batch, B]
    logprob: np.ndarray
    gap: np.ndarray
    lse_long: np.ndarray
    lse_short: np.ndarray
    lse_fused: np.ndarray
    argmax: np.ndarray          # the oracle's own decision at each position (given the history)
    margin: np.ndarray          # fused[argmax] - fused[token]


def _at(w, j: int) -> float:
    """A fusion weight at draft position j: one value for all positions, or one per position
    (Sec. 5.6 learns alpha_j and beta_j for each draft position)."""
    return float(w[j]) if np.ndim(w) else float(w)


def draft_block(head, long_logits, last_token: Sequence[int], prior, w_long: float,
                alpha, beta, first_row_long_only: bool = False,
                force: Optional[np.ndarray] = None, sequences: Optional[Sequence[int]] = None,
                temperature: float = 0.0, seed: int = 0,
                gates: Optional[np.ndarray] = None) -> DraftResult:
    """Greedy DeLS-Spec drafting of one block per sequence (Algorithm 1, decoding steps).

    long_logits: [batch, B, V] (anything indexable to rows); last_token: [batch].
    alpha, beta: scalars, or [B] sequences of per-position weights.
    gates: optional [batch, B] factors of the adaptive fusion (adaptive_gates): row (b, j)
    fuses with alpha_j * gates[b, j] and beta_j * gates[b, j].
    temperature > 0 samples every row (see combine_row) with the Gumbel noise of
    gumbel_row(seed, b, j, V).
    force: optional [batch, B] tokens that replace the decoded ones (statistics are then
    reported for the forced token), used to keep a replay aligned after a near-tie.
    sequences: optional subset of sequence indices to run (others are left at zero).
    """
    batch = len(last_token)
    B = np.asarray(long_logits[0]).shape[0]
    seqs = range(batch) if sequences is None else sequences
    out = DraftResult(*[np.zeros((batch, B), dtype=np.int32)] +
                      [np.zeros((batch, B), dtype=F64) for _ in range(6)] +
                      [np.zeros((batch, B), dtype=np.int32), np.zeros((batch, B), dtype=F64)])
    for b in seqs:
        rows = np.asarray(long_logits[b], dtype=F64)
        state = head.init_state()
        u = int(last_token[b])
        for j in range(B):
            f = None if force is None else int(force[b, j])
            g = gumbel_row(seed, b, j, rows.shape[1]) if temperature > 0 else None
            if first_row_long_only and j == 0:
                res = combine_row(rows[0], None, None, w_long, _at(alpha, 0), _at(beta, 0), force_token=f,
                                  temperature=temperature, gumbel=g)
            else:
                state, s = head.step(state, u)
                gf = 1.0 if gates is None else float(gates[b, j])
                res = combine_row(rows[j], s, prior, w_long, _at(alpha, j) * gf, _at(beta, j) * gf,
                                  force_token=f, temperature=temperature, gumbel=g)
            out.tokens[b, j] = res.token
            out.score[b, j] = res.score
            out.logprob[b, j] = res.logprob
            out.gap[b, j] = res.gap
            out.lse_long[b, j] = res.lse_long
            out.lse_short[b, j] = res.lse_short
            out.lse_fused[b, j] = res.lse_fused
            out.argmax[b, j] = res.argmax
            out.margin[b, j] = res.margin
            u = res.token
    return out


def head_rollout(head, start_token: int, steps: int) -> np.ndarray:
    """Greedy rollout of the local head alone (no long logits): each step feeds back its argmax."""
    state = head.init_state()
    u = int(start_token)
    toks = []
    for _ in range(steps):
        state, s = head.step(state, u)
        u = greedy_token(s)
        toks.append(u)
    return np.array(toks, dtype=np.int32)


# ----------------------------------------------------------------------------------------
# verification statistics (Sec. 5.1 tau; App. D rate_i)
# ----------------------------------------------------------------------------------------
def accept_len(draft: np.ndarray, target: np.ndarray) -> np.ndarray:
    """Number of leading positions where the draft equals the target, per sequence."""
    draft = np.asarray(draft)
    target = np.asarray(target)
    batch, B = draft.shape
    out = np.zeros(batch, dtype=np.int32)
    for b in range(batch):
        a = 0
        while a < B and draft[b, a] == target[b, a]:
            a += 1
        out[b] = a
    return out


def tau(accepted: np.ndarray) -> np.ndarray:
    """Acceptance length including the bonus token."""
    return np.asarray(accepted) + 1


def rate_curve(accepted: np.ndarray, B: int) -> np.ndarray:
    """rate_i = P(tau >= i) for i = 1..B+1."""
    t = tau(accepted)
    return np.array([np.mean(t >= i) for i in range(1, B + 2)], dtype=F64)


def tau_gain_ratio(tau_dels: float, tau_base: float, tau_joint: float) -> float:
    """Share of a jointly trained head's tau gain recovered: (t_dels - t_base)/(t_joint - t_base)."""
    return (tau_dels - tau_base) / (tau_joint - tau_base)


# ----------------------------------------------------------------------------------------
# App. A: unigram log-prior with additive smoothing
# ----------------------------------------------------------------------------------------
def unigram_log_prior(counts: np.ndarray, smoothing: float = 1.0) -> np.ndarray:
    c = np.asarray(counts, dtype=F64) + F64(smoothing)
    return np.log(c / np.sum(c))
