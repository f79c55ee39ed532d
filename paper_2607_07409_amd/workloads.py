"""Seeded synthetic inputs with the shapes of the DeLS-Spec drafting workloads.

This module draws random inputs only: long (DFlash) logits, local-head weights,
last accepted tokens, a log unigram prior and target tokens.  It holds none of
the method's arithmetic (no fusion, no GRU, no softmax, no argmax), so both the
CPU oracle side and the HIP side of a test can consume the same inputs.

Shapes follow the paper's setting: Qwen3 vocabulary (V = 151,936), block size
16 (Sec. 5.1), GRU hidden 1024 and rank 256 (App. A, Table 6), embedding
widths 2560 / 4096 / 5120.  bf16 inputs are produced by rounding fp32 draws to
bf16 (round to nearest, ties to even); both sides see the identical bf16
values.
"""
from __future__ import annotations

import dataclasses
import math
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Optional, Tuple

import numpy as np

QWEN3_VOCAB = 151936

# purposes for independent seed streams
_P_WEIGHTS, _P_LONG, _P_LAST, _P_K, _P_TARGET, _P_PRIOR, _P_TRUE = range(7)


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic drafting workload (all sizes explicit)."""
    name: str
    batch: int
    B: int          # draft block length (rows of long logits per sequence)
    V: int          # vocabulary
    dtype: str      # "f32" or "bf16" (long logits and head weights)
    d: int          # target-embedding width (GRU input)
    H: int          # GRU hidden size
    r: int          # low-rank width
    alphas: Tuple[float, ...]   # weight(s) on the short logits
    geom_p: float   # success probability of the target-agreement prefix length
    logits: str     # long-logit recipe: normal2 | onehot | onehot_temp | zipf
    seed: int

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS = {
    # tiny case: the oracle finishes instantly
    "tiny": Workload("tiny", 1, 4, 1024, "f32", 64, 64, 64, (0.5,), 0.5, "normal2", 0),
    # Qwen3-4B shaped, batch 1 (the headline drafting workload)
    "qwen3-4b-b1": Workload("qwen3-4b-b1", 1, 16, QWEN3_VOCAB, "bf16", 2560, 1024, 256,
                            (0.5,), 0.5, "onehot", 1),
    # Qwen3-8B shaped, batch 1, alpha sweep
    "qwen3-8b-b1": Workload("qwen3-8b-b1", 1, 16, QWEN3_VOCAB, "bf16", 4096, 1024, 256,
                            (0.25, 0.5, 1.0), 0.3, "onehot", 2),
    # serving batch 16, per-row temperature on the long logits
    "qwen3-8b-b16": Workload("qwen3-8b-b16", 16, 16, QWEN3_VOCAB, "bf16", 4096, 1024, 256,
                             (0.5,), 0.5, "onehot_temp", 3),
    # batch 64, Zipf-ranked bias on the long logits
    "b64-d5120": Workload("b64-d5120", 64, 16, QWEN3_VOCAB, "bf16", 5120, 1024, 256,
                          (0.5,), 0.5, "zipf", 4),
}
WORKLOAD_ORDER = ["tiny", "qwen3-4b-b1", "qwen3-8b-b1", "qwen3-8b-b16", "b64-d5120"]


def _rng(seed: int, purpose: int, *extra: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence(entropy=seed, spawn_key=(purpose,) + extra))


_CHUNK_ROWS_ELEMS = 1 << 22      # elements per independently seeded chunk
_THREADS = max(1, min(16, len(os.sched_getaffinity(0))))


def _normal_table(shape, scale: float, dtype: str, seed: int, purpose: int, idx: int):
    """N(0, scale^2) table of the given 2-D shape, generated in row chunks with fixed seeds
    (the values do not depend on the number of threads), stored as fp32 or bf16."""
    rows, cols = shape
    per = max(1, _CHUNK_ROWS_ELEMS // max(cols, 1))
    starts = list(range(0, rows, per))
    if dtype == "bf16":
        out = np.empty((rows, cols), dtype=np.uint16)
    else:
        out = np.empty((rows, cols), dtype=np.float32)

    def work(ci):
        r0 = starts[ci]
        r1 = min(rows, r0 + per)
        x = _rng(seed, purpose, idx, ci).standard_normal((r1 - r0, cols), dtype=np.float32)
        x *= np.float32(scale)
        out[r0:r1] = f32_to_bf16_bits(x) if dtype == "bf16" else x

    with ThreadPoolExecutor(_THREADS) as ex:
        list(ex.map(work, range(len(starts))))
    return Bf16Array(out) if dtype == "bf16" else out


# ----------------------------------------------------------------------------------------
# bf16 storage
# ----------------------------------------------------------------------------------------
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round finite fp32 values to bf16 (nearest, ties to even); returns uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    return ((u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


class Bf16Array:
    """A bf16 tensor kept as its bit patterns; indexing returns exact fp32 values."""

    def __init__(self, bits: np.ndarray):
        assert bits.dtype == np.uint16
        self.bits = np.ascontiguousarray(bits)

    @classmethod
    def from_f32(cls, x: np.ndarray) -> "Bf16Array":
        return cls(f32_to_bf16_bits(x))

    @property
    def shape(self):
        return self.bits.shape

    @property
    def nbytes(self):
        return self.bits.nbytes

    def __getitem__(self, idx):
        return bf16_bits_to_f32(np.asarray(self.bits[idx]))

    def __array__(self, dtype=None, copy=None):
        v = bf16_bits_to_f32(self.bits)
        return v if dtype is None else v.astype(dtype)

    def __len__(self):
        return self.bits.shape[0]


def _store(x: np.ndarray, dtype: str):
    if dtype == "bf16":
        return Bf16Array.from_f32(x)
    if dtype == "f32":
        return np.ascontiguousarray(x, dtype=np.float32)
    raise ValueError(dtype)


def values_f32(a) -> np.ndarray:
    """fp32 values of a stored tensor (exact)."""
    return np.asarray(a, dtype=np.float32)


# ----------------------------------------------------------------------------------------
# local head weights (GRU head of App. A: E_tgt, W_ih, W_hh, W_rank, W_vocab)
# ----------------------------------------------------------------------------------------
@dataclasses.dataclass
class HeadWeights:
    V: int
    d: int
    H: int
    r: int
    dtype: str
    emb: object      # [V, d]
    w_ih: object     # [3H, d], gate rows (r, z, n)
    w_hh: object     # [3H, H], gate rows (r, z, n)
    w_rank: object   # [r, H]
    w_vocab: object  # [V, r]

    def arrays(self):
        return dict(emb=self.emb, w_ih=self.w_ih, w_hh=self.w_hh, w_rank=self.w_rank,
                    w_vocab=self.w_vocab)


STRESS_VOCAB_GAIN = 10.0


def make_head(wl: Workload, init: str = "baseline", seed: Optional[int] = None) -> HeadWeights:
    """Random local-head weights.

    baseline: every weight ~ N(0, 0.02^2)  (short logits of order 1e-3).
    stress:   E ~ N(0,1), W_ih ~ N(0,1/d), W_hh, W_rank ~ N(0,1/H),
              W_vocab ~ N(0, g^2/r) with g = STRESS_VOCAB_GAIN, so that the short
              logits have a spread of a few units and change many argmaxes.
    """
    seed = wl.seed if seed is None else seed
    V, d, H, r = wl.V, wl.d, wl.H, wl.r
    if init == "baseline":
        sd = dict(emb=0.02, w_ih=0.02, w_hh=0.02, w_rank=0.02, w_vocab=0.02)
    elif init == "stress":
        sd = dict(emb=1.0, w_ih=1.0 / math.sqrt(d), w_hh=1.0 / math.sqrt(H),
                  w_rank=1.0 / math.sqrt(H), w_vocab=STRESS_VOCAB_GAIN / math.sqrt(r))
    elif init == "zero":
        sd = dict(emb=0.0, w_ih=0.0, w_hh=0.0, w_rank=0.0, w_vocab=0.0)
    else:
        raise ValueError(init)
    shapes = dict(emb=(V, d), w_ih=(3 * H, d), w_hh=(3 * H, H), w_rank=(r, H), w_vocab=(V, r))
    out = {}
    for i, name in enumerate(["emb", "w_ih", "w_hh", "w_rank", "w_vocab"]):
        out[name] = _normal_table(shapes[name], sd[name], wl.dtype, seed, _P_WEIGHTS, i)
    return HeadWeights(V, d, H, r, wl.dtype, **out)


def make_markov_head(V: int, dr: int, dtype: str, seed: int, scale: float = 1.0):
    """Random Markov-head tables E_M [V, dr] and W_M [V, dr] (App. A)."""
    em = _rng(seed, _P_WEIGHTS, 10).standard_normal((V, dr), dtype=np.float32) * np.float32(scale)
    wm = _rng(seed, _P_WEIGHTS, 11).standard_normal((V, dr), dtype=np.float32) * np.float32(scale)
    return _store(em, dtype), _store(wm, dtype)


# ----------------------------------------------------------------------------------------
# long (DFlash) logits
# ----------------------------------------------------------------------------------------
def zipf_ranks(V: int, seed: int) -> np.ndarray:
    """A seeded permutation giving each token a frequency rank in 1..V."""
    perm = _rng(seed, _P_LONG, 999).permutation(V)
    ranks = np.empty(V, dtype=np.int64)
    ranks[perm] = np.arange(1, V + 1)
    return ranks


def make_token_stream(n: int, V: int, seed: int, s: float = 1.1) -> np.ndarray:
    """n int32 token ids with Zipf(s) frequencies over a seeded ranking of the vocabulary
    (inverse-CDF draws, in chunks)."""
    order = np.argsort(zipf_ranks(V, seed))          # token of rank k + 1
    cdf = np.cumsum(1.0 / np.arange(1, V + 1, dtype=np.float64) ** s)
    cdf /= cdf[-1]
    g = _rng(seed, _P_LONG, 998)
    out = np.empty(n, dtype=np.int32)
    step = 1 << 22
    for i in range(0, n, step):
        m = min(step, n - i)
        out[i:i + m] = order[np.minimum(np.searchsorted(cdf, g.random(m), side="right"), V - 1)]
    return out


def make_long_logits(wl: Workload, seed: Optional[int] = None):
    """[batch, B, V] long logits following the workload's recipe."""
    seed = wl.seed if seed is None else seed
    bt, B, V = wl.batch, wl.B, wl.V
    if wl.logits == "normal2":
        x = _rng(seed, _P_LONG).standard_normal((bt, B, V), dtype=np.float32) * np.float32(2.0)
        return _store(x, wl.dtype)
    if wl.logits not in ("onehot", "onehot_temp", "zipf"):
        raise ValueError(wl.logits)
    bias = None
    if wl.logits == "zipf":
        bias = (-1.1 * np.log(zipf_ranks(V, seed).astype(np.float64))).astype(np.float32)
    out = np.empty((bt, B, V), dtype=np.uint16 if wl.dtype == "bf16" else np.float32)

    def work(b):   # one independent stream per sequence
        g = _rng(seed, _P_LONG, b)
        x = g.standard_normal((B, V), dtype=np.float32) * np.float32(3.0)
        if bias is not None:
            x += bias
        else:
            true = g.integers(0, V, size=B)
            x[np.arange(B), true] += np.float32(8.0)
            if wl.logits == "onehot_temp":
                x /= g.uniform(0.5, 2.0, size=(B, 1)).astype(np.float32)
        out[b] = f32_to_bf16_bits(x) if wl.dtype == "bf16" else x

    with ThreadPoolExecutor(_THREADS) as ex:
        list(ex.map(work, range(bt)))
    return Bf16Array(out) if wl.dtype == "bf16" else out


def mask_long_logits(long, frac: float, seed: int, single=()):
    """A copy of stored long logits [batch, B, V] with a seeded fraction of the entries set to -inf
    (masked tokens); each (b, j) in `single` keeps one finite entry only, at a seeded token.
    Returns (masked copy, {(b, j): the kept token})."""
    g = _rng(seed, 40)
    bf = isinstance(long, Bf16Array)
    arr = long.bits.copy() if bf else np.array(long, dtype=np.float32, copy=True)
    neg_inf = np.uint16(0xFF80) if bf else np.float32(-np.inf)
    arr[g.random(arr.shape) < frac] = neg_inf
    kept = {}
    for (b, j) in single:
        t = int(g.integers(0, arr.shape[2]))
        keep = arr[b, j, t]
        if bf and keep == neg_inf:
            keep = np.uint16(0x3F80)          # 1.0
        elif not bf and not np.isfinite(keep):
            keep = np.float32(1.0)
        arr[b, j, :] = neg_inf
        arr[b, j, t] = keep
        kept[(b, j)] = t
    return (Bf16Array(arr) if bf else arr), kept


def make_zipf_log_prior(V: int, seed: int, s: float = 1.1) -> np.ndarray:
    """[V] fp32 log unigram prior of a Zipf(s) law over seeded ranks (a normalised log-distribution)."""
    ranks = zipf_ranks(V, seed).astype(np.float64)
    logw = -s * np.log(ranks)
    m = logw.max()
    lz = m + np.log(np.sum(np.exp(logw - m)))
    return (logw - lz).astype(np.float32)


def make_last_token(wl: Workload, seed: Optional[int] = None) -> np.ndarray:
    seed = wl.seed if seed is None else seed
    return _rng(seed, _P_LAST).integers(0, wl.V, size=wl.batch).astype(np.int32)


def make_targets(draft: np.ndarray, wl: Workload, seed: Optional[int] = None,
                 k: Optional[np.ndarray] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Target tokens whose first k positions equal `draft`, k ~ Geometric(p) failures, capped at B.

    Positions from k on are uniform over V (an accidental match is possible).
    Returns (targets [batch, B] int32, k [batch] int32).
    """
    seed = wl.seed if seed is None else seed
    bt, B = draft.shape
    if k is None:
        k = _rng(seed, _P_K).geometric(wl.geom_p, size=bt) - 1
    k = np.minimum(np.asarray(k, dtype=np.int64), B)
    t = _rng(seed, _P_TARGET).integers(0, wl.V, size=(bt, B))
    for b in range(bt):
        t[b, :k[b]] = draft[b, :k[b]]
    return t.astype(np.int32), k.astype(np.int32)


def paper_shaped_k(n: int, seed: int) -> np.ndarray:
    """Accepted-draft counts whose survival curve follows the DeLS-Spec column of the paper's
    acceptance-rate table (App. D): P(tau >= i) for i = 1..16, tau = accepted + 1."""
    surv = np.array([1.0, .8145, .6510, .5269, .4380, .3699, .3163, .2749, .2411, .2124,
                     .1885, .1683, .1495, .1342, .1196, .1062])
    pmf = np.append(surv[:-1] - surv[1:], surv[-1])  # P(tau = i), i = 1..16
    tau = _rng(seed, _P_K, 7).choice(np.arange(1, 17), size=n, p=pmf / pmf.sum())
    return (tau - 1).astype(np.int32)


# ----------------------------------------------------------------------------------------
# one complete problem instance
# ----------------------------------------------------------------------------------------
@dataclasses.dataclass
class Problem:
    wl: Workload
    head: HeadWeights
    long_logits: object      # [batch, B, V]
    last_token: np.ndarray   # [batch]
    prior: Optional[np.ndarray]


def make_problem(wl: Workload, init: str = "baseline", with_prior: bool = False) -> Problem:
    return Problem(wl, make_head(wl, init), make_long_logits(wl), make_last_token(wl),
                   make_zipf_log_prior(wl.V, wl.seed) if with_prior else None)


def make_logit_rows(rows: int, V: int, dtype: str, seed: int, recipe: str = "onehot", scale: float = 3.0,
                    purpose: int = 20):
    """[rows, V] logits: 'normal' = N(0, scale^2); 'onehot' = scale*N(0,1) + 8 on one random token."""
    out = np.empty((rows, V), dtype=np.uint16 if dtype == "bf16" else np.float32)

    def work(i):
        g = _rng(seed, purpose, i)
        x = g.standard_normal(V, dtype=np.float32) * np.float32(scale)
        if recipe == "onehot":
            x[g.integers(0, V)] += np.float32(8.0)
        elif recipe != "normal":
            raise ValueError(recipe)
        out[i] = f32_to_bf16_bits(x) if dtype == "bf16" else x

    with ThreadPoolExecutor(_THREADS) as ex:
        list(ex.map(work, range(rows)))
    return Bf16Array(out) if dtype == "bf16" else out
