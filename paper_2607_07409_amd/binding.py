"""Python binding of libdels (ctypes): argument marshalling only.

Every computation runs in the HIP library; torch tensors only provide device memory
and the stream.  Calling anything here without the built library raises at once.
"""
from __future__ import annotations

import contextlib
import ctypes
import os
from typing import Optional

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdels.so")
STRESS_LIB_PATH = os.path.join(_HERE, "libdels_stress.so")   # test build: pauses before every hand-off

DLS_F32, DLS_BF16 = 0, 1
DLS_HEAD_RNN, DLS_HEAD_MARKOV = 0, 1
DLS_FIRST_ROW_LONG_ONLY = 0x1
DLS_EXCLUSIVE_DEVICE = 0x2
STATUS = {0: "DLS_OK", 1: "DLS_ERR_ARG", 2: "DLS_ERR_SHAPE", 3: "DLS_ERR_DTYPE",
          4: "DLS_ERR_WORKSPACE", 5: "DLS_ERR_DEVICE", 6: "DLS_ERR_HIP"}
STATS_FIELDS = ("score", "logprob", "gap", "lse_long", "lse_short", "lse_fused")


class DlsError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


class Fusion(ctypes.Structure):
    _fields_ = [("w_long", ctypes.c_float), ("alpha", ctypes.c_float), ("beta", ctypes.c_float),
                ("flags", ctypes.c_uint32)]


class Schedule(ctypes.Structure):
    _fields_ = [("alpha", ctypes.c_void_p), ("beta", ctypes.c_void_p)]


class Sampling(ctypes.Structure):
    _fields_ = [("temperature", ctypes.c_float), ("reserved", ctypes.c_uint32), ("seed", ctypes.c_uint64)]


class Adaptive(ctypes.Structure):
    _fields_ = [("measure", ctypes.c_int32), ("h_lo", ctypes.c_float), ("h_hi", ctypes.c_float),
                ("reserved", ctypes.c_uint32)]


UNC_ENTROPY, UNC_MAXPROB = 0, 1
UNC_FIELDS = ("entropy", "max_prob", "u", "gate")


class RowStats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_float) for n in STATS_FIELDS]


class LocalHeadC(ctypes.Structure):
    _fields_ = [("V", ctypes.c_int32), ("d", ctypes.c_int32), ("H", ctypes.c_int32),
                ("r", ctypes.c_int32), ("dtype", ctypes.c_int),
                ("emb", ctypes.c_void_p), ("w_ih", ctypes.c_void_p), ("w_hh", ctypes.c_void_p),
                ("w_rank", ctypes.c_void_p), ("w_vocab", ctypes.c_void_p), ("prepared", ctypes.c_void_p),
                ("kind", ctypes.c_int32), ("reserved", ctypes.c_int32), ("prepared_bytes", ctypes.c_size_t)]


_lib = None
_vp, _i32, _i64, _sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t


def lib() -> ctypes.CDLL:
    """The loaded HIP library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        _lib = load(LIB_PATH)
    return _lib


_loaded = {}


def load(path: str) -> ctypes.CDLL:
    """A build of the library at `path` (the product library, or the delay-injecting test build
    libdels_stress.so), with the argument types of every entry point; loaded once per path."""
    if path not in _loaded:
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is missing: build it with __graft_entry__.build()")
        _loaded[path] = _configure(ctypes.CDLL(path))
    return _loaded[path]


@contextlib.contextmanager
def using(path: str):
    """Route every call of this module to the library at `path` inside the block."""
    global _lib
    prev = lib()
    _lib = load(path)
    try:
        yield _lib
    finally:
        _lib = prev


def _configure(L: ctypes.CDLL) -> ctypes.CDLL:
    """Argument and result types of every entry point of dels.h."""
    L.dls_combine_logits_workspace_size.restype = _sz
    L.dls_combine_logits_workspace_size.argtypes = [_i64, _i32]
    L.dls_combine_logits.restype = ctypes.c_int
    L.dls_combine_logits.argtypes = [_vp, _vp, ctypes.c_int, _vp, _i64, _i32, Fusion, _vp, _vp, _vp,
                                     _vp, _sz, _vp]
    L.dls_draft_block_workspace_size.restype = _sz
    L.dls_draft_block_workspace_size.argtypes = [ctypes.POINTER(LocalHeadC), _i32, _i32]
    L.dls_draft_block.restype = ctypes.c_int
    L.dls_draft_block.argtypes = [ctypes.POINTER(LocalHeadC), _vp, ctypes.c_int, _vp, _vp, _i32, _i32,
                                  Fusion, _vp, _vp, _vp, _sz, _vp]
    L.dls_draft_block_scheduled.restype = ctypes.c_int
    L.dls_draft_block_scheduled.argtypes = [ctypes.POINTER(LocalHeadC), _vp, ctypes.c_int, _vp, _vp, _i32, _i32,
                                            Fusion, Schedule, _vp, _vp, _vp, _sz, _vp]
    L.dls_draft_block_sampled.restype = ctypes.c_int
    L.dls_draft_block_sampled.argtypes = [ctypes.POINTER(LocalHeadC), _vp, ctypes.c_int, _vp, _vp, _i32, _i32,
                                          Fusion, Schedule, Sampling, _vp, _vp, _vp, _sz, _vp]
    L.dls_long_uncertainty_workspace_size.restype = _sz
    L.dls_long_uncertainty_workspace_size.argtypes = [_i64, _i32]
    L.dls_long_uncertainty.restype = ctypes.c_int
    L.dls_long_uncertainty.argtypes = [_vp, ctypes.c_int, _i64, _i32, Adaptive, _vp, _vp, _sz, _vp]
    L.dls_draft_block_adaptive.restype = ctypes.c_int
    L.dls_draft_block_adaptive.argtypes = [ctypes.POINTER(LocalHeadC), _vp, ctypes.c_int, _vp, _vp, _i32, _i32,
                                           Fusion, Schedule, Sampling, Adaptive, _vp, _vp, _vp, _vp, _sz, _vp]
    L.dls_prepare_head_size.restype = _sz
    L.dls_prepare_head_size.argtypes = [ctypes.POINTER(LocalHeadC)]
    L.dls_prepare_head.restype = ctypes.c_int
    L.dls_prepare_head.argtypes = [ctypes.POINTER(LocalHeadC), _vp, _sz, _vp]
    L.dls_draft_block_noalloc.restype = ctypes.c_int
    L.dls_draft_block_noalloc.argtypes = [ctypes.POINTER(LocalHeadC), _vp, ctypes.c_int, _vp, _vp, _i32, _i32,
                                          Fusion, _vp, _vp, _vp]
    L.dls_draft_block_error.restype = ctypes.c_int
    L.dls_draft_block_error.argtypes = [_vp, _sz, _vp, _vp]
    L.dls_draft_block_path.restype = ctypes.c_int
    L.dls_draft_block_path.argtypes = [ctypes.POINTER(LocalHeadC), _i32, _i32, ctypes.c_int, ctypes.c_int]
    L.dls_unigram_log_prior.restype = ctypes.c_int
    L.dls_unigram_log_prior.argtypes = [_vp, _i64, _i32, ctypes.c_float, _vp, _vp, _vp]
    L.dls_accept_len.restype = ctypes.c_int
    L.dls_accept_len.argtypes = [_vp, _vp, _i32, _i32, _vp, _vp]
    L.dls_measure_read.restype = ctypes.c_int
    L.dls_measure_read.argtypes = [_vp, _sz, _vp, _vp]
    L.dls_measure_mfma.restype = ctypes.c_int
    L.dls_measure_mfma.argtypes = [_i32, _i32, ctypes.c_float, _vp, _vp]
    L.dls_status_string.restype = ctypes.c_char_p
    L.dls_status_string.argtypes = [ctypes.c_int]
    L.dls_last_error.restype = ctypes.c_char_p
    L.dls_last_error.argtypes = []
    L.dls_abi_version.restype = ctypes.c_int
    return L


def _check(status: int):
    if status != 0:
        raise DlsError(status, lib().dls_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return DLS_BF16
    if t.dtype == torch.float32:
        return DLS_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def fusion(w_long=1.0, alpha=0.3, beta=0.3, first_row_long_only=False, exclusive_device=False) -> Fusion:
    return Fusion(w_long, alpha, beta, (DLS_FIRST_ROW_LONG_ONLY if first_row_long_only else 0) |
                  (DLS_EXCLUSIVE_DEVICE if exclusive_device else 0))


# -----------------------------------------------------------------------------------
# host data -> device tensors
# -----------------------------------------------------------------------------------
def as_tensor(x, device="cuda") -> torch.Tensor:
    """Device tensor holding exactly the given values (bf16 bit patterns stay bf16)."""
    bits = getattr(x, "bits", None)
    if bits is not None:
        return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(device)
    a = np.ascontiguousarray(x)
    return torch.from_numpy(a).to(device)


class LocalHead:
    """Device copy of a local head (App. A) and its C descriptor: the RNN head (E_tgt, W_ih,
    W_hh, W_rank, W_vocab) or, built with LocalHead.markov, the Markov head (E_M, W_M)."""

    def __init__(self, emb, w_ih, w_hh, w_rank, w_vocab):
        ts = [emb, w_ih, w_hh, w_rank, w_vocab]
        dt = ts[0].dtype
        if any(t.dtype != dt for t in ts):
            raise TypeError("all head tensors must share one dtype")
        self.emb, self.w_ih, self.w_hh, self.w_rank, self.w_vocab = [t.contiguous() for t in ts]
        V, d = self.emb.shape
        H = self.w_hh.shape[1]
        r = self.w_rank.shape[0]
        self.V, self.d, self.H, self.r = V, d, H, r
        self.kind = DLS_HEAD_RNN
        self.prepared = None
        self.c = LocalHeadC(V, d, H, r, _dtype_code(self.emb), self.emb.data_ptr(), self.w_ih.data_ptr(),
                            self.w_hh.data_ptr(), self.w_rank.data_ptr(), self.w_vocab.data_ptr(), None,
                            DLS_HEAD_RNN, 0)

    @classmethod
    def markov(cls, e_m: torch.Tensor, w_m: torch.Tensor) -> "LocalHead":
        """Markov head: rho = E_M[previous token] ([V, r]), l_S = W_M rho ([V, r])."""
        if e_m.dtype != w_m.dtype or e_m.shape != w_m.shape:
            raise TypeError("E_M and W_M must share dtype and shape [V, r]")
        self = cls.__new__(cls)
        self.emb, self.w_vocab = e_m.contiguous(), w_m.contiguous()
        self.w_ih = self.w_hh = self.w_rank = None
        self.V, self.r = self.emb.shape
        self.d = self.H = 0
        self.kind = DLS_HEAD_MARKOV
        self.prepared = None
        self.c = LocalHeadC(self.V, 0, 0, self.r, _dtype_code(self.emb), self.emb.data_ptr(), None, None, None,
                            self.w_vocab.data_ptr(), None, DLS_HEAD_MARKOV, 0)
        return self

    def prepare(self, stream=None) -> "LocalHead":
        """Fill the prepared form (folded input table, operand-ordered weights) on the device."""
        L = lib()
        n = int(L.dls_prepare_head_size(ctypes.byref(self.c)))
        buf = torch.empty(n, dtype=torch.uint8, device=self.emb.device)
        _check(L.dls_prepare_head(ctypes.byref(self.c), _ptr(buf), n, _stream(stream)))
        self.prepared = buf
        self.c.prepared = buf.data_ptr()
        self.c.prepared_bytes = n
        return self

    def unprepare(self) -> "LocalHead":
        self.prepared = None
        self.c.prepared = None
        self.c.prepared_bytes = 0
        return self

    def twin(self) -> "LocalHead":
        """A new descriptor over the same weight tensors (unprepared)."""
        if self.kind == DLS_HEAD_MARKOV:
            return LocalHead.markov(self.emb, self.w_vocab)
        return LocalHead(self.emb, self.w_ih, self.w_hh, self.w_rank, self.w_vocab)

    def path(self, batch: int, B: int, long_dtype=torch.bfloat16, has_prior=False) -> int:
        """1 if dls_draft_block would use the persistent kernel, 0 for per-position launches."""
        code = DLS_BF16 if long_dtype == torch.bfloat16 else DLS_F32
        return int(lib().dls_draft_block_path(ctypes.byref(self.c), batch, B, code, int(bool(has_prior))))

    @classmethod
    def from_weights(cls, hw, device="cuda") -> "LocalHead":
        return cls(*[as_tensor(a, device) for a in (hw.emb, hw.w_ih, hw.w_hh, hw.w_rank, hw.w_vocab)])

    @classmethod
    def markov_from_weights(cls, e_m, w_m, device="cuda") -> "LocalHead":
        return cls.markov(as_tensor(e_m, device), as_tensor(w_m, device))

    def nbytes(self) -> int:
        return sum(t.numel() * t.element_size() for t in (self.emb, self.w_ih, self.w_hh, self.w_rank,
                                                           self.w_vocab) if t is not None)


# -----------------------------------------------------------------------------------
# entry points
# -----------------------------------------------------------------------------------
def combine_logits_workspace_size(rows: int, V: int) -> int:
    return int(lib().dls_combine_logits_workspace_size(rows, V))


def combine_logits(long_logits: torch.Tensor, short_logits: torch.Tensor, prior=None, w_long=1.0, alpha=0.3,
                   beta=0.3, want_stats=True, want_scores=False, out=None, workspace=None, stream=None):
    """Fused combine + argmax of [rows, V] long and short logits.  Returns (tokens, stats, scores);
    stats is a [rows, 6] float32 tensor (fields STATS_FIELDS) or None."""
    L = lib()
    rows, V = long_logits.shape
    dev = long_logits.device
    if out is None:
        tok = torch.empty(rows, dtype=torch.int32, device=dev)
        st = torch.empty((rows, 6), dtype=torch.float32, device=dev) if want_stats else None
        sc = torch.empty((rows, V), dtype=torch.float32, device=dev) if want_scores else None
    else:
        tok, st, sc = out
    need = L.dls_combine_logits_workspace_size(rows, V)
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
    _check(L.dls_combine_logits(_ptr(long_logits), _ptr(short_logits), _dtype_code(long_logits), _ptr(prior),
                                rows, V, fusion(w_long, alpha, beta), _ptr(tok), _ptr(st), _ptr(sc),
                                _ptr(workspace), workspace.numel(), _stream(stream)))
    return tok, st, sc


def draft_block_workspace_size(head: LocalHead, batch: int, B: int) -> int:
    return int(lib().dls_draft_block_workspace_size(ctypes.byref(head.c), batch, B))


def draft_workspace(head: LocalHead, batch: int, B: int, device=None) -> torch.Tensor:
    """A zero-filled draft workspace (the persistent kernel requires zeros before first use)."""
    n = max(256, draft_block_workspace_size(head, batch, B))
    return torch.zeros(n, dtype=torch.uint8, device=device or head.emb.device)


DLS_DRAFT_ERR_STALLED, DLS_DRAFT_ERR_PREPARED = 1, 2


def workspace_error(workspace: Optional[torch.Tensor], stream=None) -> int:
    """The error word of a drafting workspace (None: the scratch of draft_block_noalloc on the
    current device), read through dls_draft_block_error after the work queued on the stream;
    synchronises.  0, DLS_DRAFT_ERR_STALLED or DLS_DRAFT_ERR_PREPARED."""
    dev = workspace.device if workspace is not None else torch.device("cuda", torch.cuda.current_device())
    out = torch.full((1,), -7, dtype=torch.int32, device=dev)
    _check(lib().dls_draft_block_error(_ptr(workspace), 0 if workspace is None else workspace.numel(), _ptr(out),
                                       _stream(stream)))
    return int(out.item())


def draft_block(head: LocalHead, long_logits: torch.Tensor, last_token: Optional[torch.Tensor], prior=None,
                w_long=1.0, alpha=0.3, beta=0.3, first_row_long_only=False, want_stats=True, out=None,
                workspace=None, stream=None, temperature=0.0, seed=0, exclusive_device=False, adaptive=None,
                out_uncertainty=None):
    """Draft one block per sequence.  long_logits [batch, B, V]; returns (tokens [batch, B], stats
    [batch, B, 6] or None).  alpha and beta are scalars or [B] per-position weights.
    temperature 0 decodes greedily; T > 0 samples from softmax(l / T) with the Philox noise of
    `seed` (a 64-bit integer).  exclusive_device: the caller runs nothing else on the device
    during the call (DLS_EXCLUSIVE_DEVICE: an ordinary instead of a cooperative dispatch).
    adaptive = (measure, h_lo, h_hi): adaptive fusion through dls_draft_block_adaptive; the
    return value then has a third element, the rows' uncertainty [batch, B, 4] (UNC_FIELDS)."""
    L = lib()
    batch, B, V = long_logits.shape
    dev = long_logits.device
    if out is None:
        tok = torch.empty((batch, B), dtype=torch.int32, device=dev)
        st = torch.empty((batch, B, 6), dtype=torch.float32, device=dev) if want_stats else None
    else:
        tok, st = out
    if workspace is None:
        workspace = draft_workspace(head, batch, B, dev)
    scheduled = np.ndim(alpha) > 0 or np.ndim(beta) > 0
    sampled = temperature != 0.0
    f = fusion(w_long, 0.0 if np.ndim(alpha) else alpha, 0.0 if np.ndim(beta) else beta, first_row_long_only,
               exclusive_device)
    if scheduled or sampled or adaptive is not None:
        # per-position weights: host arrays of B values (kept alive across the call)
        al = np.ascontiguousarray(alpha, np.float32) if np.ndim(alpha) else None
        be = np.ascontiguousarray(beta, np.float32) if np.ndim(beta) else None
        for arr in (al, be):
            if arr is not None and arr.shape != (B,):
                raise ValueError(f"per-position weights need {B} values")
        sch = Schedule(None if al is None else al.ctypes.data, None if be is None else be.ctypes.data)
        if adaptive is not None:
            unc = out_uncertainty if out_uncertainty is not None else \
                torch.empty((batch, B, 4), dtype=torch.float32, device=dev)
            smp = Sampling(float(temperature), 0, int(seed) & 0xFFFFFFFFFFFFFFFF)
            _check(L.dls_draft_block_adaptive(ctypes.byref(head.c), _ptr(long_logits), _dtype_code(long_logits),
                                              _ptr(last_token), _ptr(prior), batch, B, f, sch, smp,
                                              adaptive_rule(*adaptive), _ptr(unc), _ptr(tok), _ptr(st),
                                              _ptr(workspace), workspace.numel(), _stream(stream)))
            return tok, st, unc
        if sampled:
            smp = Sampling(float(temperature), 0, int(seed) & 0xFFFFFFFFFFFFFFFF)
            _check(L.dls_draft_block_sampled(ctypes.byref(head.c), _ptr(long_logits), _dtype_code(long_logits),
                                             _ptr(last_token), _ptr(prior), batch, B, f, sch, smp, _ptr(tok),
                                             _ptr(st), _ptr(workspace), workspace.numel(), _stream(stream)))
        else:
            _check(L.dls_draft_block_scheduled(ctypes.byref(head.c), _ptr(long_logits), _dtype_code(long_logits),
                                               _ptr(last_token), _ptr(prior), batch, B, f, sch, _ptr(tok),
                                               _ptr(st), _ptr(workspace), workspace.numel(), _stream(stream)))
    else:
        _check(L.dls_draft_block(ctypes.byref(head.c), _ptr(long_logits), _dtype_code(long_logits),
                                 _ptr(last_token), _ptr(prior), batch, B, f, _ptr(tok), _ptr(st), _ptr(workspace),
                                 workspace.numel(), _stream(stream)))
    return tok, st


def adaptive_rule(measure: int, h_lo: float, h_hi: float) -> Adaptive:
    return Adaptive(int(measure), float(h_lo), float(h_hi), 0)


def long_uncertainty_workspace_size(rows: int, V: int) -> int:
    return int(lib().dls_long_uncertainty_workspace_size(rows, V))


def long_uncertainty(long_logits: torch.Tensor, measure: int, h_lo: float, h_hi: float, out=None, workspace=None,
                     stream=None) -> torch.Tensor:
    """Entropy, maximum probability, measure u and gate of every row of long logits [..., V]:
    a float32 tensor [..., 4] (UNC_FIELDS)."""
    L = lib()
    V = long_logits.shape[-1]
    rows = long_logits.numel() // V if V else 0
    dev = long_logits.device
    if out is None:
        out = torch.empty((*long_logits.shape[:-1], 4), dtype=torch.float32, device=dev)
    need = long_uncertainty_workspace_size(rows, V)
    if workspace is None and need:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    _check(L.dls_long_uncertainty(_ptr(long_logits), _dtype_code(long_logits), rows, V,
                                  adaptive_rule(measure, h_lo, h_hi), _ptr(out), _ptr(workspace),
                                  0 if workspace is None else workspace.numel(), _stream(stream)))
    return out


def draft_block_noalloc(head: LocalHead, long_logits: torch.Tensor, last_token: Optional[torch.Tensor], prior=None,
                        w_long=1.0, alpha=0.3, beta=0.3, first_row_long_only=False, want_stats=True, out=None,
                        stream=None, exclusive_device=False):
    """draft_block through dls_draft_block_noalloc: no workspace, the library's per-GPU scratch."""
    L = lib()
    batch, B, V = long_logits.shape
    dev = long_logits.device
    if out is None:
        tok = torch.empty((batch, B), dtype=torch.int32, device=dev)
        st = torch.empty((batch, B, 6), dtype=torch.float32, device=dev) if want_stats else None
    else:
        tok, st = out
    f = fusion(w_long, alpha, beta, first_row_long_only, exclusive_device)
    _check(L.dls_draft_block_noalloc(ctypes.byref(head.c), _ptr(long_logits), _dtype_code(long_logits),
                                     _ptr(last_token), _ptr(prior), batch, B, f, _ptr(tok), _ptr(st),
                                     _stream(stream)))
    return tok, st


def accept_len(draft: torch.Tensor, target: torch.Tensor, out=None, stream=None) -> torch.Tensor:
    """Leading positions where draft == target, per sequence ([batch] int32)."""
    L = lib()
    batch, B = draft.shape
    if out is None:
        out = torch.empty(batch, dtype=torch.int32, device=draft.device)
    _check(L.dls_accept_len(_ptr(draft), _ptr(target), batch, B, _ptr(out), _stream(stream)))
    return out


def unigram_log_prior(tokens: torch.Tensor, V: int, smoothing: float = 1.0, out=None, stream=None):
    """Unigram log-prior of a token stream (App. A): returns (log_prior [V] float32,
    counts [V + 1] int64 holding c(v) and the number of counted tokens)."""
    L = lib()
    n = tokens.numel()
    dev = tokens.device
    if out is None:
        counts = torch.empty(V + 1, dtype=torch.int64, device=dev)
        logp = torch.empty(V, dtype=torch.float32, device=dev)
    else:
        logp, counts = out
    _check(L.dls_unigram_log_prior(_ptr(tokens) if n else None, n, V, smoothing, _ptr(counts), _ptr(logp),
                                   _stream(stream)))
    return logp, counts


MEASURE_READ_WORDS = 8192


def measure_read(buf: torch.Tensor, out=None, stream=None) -> torch.Tensor:
    """Stream every byte of `buf` once (the attainable HBM read bandwidth when it is much
    larger than the caches); returns the DLS_MEASURE_READ_WORDS uint32 checksum words, stored
    as int32, whose XOR is the XOR of the buffer's 32-bit words."""
    L = lib()
    if not buf.is_contiguous():
        raise ValueError("buf must be contiguous")
    if out is None:
        out = torch.empty(MEASURE_READ_WORDS, dtype=torch.int32, device=buf.device)
    _check(L.dls_measure_read(_ptr(buf), buf.numel() * buf.element_size(), _ptr(out), _stream(stream)))
    return out


def measure_mfma(groups: int, iters: int, x: float = 1.0 / 64, out=None, stream=None,
                 device=None) -> torch.Tensor:
    """Run groups * 4 * iters * 4 dense bf16 32x32x16 matrix-core products (32768 flops each);
    returns one float per thread, each exactly iters * 1024 * x^2."""
    L = lib()
    if out is None:
        out = torch.empty(groups * 256, dtype=torch.float32, device=device or "cuda")
    _check(L.dls_measure_mfma(groups, iters, x, _ptr(out), _stream(stream)))
    return out
