"""Host-side tests of the C ABI: the library loads, exports every function declared in
include/dels.h, its structs have the layout a C compiler gives them, and bad arguments
are rejected with status codes before any device call.  No kernel is launched.
"""
import ctypes
import os
import re
import subprocess

import pytest
import torch

from paper_2607_07409_amd import binding as b

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dels.h")
HAS_GPU = torch.cuda.is_available()

# fake, 256-byte-aligned device addresses: only ever passed to calls that fail validation
# (or, without a GPU, stop at the device check)
FAKE = [ctypes.c_void_p(0x7f0000000000 + 0x100000 * i) for i in range(16)]


def _declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(dls_[a-z_]+)\s*\(", src)))


def test_exports_every_declared_function():
    L = b.lib()
    names = _declared_functions()
    assert {"dls_draft_block", "dls_combine_logits", "dls_accept_len"} <= set(names)
    for n in names:
        assert hasattr(L, n), n
    out = subprocess.run(["nm", "-D", "--defined-only", b.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r"\bT (dls_\w+)", out))
    assert set(names) <= exported


def test_struct_layout_matches_c(tmp_path):
    prog = tmp_path / "lay.c"
    prog.write_text(f'''#include <stdio.h>
#include <stddef.h>
#include "{HEADER}"
int main(void) {{
  printf("%zu %zu %zu %zu %zu %zu %zu %zu %zu %zu %zu %zu %zu %zu %zu\\n", sizeof(dls_local_head),
         sizeof(dls_row_stats), sizeof(dls_fusion), offsetof(dls_local_head, dtype), offsetof(dls_local_head, emb),
         offsetof(dls_local_head, w_vocab), offsetof(dls_fusion, flags), offsetof(dls_local_head, kind),
         sizeof(dls_sampling), offsetof(dls_sampling, seed), offsetof(dls_local_head, prepared_bytes),
         sizeof(dls_adaptive), offsetof(dls_adaptive, h_hi), sizeof(dls_row_uncertainty),
         offsetof(dls_row_uncertainty, gate));
  return 0;
}}''')
    exe = tmp_path / "lay"
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", str(prog), "-o", str(exe)], check=True)
    got = [int(x) for x in subprocess.run([str(exe)], capture_output=True, text=True).stdout.split()]
    want = [ctypes.sizeof(b.LocalHeadC), ctypes.sizeof(b.RowStats), ctypes.sizeof(b.Fusion),
            b.LocalHeadC.dtype.offset, b.LocalHeadC.emb.offset, b.LocalHeadC.w_vocab.offset,
            b.Fusion.flags.offset, b.LocalHeadC.kind.offset, ctypes.sizeof(b.Sampling), b.Sampling.seed.offset,
            b.LocalHeadC.prepared_bytes.offset, ctypes.sizeof(b.Adaptive), b.Adaptive.h_hi.offset, 16,
            4 * b.UNC_FIELDS.index("gate")]
    assert got == want


def test_header_compiles_as_cpp(tmp_path):
    src = tmp_path / "h.cpp"
    src.write_text(f'#include "{HEADER}"\nint main() {{ return dls_abi_version() == 4 ? 0 : 1; }}\n')
    subprocess.run(["g++", "-std=c++17", "-Wall", "-Werror", "-c", str(src), "-o", str(tmp_path / "h.o")],
                   check=True)


def test_status_strings():
    L = b.lib()
    for code, name in b.STATUS.items():
        assert L.dls_status_string(code).decode() == name
    assert L.dls_status_string(99).decode() == "DLS_UNKNOWN_STATUS"
    assert L.dls_abi_version() == 4


def _head(**kw):
    h = dict(V=1000, d=64, H=32, r=16, dtype=b.DLS_BF16, emb=FAKE[0].value, w_ih=FAKE[1].value,
             w_hh=FAKE[2].value, w_rank=FAKE[3].value, w_vocab=FAKE[4].value)
    h.update(kw)
    return b.LocalHeadC(**h)


def _markov(**kw):
    """A Markov head: only E_M (emb) and W_M (w_vocab); d, H and the GRU pointers unused."""
    h = dict(V=1000, d=0, H=0, r=16, dtype=b.DLS_BF16, emb=FAKE[0].value, w_ih=None, w_hh=None, w_rank=None,
             w_vocab=FAKE[4].value, kind=b.DLS_HEAD_MARKOV)
    h.update(kw)
    return b.LocalHeadC(**h)


def _draft(head, **kw):
    a = dict(long=FAKE[5], ldt=b.DLS_BF16, last=FAKE[6], prior=None, batch=2, B=4, f=b.fusion(),
             tok=FAKE[7], st=FAKE[8], ws=FAKE[9], wsb=1 << 30)
    a.update(kw)
    L = b.lib()
    rc = L.dls_draft_block(ctypes.byref(head), a["long"], a["ldt"], a["last"], a["prior"], a["batch"], a["B"],
                           a["f"], a["tok"], a["st"], a["ws"], a["wsb"], None)
    return rc, L.dls_last_error().decode()


def _sampled(head, temperature, reserved=0, seed=0, **kw):
    a = dict(long=FAKE[5], ldt=b.DLS_BF16, last=FAKE[6], prior=None, batch=2, B=4, f=b.fusion(),
             tok=FAKE[7], st=FAKE[8], ws=FAKE[9], wsb=1 << 30)
    a.update(kw)
    L = b.lib()
    rc = L.dls_draft_block_sampled(ctypes.byref(head), a["long"], a["ldt"], a["last"], a["prior"], a["batch"],
                                   a["B"], a["f"], b.Schedule(None, None), b.Sampling(temperature, reserved, seed),
                                   a["tok"], a["st"], a["ws"], a["wsb"], None)
    return rc, L.dls_last_error().decode()


def test_sampled_draft_rejects_bad_temperature():
    for T in (-1.0, float("nan"), float("inf"), 1e-45, 1e31):
        rc, msg = _sampled(_head(), T)
        assert b.STATUS[rc] == "DLS_ERR_ARG", (T, msg)
        assert "temperature" in msg
    rc, msg = _sampled(_head(), 1.0, reserved=1)
    assert b.STATUS[rc] == "DLS_ERR_ARG" and "reserved" in msg
    # argument checks of the plain entry point apply too
    assert b.STATUS[_sampled(_head(V=0), 1.0)[0]] == "DLS_ERR_SHAPE"
    assert _sampled(_head(), 1.0, batch=0, long=None, tok=None)[0] == 0


@pytest.mark.skipif(HAS_GPU, reason="would launch on fake pointers when a GPU is present")
def test_sampled_valid_arguments_stop_at_device_check():
    for T in (0.0, 1.0, 0.25, 1e-6):
        rc, msg = _sampled(_head(), T, seed=(1 << 64) - 1)
        assert b.STATUS[rc] == "DLS_ERR_DEVICE", (T, msg)


def test_draft_block_rejects_bad_arguments():
    E = {v: k for k, v in b.STATUS.items()}
    cases = [
        (dict(head=_head(V=0)), "DLS_ERR_SHAPE"),
        (dict(head=_head(d=12)), "DLS_ERR_SHAPE"),
        (dict(head=_head(H=4)), "DLS_ERR_SHAPE"),
        (dict(head=_head(r=1024)), "DLS_ERR_SHAPE"),
        (dict(head=_head(dtype=7)), "DLS_ERR_DTYPE"),
        (dict(head=_head(w_rank=None)), "DLS_ERR_ARG"),
        (dict(head=_head(w_vocab=FAKE[4].value + 2)), "DLS_ERR_ARG"),
        (dict(head=_head(), ldt=5), "DLS_ERR_DTYPE"),
        (dict(head=_head(), batch=257), "DLS_ERR_SHAPE"),
        (dict(head=_head(), B=65), "DLS_ERR_SHAPE"),
        (dict(head=_head(), long=None), "DLS_ERR_ARG"),
        (dict(head=_head(), last=None), "DLS_ERR_ARG"),
        (dict(head=_head(), tok=None), "DLS_ERR_ARG"),
        (dict(head=_head(), long=ctypes.c_void_p(FAKE[5].value + 4)), "DLS_ERR_ARG"),
        (dict(head=_head(), wsb=16), "DLS_ERR_WORKSPACE"),
        (dict(head=_head(), ws=None), "DLS_ERR_ARG"),
        (dict(head=_head(), f=b.Fusion(1.0, float("nan"), 0.0, 0)), "DLS_ERR_ARG"),
        (dict(head=_head(), f=b.Fusion(1.0, 0.5, 0.0, 0x10)), "DLS_ERR_ARG"),
        (dict(head=_head(kind=7)), "DLS_ERR_ARG"),
        (dict(head=_markov(r=12)), "DLS_ERR_SHAPE"),
        (dict(head=_markov(emb=None)), "DLS_ERR_ARG"),
        (dict(head=_markov(w_vocab=None)), "DLS_ERR_ARG"),
    ]
    for kw, want in cases:
        head = kw.pop("head")
        rc, msg = _draft(head, **kw)
        assert b.STATUS[rc] == want, (kw, msg)
        assert msg
    # empty work is a no-op, even with NULL pointers
    assert _draft(_head(), batch=0, long=None, tok=None)[0] == 0
    assert _draft(_head(), B=0, long=None, tok=None)[0] == 0


@pytest.mark.skipif(HAS_GPU, reason="would launch on fake pointers when a GPU is present")
def test_valid_arguments_stop_at_device_check():
    rc, msg = _draft(_head())
    assert b.STATUS[rc] == "DLS_ERR_DEVICE", msg
    rc, msg = _draft(_markov())          # a valid Markov head with d = H = 0 and no GRU tensors
    assert b.STATUS[rc] == "DLS_ERR_DEVICE", msg
    # the literal first-row reading does not need the last token
    rc, _ = _draft(_head(), last=None, f=b.fusion(first_row_long_only=True))
    assert b.STATUS[rc] == "DLS_ERR_DEVICE"
    rc, _ = _draft(_head(), f=b.fusion(first_row_long_only=True, exclusive_device=True))   # both flags known
    assert b.STATUS[rc] == "DLS_ERR_DEVICE"
    L = b.lib()
    rc = L.dls_combine_logits(FAKE[0], FAKE[1], b.DLS_BF16, None, 4, 1000, b.fusion(), FAKE[2], None, None,
                              FAKE[3], 1 << 20, None)
    assert b.STATUS[rc] == "DLS_ERR_DEVICE"
    assert b.STATUS[L.dls_accept_len(FAKE[0], FAKE[1], 4, 16, FAKE[2], None)] == "DLS_ERR_DEVICE"


def test_combine_rejects_bad_arguments():
    L = b.lib()

    def call(long=FAKE[0], short=FAKE[1], dt=b.DLS_BF16, prior=None, rows=4, V=1000, f=None, tok=FAKE[2],
             ws=FAKE[3], wsb=1 << 20, scores=None):
        return b.STATUS[L.dls_combine_logits(long, short, dt, prior, rows, V, f or b.fusion(), tok, None, scores,
                                             ws, wsb, None)]

    assert call(dt=3) == "DLS_ERR_DTYPE"
    assert call(V=0) == "DLS_ERR_SHAPE"
    assert call(rows=-1) == "DLS_ERR_SHAPE"
    assert call(short=None) == "DLS_ERR_ARG"
    assert call(tok=None) == "DLS_ERR_ARG"
    assert call(long=ctypes.c_void_p(FAKE[0].value + 8)) == "DLS_ERR_ARG"
    assert call(scores=ctypes.c_void_p(FAKE[4].value + 4)) == "DLS_ERR_ARG"
    assert call(prior=ctypes.c_void_p(FAKE[5].value + 2)) == "DLS_ERR_ARG"
    assert call(rows=4096, V=151936, wsb=16) == "DLS_ERR_WORKSPACE"
    assert call(f=b.Fusion(float("inf"), 0.5, 0.0, 0)) == "DLS_ERR_ARG"
    assert call(rows=0, long=None, short=None, tok=None) == "DLS_OK"


def test_accept_len_rejects_bad_arguments():
    L = b.lib()
    assert b.STATUS[L.dls_accept_len(FAKE[0], FAKE[1], -1, 16, FAKE[2], None)] == "DLS_ERR_SHAPE"
    assert b.STATUS[L.dls_accept_len(FAKE[0], FAKE[1], 4, 5000, FAKE[2], None)] == "DLS_ERR_SHAPE"
    assert b.STATUS[L.dls_accept_len(None, FAKE[1], 4, 16, FAKE[2], None)] == "DLS_ERR_ARG"
    assert b.STATUS[L.dls_accept_len(FAKE[0], FAKE[1], 4, 16, None, None)] == "DLS_ERR_ARG"
    assert b.STATUS[L.dls_accept_len(None, None, 0, 16, None, None)] == "DLS_OK"


def test_workspace_size_queries():
    L = b.lib()
    assert L.dls_combine_logits_workspace_size(0, 100) == 0
    assert L.dls_combine_logits_workspace_size(16, 151936) > 0
    h = _head(V=151936, d=2560, H=1024, r=256)
    s1 = L.dls_draft_block_workspace_size(ctypes.byref(h), 1, 16)
    s64 = L.dls_draft_block_workspace_size(ctypes.byref(h), 64, 16)
    assert 0 < s1 < s64
    assert L.dls_draft_block_workspace_size(None, 1, 16) == 0


def test_markov_sizes():
    """A Markov head needs no GRU buffers: its prepared form is W_M in operand order only."""
    L = b.lib()
    m = _markov(V=151936, r=256)
    assert L.dls_draft_block_workspace_size(ctypes.byref(m), 1, 16) > 0
    pm = L.dls_prepare_head_size(ctypes.byref(m))
    nt = (151936 + 15) // 16
    assert nt * 16 * 256 * 2 <= pm <= nt * 16 * 256 * 2 + 4096
    h = _head(V=151936, d=2560, H=1024, r=256)
    assert L.dls_prepare_head_size(ctypes.byref(h)) > pm + 151936 * 3 * 1024 * 4


def test_unigram_prior_rejects_bad_arguments():
    L = b.lib()

    def call(tokens=FAKE[0], n=100, V=1000, smoothing=1.0, counts=FAKE[1], out=FAKE[2]):
        return b.STATUS[L.dls_unigram_log_prior(tokens, n, V, smoothing, counts, out, None)]

    assert call(n=-1) == "DLS_ERR_SHAPE"
    assert call(V=0) == "DLS_ERR_SHAPE"
    assert call(smoothing=-1.0) == "DLS_ERR_ARG"
    assert call(smoothing=float("nan")) == "DLS_ERR_ARG"
    assert call(tokens=None) == "DLS_ERR_ARG"
    assert call(counts=None) == "DLS_ERR_ARG"
    assert call(counts=ctypes.c_void_p(FAKE[1].value + 4)) == "DLS_ERR_ARG"
    if not HAS_GPU:
        assert call() == "DLS_ERR_DEVICE"
        assert call(tokens=None, n=0) == "DLS_ERR_DEVICE"


def _noalloc(head, **kw):
    a = dict(long=FAKE[5], ldt=b.DLS_BF16, last=FAKE[6], prior=None, batch=2, B=4, f=b.fusion(),
             tok=FAKE[7], st=FAKE[8])
    a.update(kw)
    L = b.lib()
    rc = L.dls_draft_block_noalloc(ctypes.byref(head), a["long"], a["ldt"], a["last"], a["prior"], a["batch"], a["B"],
                                   a["f"], a["tok"], a["st"], None)
    return rc, L.dls_last_error().decode()


def test_noalloc_rejects_bad_arguments_and_oversized_calls():
    """The allocation-free entry point applies the checks of dls_draft_block and refuses calls whose
    workspace would exceed its fixed scratch array (32 MiB), before any device call."""
    assert b.STATUS[_noalloc(_head(V=0))[0]] == "DLS_ERR_SHAPE"
    assert b.STATUS[_noalloc(_head(), tok=None)[0]] == "DLS_ERR_ARG"
    assert b.STATUS[_noalloc(_head(), batch=257)[0]] == "DLS_ERR_SHAPE"
    assert _noalloc(_head(), batch=0, long=None, tok=None)[0] == 0
    L = b.lib()
    big = _head(V=151936, d=4096, H=4096, r=256)
    need = L.dls_draft_block_workspace_size(ctypes.byref(big), 256, 64)
    assert need > 32 << 20
    rc, msg = _noalloc(big, batch=256, B=64)
    assert b.STATUS[rc] == "DLS_ERR_WORKSPACE" and "scratch" in msg, msg
    # the Qwen3-shaped heads fit up to batch 64 at B = 16
    q = _head(V=151936, d=5120, H=1024, r=256)
    assert L.dls_draft_block_workspace_size(ctypes.byref(q), 64, 16) <= 32 << 20


@pytest.mark.skipif(HAS_GPU, reason="would launch on fake pointers when a GPU is present")
def test_noalloc_valid_arguments_stop_at_device_check():
    rc, msg = _noalloc(_head())
    assert b.STATUS[rc] == "DLS_ERR_DEVICE", msg


def test_prepared_buffer_size_is_checked():
    """A prepared buffer smaller than the head's prepared form, or misaligned, is refused on the
    host (the kernel would read past its end)."""
    L = b.lib()
    h = _head(V=4096, d=64, H=64, r=128)
    need = L.dls_prepare_head_size(ctypes.byref(h))
    assert need > 0
    small = _head(V=4096, d=64, H=64, r=128, prepared=FAKE[10].value, prepared_bytes=need - 1)
    rc, msg = _draft(small)
    assert b.STATUS[rc] == "DLS_ERR_WORKSPACE" and "prepared" in msg, msg
    assert L.dls_draft_block_path(ctypes.byref(small), 2, 4, b.DLS_BF16, 0) == -1
    assert b.STATUS[_noalloc(small)[0]] == "DLS_ERR_WORKSPACE"
    skew = _head(V=4096, d=64, H=64, r=128, prepared=FAKE[10].value + 16, prepared_bytes=need)
    assert b.STATUS[_draft(skew)[0]] == "DLS_ERR_ARG"
    ok = _head(V=4096, d=64, H=64, r=128, prepared=FAKE[10].value, prepared_bytes=need)
    if not HAS_GPU:
        assert b.STATUS[_draft(ok)[0]] == "DLS_ERR_DEVICE"


def test_error_query_rejects_bad_arguments():
    L = b.lib()
    assert b.STATUS[L.dls_draft_block_error(FAKE[0], 1 << 20, None, None)] == "DLS_ERR_ARG"
    assert b.STATUS[L.dls_draft_block_error(FAKE[0], 1 << 20, ctypes.c_void_p(FAKE[1].value + 2), None)] == \
        "DLS_ERR_ARG"
    assert b.STATUS[L.dls_draft_block_error(FAKE[0], 64, FAKE[1], None)] == "DLS_ERR_WORKSPACE"
    assert b.STATUS[L.dls_draft_block_error(ctypes.c_void_p(FAKE[0].value + 16), 1 << 20, FAKE[1], None)] == \
        "DLS_ERR_WORKSPACE"
    if not HAS_GPU:
        assert b.STATUS[L.dls_draft_block_error(FAKE[0], 1 << 20, FAKE[1], None)] == "DLS_ERR_DEVICE"
        assert b.STATUS[L.dls_draft_block_error(None, 0, FAKE[1], None)] == "DLS_ERR_DEVICE"


def _adaptive(head, rule, unc=FAKE[10], **kw):
    a = dict(long=FAKE[5], ldt=b.DLS_BF16, last=FAKE[6], prior=None, batch=2, B=4, f=b.fusion(),
             tok=FAKE[7], st=FAKE[8], ws=FAKE[9], wsb=1 << 30)
    a.update(kw)
    L = b.lib()
    rc = L.dls_draft_block_adaptive(ctypes.byref(head), a["long"], a["ldt"], a["last"], a["prior"], a["batch"],
                                    a["B"], a["f"], b.Schedule(None, None), b.Sampling(0.0, 0, 0), rule, unc,
                                    a["tok"], a["st"], a["ws"], a["wsb"], None)
    return rc, L.dls_last_error().decode()


def _unc(rule, long=FAKE[0], dt=b.DLS_BF16, rows=16, V=151936, out=FAKE[1], ws=FAKE[2], wsb=1 << 24):
    L = b.lib()
    rc = L.dls_long_uncertainty(long, dt, rows, V, rule, out, ws, wsb, None)
    return b.STATUS[rc], L.dls_last_error().decode()


BAD_RULES = [b.Adaptive(2, 0.0, 1.0, 0), b.Adaptive(-1, 0.0, 1.0, 0), b.Adaptive(0, 0.5, 0.5, 0),
             b.Adaptive(1, 0.7, 0.2, 0), b.Adaptive(0, float("nan"), 1.0, 0), b.Adaptive(0, 0.0, float("inf"), 0),
             b.Adaptive(0, 0.0, 1.0, 3)]


def test_adaptive_rejects_bad_rules():
    for rule in BAD_RULES:
        st, msg = _unc(rule)
        assert st == "DLS_ERR_ARG", (rule.measure, rule.h_lo, rule.h_hi, msg)
        rc, msg = _adaptive(_head(), rule)
        assert b.STATUS[rc] == "DLS_ERR_ARG", msg
    good = b.adaptive_rule(b.UNC_ENTROPY, 0.1, 0.9)
    assert b.STATUS[_adaptive(_head(), good, unc=None)[0]] == "DLS_ERR_ARG"
    assert b.STATUS[_adaptive(_head(), good, unc=ctypes.c_void_p(FAKE[10].value + 2))[0]] == "DLS_ERR_ARG"
    assert b.STATUS[_adaptive(_head(), good, B=65)[0]] == "DLS_ERR_SHAPE"
    assert _adaptive(_head(), good, batch=0, long=None, tok=None, unc=None)[0] == 0


def test_long_uncertainty_rejects_bad_arguments():
    good = b.adaptive_rule(b.UNC_MAXPROB, -0.5, 0.5)
    assert _unc(good, dt=9)[0] == "DLS_ERR_DTYPE"
    assert _unc(good, V=0)[0] == "DLS_ERR_SHAPE"
    assert _unc(good, rows=-1)[0] == "DLS_ERR_SHAPE"
    assert _unc(good, long=None)[0] == "DLS_ERR_ARG"
    assert _unc(good, out=None)[0] == "DLS_ERR_ARG"
    assert _unc(good, long=ctypes.c_void_p(FAKE[0].value + 4))[0] == "DLS_ERR_ARG"
    need = b.long_uncertainty_workspace_size(16, 151936)
    assert need > 0
    assert _unc(good, wsb=need - 1)[0] == "DLS_ERR_WORKSPACE"
    assert _unc(good, ws=None)[0] == "DLS_ERR_ARG"
    assert _unc(good, rows=0, long=None, out=None)[0] == "DLS_OK"
    # enough rows to cover the GPU: one range per row, no workspace
    assert b.long_uncertainty_workspace_size(4096, 151936) == 0
    assert _unc(good, rows=4096, ws=None, wsb=0)[0] in ("DLS_ERR_DEVICE", "DLS_OK")


def test_draft_workspace_includes_the_uncertainty_partials():
    L = b.lib()
    h = _head(V=151936, d=64, H=32, r=16)
    plain = L.dls_draft_block_workspace_size(ctypes.byref(h), 1, 16)
    assert plain >= b.long_uncertainty_workspace_size(16, 151936) > 0


@pytest.mark.skipif(HAS_GPU, reason="would launch on fake pointers when a GPU is present")
def test_adaptive_valid_arguments_stop_at_device_check():
    for m in (b.UNC_ENTROPY, b.UNC_MAXPROB):
        rc, msg = _adaptive(_head(), b.adaptive_rule(m, -1.0, 2.0))
        assert b.STATUS[rc] == "DLS_ERR_DEVICE", msg
        assert _unc(b.adaptive_rule(m, 0.2, 0.3))[0] == "DLS_ERR_DEVICE"


def test_measure_helpers_reject_bad_arguments():
    L = b.lib()
    rd = lambda buf=FAKE[0], n=1 << 20, out=FAKE[1]: b.STATUS[L.dls_measure_read(buf, n, out, None)]
    assert rd(n=0) == "DLS_ERR_SHAPE"
    assert rd(n=(1 << 20) + 8) == "DLS_ERR_SHAPE"
    assert rd(buf=None) == "DLS_ERR_ARG"
    assert rd(out=None) == "DLS_ERR_ARG"
    assert rd(buf=ctypes.c_void_p(FAKE[0].value + 4)) == "DLS_ERR_ARG"
    assert rd(out=ctypes.c_void_p(FAKE[1].value + 2)) == "DLS_ERR_ARG"
    mf = lambda g=8, it=16, x=1.0 / 64, out=FAKE[2]: b.STATUS[L.dls_measure_mfma(g, it, x, out, None)]
    assert mf(g=0) == "DLS_ERR_SHAPE"
    assert mf(g=65537) == "DLS_ERR_SHAPE"
    assert mf(it=0) == "DLS_ERR_SHAPE"
    assert mf(it=(1 << 18) + 1) == "DLS_ERR_SHAPE"
    assert mf(g=65536, it=1 << 18) == "DLS_ERR_SHAPE"          # groups x iters above 2^24
    for x in (0.0, 0.75, 2.0, 2.0 ** -21, -0.5, float("nan"), float("inf")):
        assert mf(x=x) == "DLS_ERR_ARG", x
    assert mf(out=None) == "DLS_ERR_ARG"
    assert mf(out=ctypes.c_void_p(FAKE[2].value + 2)) == "DLS_ERR_ARG"
    if not HAS_GPU:
        assert rd() == "DLS_ERR_DEVICE"
        for x in (1.0, 2.0 ** -20, 0.5):
            assert mf(x=x, it=1 << 18, g=64) == "DLS_ERR_DEVICE", x
