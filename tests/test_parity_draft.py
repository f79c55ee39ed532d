"""GPU parity of dls_draft_block and dls_accept_len against the oracle, on all five
drafting workloads (tiny; Qwen3-4B and -8B shaped at batch 1; batch 16; batch 64),
with baseline and stress-scaled head weights, both first-row readings, the prior term,
a ragged small problem and mixed dtypes.
"""
import functools

import numpy as np
import pytest
import torch

from oracle import dels_oracle as O
from paper_2607_07409_amd import binding as B
from paper_2607_07409_amd import workloads as W
from parity_util import TOL, check_draft

pytestmark = pytest.mark.gpu


@functools.lru_cache(maxsize=2)
def _problem(name, init, V=None, d=None, H=None, r=None, Bk=None, batch=None, dtype=None):
    wl = W.WORKLOADS[name]
    kw = {k: v for k, v in dict(V=V, d=d, H=H, r=r, B=Bk, batch=batch, dtype=dtype).items() if v is not None}
    if kw:
        wl = wl.with_(**kw)
    hw = W.make_head(wl, init)
    head = B.LocalHead.from_weights(hw)
    return dict(wl=wl, hw=hw, head=head, oracle=O.RnnHead.from_weights(hw),
                long_h=W.make_long_logits(wl), last=W.make_last_token(wl),
                prior=W.make_zipf_log_prior(wl.V, wl.seed), prepared=None)


def _head(p, prepared):
    """The unprepared head, or a prepared twin sharing its weight tensors."""
    if not prepared:
        return p["head"]
    if p["prepared"] is None:
        h = p["head"]
        p["prepared"] = B.LocalHead(h.emb, h.w_ih, h.w_hh, h.w_rank, h.w_vocab).prepare()
    return p["prepared"]


def _draft(p, alpha, beta=0.0, with_prior=False, literal=False, long_h=None, prepared=False, expect_path=None):
    long_h = p["long_h"] if long_h is None else long_h
    lt = B.as_tensor(long_h)
    last = torch.from_numpy(p["last"]).cuda()
    prior = torch.from_numpy(p["prior"]).cuda() if with_prior else None
    head = _head(p, prepared)
    path = head.path(lt.shape[0], lt.shape[1], lt.dtype, with_prior)
    if expect_path is not None:
        assert path == expect_path, f"draft path {path}, expected {expect_path}"
    ws = B.draft_workspace(head, lt.shape[0], lt.shape[1])
    tok, st = B.draft_block(head, lt, last, prior, 1.0, alpha, beta, first_row_long_only=literal, workspace=ws)
    torch.cuda.synchronize()
    assert B.workspace_error(ws) == 0
    return tok.cpu().numpy(), st.cpu().numpy()


def _check(p, alpha, beta=0.0, with_prior=False, literal=False, sequences=None, prepared=False):
    tok, st = _draft(p, alpha, beta, with_prior, literal, prepared=prepared,
                     expect_path=1 if prepared else 0)
    rep = check_draft(tok, st, p["oracle"], p["long_h"], p["last"], p["prior"] if with_prior else None,
                      1.0, alpha, beta if with_prior else 0.0, literal, sequences)
    print(f"{p['wl'].name}: near_ties={rep['near_ties']} fusion_active={rep['fusion_active']:.2f} "
          f"errs={rep['errs']}")
    return tok, st, rep


@pytest.mark.parametrize("init", ["baseline", "stress"])
@pytest.mark.parametrize("literal", [False, True])
@pytest.mark.parametrize("with_prior", [False, True])
def test_tiny(init, literal, with_prior):
    p = _problem("tiny", init)
    _check(p, 0.5, 0.5, with_prior, literal)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_small_ragged(dtype):
    """V not a multiple of any tile, rows of the long logits misaligned, d/H/r small and odd multiples of 8."""
    p = _problem("qwen3-8b-b16", "stress", V=5003, d=72, H=40, r=24, Bk=7, batch=3, dtype=dtype)
    _, _, rep = _check(p, 1.0)
    assert rep["fusion_active"] > 0.2


def test_mixed_dtypes():
    """fp32 head weights with bf16 long logits and the reverse."""
    p = _problem("qwen3-8b-b16", "stress", V=3001, d=64, H=64, r=32, Bk=5, batch=2, dtype="f32")
    lb = W.Bf16Array.from_f32(np.asarray(p["long_h"], np.float32))
    tok, st = _draft(p, 0.5, long_h=lb)
    check_draft(tok, st, p["oracle"], lb, p["last"], None, 1.0, 0.5, 0.0)


@pytest.mark.parametrize("prepared", [False, True])
@pytest.mark.parametrize("init", ["baseline", "stress"])
def test_qwen3_4b_b1(init, prepared):
    p = _problem("qwen3-4b-b1", init)
    tok, st, rep = _check(p, 0.5, prepared=prepared)
    if init == "stress":
        assert rep["fusion_active"] > 0.3
    # literal first-row reading on the same inputs
    _check(p, 0.5, literal=True, prepared=prepared)


@pytest.mark.parametrize("prepared", [False, True])
@pytest.mark.parametrize("alpha", [0.25, 0.5, 1.0])
def test_qwen3_8b_b1_alpha_sweep(alpha, prepared):
    p = _problem("qwen3-8b-b1", "stress")
    _check(p, alpha, prepared=prepared)


@pytest.mark.parametrize("prepared", [False, True])
def test_qwen3_8b_b1_alpha_zero_is_dflash(prepared):
    p = _problem("qwen3-8b-b1", "stress")
    tok, _ = _draft(p, 0.0, prepared=prepared)
    assert np.array_equal(tok, np.argmax(np.asarray(p["long_h"], np.float32), axis=2))


@pytest.mark.parametrize("prepared", [False, True])
@pytest.mark.parametrize("init", ["baseline", "stress"])
def test_serving_b16(init, prepared):
    """Every sequence of the batch-16 workload, element by element against the oracle."""
    p = _problem("qwen3-8b-b16", init)
    _check(p, 0.5, prepared=prepared)


@pytest.mark.parametrize("prepared", [False, True])
def test_serving_b64(prepared):
    """Every sequence of the batch-64 workload (four 16-sequence M tiles of the wide kernel)."""
    p = _problem("b64-d5120", "stress")
    _check(p, 0.5, prepared=prepared)


@pytest.mark.parametrize("prepared", [False, True])
def test_serving_b64_prior(prepared):
    """beta = alpha with the Zipf log-prior (the paper's alpha = beta diagonal), every sequence."""
    p = _problem("b64-d5120", "stress")
    _check(p, 0.5, 0.5, with_prior=True, prepared=prepared)


@pytest.mark.parametrize("prepared", [False, True])
@pytest.mark.parametrize("w_long", [1.0, 0.0])
@pytest.mark.parametrize("name", ["qwen3-4b-b1", "qwen3-8b-b16", "b64-d5120"])
def test_masked_long_logits(name, w_long, prepared):
    """-inf long logits (masked tokens, allowed by the ABI) through dls_draft_block, every sequence:
    narrow (batch 1) and wide (batch 16: one M tile; batch 64: four) persistent kernels and the
    per-position launches.  With w_long = 1 a masked token is never drafted, and a row that keeps a
    single finite entry drafts that entry; with w_long = 0 the long term, masks included, is absent
    (the head alone decides).  Statistics against the oracle within the tolerance."""
    p = _problem(name, "stress")
    wl = p["wl"]
    single = [(0, 2), (wl.batch - 1, wl.B - 1)]
    masked, kept = W.mask_long_logits(p["long_h"], 0.3, 17, single)
    lt = B.as_tensor(masked)
    last = torch.from_numpy(p["last"]).cuda()
    head = _head(p, prepared)
    assert head.path(wl.batch, wl.B, lt.dtype, False) == (1 if prepared else 0)
    ws = B.draft_workspace(head, wl.batch, wl.B)
    tok, st = B.draft_block(head, lt, last, None, w_long, 0.5, 0.0, workspace=ws)
    torch.cuda.synchronize()
    assert B.workspace_error(ws) == 0
    tok, st = tok.cpu().numpy(), st.cpu().numpy()
    if w_long > 0:
        bits = masked.bits
        for b in range(wl.batch):
            for j in range(wl.B):
                assert bits[b, j, tok[b, j]] != 0xFF80, (b, j)
        for (b, j), t in kept.items():
            assert tok[b, j] == t, (b, j)
    rep = check_draft(tok, st, p["oracle"], masked, p["last"], None, w_long, 0.5, 0.0)
    print(f"{name} masked w_long={w_long}: near_ties={rep['near_ties']} errs={rep['errs']}")


# ---------------------------------------------------------------------------------------------
# persistent kernel on small shapes (oracle in seconds): ragged vocabularies, few tiles per CU,
# both first-row readings, the prior, float32 long logits, batches spanning several 16-slot tiles
# ---------------------------------------------------------------------------------------------
SMALL = [
    dict(V=5003, d=96, H=128, r=128, Bk=7, batch=3),
    dict(V=7001, d=64, H=256, r=256, Bk=9, batch=2),
    dict(V=1024, d=64, H=128, r=128, Bk=4, batch=1),
    dict(V=4099, d=128, H=128, r=128, Bk=5, batch=37),
    dict(V=2053, d=64, H=512, r=128, Bk=5, batch=9),      # wide, h staged in two K chunks
]


@pytest.mark.parametrize("shape", range(len(SMALL)))
@pytest.mark.parametrize("literal", [False, True])
def test_persistent_small(shape, literal):
    sh = SMALL[shape]
    p = _problem("qwen3-8b-b16", "stress", dtype="bf16", **sh)
    seqs = list(range(min(sh["batch"], 6))) + ([sh["batch"] - 1] if sh["batch"] > 6 else [])
    _, _, rep = _check(p, 0.7, literal=literal, prepared=True, sequences=seqs)
    assert rep["fusion_active"] > 0.2


EXTREME = [
    dict(V=4099, d=64, H=128, r=128, Bk=64, batch=3),     # the longest block (64 positions)
    dict(V=1031, d=64, H=128, r=128, Bk=64, batch=64),    # the largest batch with the longest block
    dict(V=2053, d=64, H=128, r=128, Bk=1, batch=5),      # a single position
]


@pytest.mark.parametrize("shape", range(len(EXTREME)))
def test_persistent_extreme_block_sizes(shape):
    sh = EXTREME[shape]
    p = _problem("qwen3-8b-b16", "stress", dtype="bf16", **sh)
    seqs = sorted({0, sh["batch"] // 2, sh["batch"] - 1})
    _check(p, 0.6, prepared=True, sequences=seqs)
    _check(p, 0.6, 0.4, with_prior=True, literal=True, prepared=True, sequences=seqs[:1])


@pytest.mark.parametrize("batch", [65, 256])
def test_batches_split_into_launches(batch):
    """Above 64 sequences (up to the ABI's maximum of 256) a prepared head runs consecutive
    persistent launches of at most 64 sequences on one workspace; the first and last sequence of
    every launch are compared, greedy and with the prior and the literal first row."""
    p = _problem("qwen3-8b-b16", "stress", dtype="bf16", V=2053, d=64, H=128, r=128, Bk=3, batch=batch)
    seqs = sorted({s for b0 in range(0, batch, 64) for s in (b0, min(b0 + 63, batch - 1))})
    tok, st = _draft(p, 0.6, prepared=True, expect_path=1)
    check_draft(tok, st, p["oracle"], p["long_h"], p["last"], None, 1.0, 0.6, 0.0, sequences=seqs)
    tok, st = _draft(p, 0.6, 0.4, with_prior=True, literal=True, prepared=True, expect_path=1)
    check_draft(tok, st, p["oracle"], p["long_h"], p["last"], p["prior"], 1.0, 0.6, 0.4, True, seqs)


@pytest.mark.parametrize("batch", [4, 5, 15, 16, 17, 31, 32, 33, 47, 48, 49, 63])
def test_batch_sweep_across_m_tiles(batch):
    """Every batch size on either side of the narrow/wide switch (4 | 5) and of each 16-sequence M
    tile boundary, where the token merge changes hands (one M tile: every GRU workgroup merges;
    several: workgroup NG + b merges sequence b), every sequence compared, greedy and with the
    prior and the literal first row."""
    p = _problem("qwen3-8b-b16", "stress", dtype="bf16", V=2053, d=64, H=128, r=128, Bk=3, batch=batch)
    tok, st = _draft(p, 0.6, prepared=True, expect_path=1)
    check_draft(tok, st, p["oracle"], p["long_h"], p["last"], None, 1.0, 0.6, 0.0)
    tok, st = _draft(p, 0.6, 0.4, with_prior=True, literal=True, prepared=True, expect_path=1)
    check_draft(tok, st, p["oracle"], p["long_h"], p["last"], p["prior"], 1.0, 0.6, 0.4, True)


def test_split_launches_sample_by_sequence_index():
    """Sampling keys the noise by the sequence's index in the whole call: at batch 80 (launches of
    64 and 16 sequences) the draws of sequences 63, 64 and 79 are the oracle's for that index, and
    a sequence drafts the same tokens whether the call is split or not."""
    p = _problem("qwen3-8b-b16", "stress", dtype="bf16", V=2053, d=64, H=128, r=128, Bk=4, batch=80)
    head = _head(p, True)
    lt = B.as_tensor(p["long_h"])
    last = torch.from_numpy(p["last"]).cuda()
    tok, st = B.draft_block(head, lt, last, None, 1.0, 0.6, 0.0, temperature=1.0, seed=99)
    torch.cuda.synchronize()
    tok, st = tok.cpu().numpy(), st.cpu().numpy()
    check_draft(tok, st, p["oracle"], p["long_h"], p["last"], None, 1.0, 0.6, 0.0,
                sequences=[0, 63, 64, 79], temperature=1.0, seed=99)
    # the unsplit per-position launches on the same call draw the same noise
    tok2, _ = B.draft_block(p["head"], lt, last, None, 1.0, 0.6, 0.0, temperature=1.0, seed=99)
    torch.cuda.synchronize()
    same = (tok2.cpu().numpy() == tok).all(axis=1)
    assert same.mean() > 0.9, same.mean()   # sequences may part at a near-tie of the two paths


@pytest.mark.parametrize("shape", [0, 3])
def test_persistent_small_prior(shape):
    p = _problem("qwen3-8b-b16", "stress", dtype="bf16", **SMALL[shape])
    _check(p, 0.5, 0.5, with_prior=True, prepared=True, sequences=[0, 1, 2])


def test_persistent_f32_long_logits():
    p = _problem("qwen3-8b-b16", "stress", dtype="bf16", **SMALL[0])
    lf = np.asarray(p["long_h"], np.float32) + np.float32(1e-3)     # not bf16-representable
    tok, st = _draft(p, 0.5, long_h=lf, prepared=True, expect_path=1)
    check_draft(tok, st, p["oracle"], lf, p["last"], None, 1.0, 0.5, 0.0)


def test_persistent_repeat_and_paths_agree():
    """Back-to-back calls on one workspace (the epoch tags of the hand-offs advance every call)
    are bit-identical, and agree with the per-position launches on the tokens."""
    p = _problem("qwen3-8b-b16", "stress", dtype="bf16", **SMALL[1])
    head = _head(p, True)
    lt = B.as_tensor(p["long_h"])
    last = torch.from_numpy(p["last"]).cuda()
    ws = B.draft_workspace(head, lt.shape[0], lt.shape[1])
    outs = []
    for i in range(6):
        tok, st = B.draft_block(head, lt, last, None, 1.0, 0.5, 0.0, first_row_long_only=bool(i % 2), workspace=ws)
        outs.append((tok.clone(), st.clone()))
    torch.cuda.synchronize()
    assert B.workspace_error(ws) == 0
    for i in range(2, 6):   # bit patterns: the literal reading's first row has NaN lse_short
        assert torch.equal(outs[i][0], outs[i % 2][0])
        assert torch.equal(outs[i][1].view(torch.int32), outs[i % 2][1].view(torch.int32))
    tok1, _ = _draft(p, 0.5, prepared=False)
    tok_p, _ = _draft(p, 0.5, prepared=True)
    ref = O.draft_block(p["oracle"], p["long_h"], p["last"], None, 1.0, 0.5, 0.0)
    for t in (tok1, tok_p):
        near = (t != ref.tokens)
        assert np.all(ref.gap[near] < TOL)


def test_persistent_workspace_shared_across_shapes():
    """One workspace serves calls of different batch sizes and block lengths in turn, each with
    other inputs than the call before (wide batches hand h over with 8-bit position tags, so a
    call must not see words left by an earlier one): every call returns the bits of the same
    call on a fresh workspace."""
    p = _problem("qwen3-8b-b16", "stress", dtype="bf16", **SMALL[3])   # batch 37, 5 positions
    head = _head(p, True)
    ws = B.draft_workspace(head, 64, 16)
    shapes = [(37, 5), (6, 3), (37, 5), (20, 4), (2, 5), (37, 5), (37, 5)]
    for k, (b, bk) in enumerate(shapes):
        lt = B.as_tensor(np.ascontiguousarray(p["long_h"][:b, :bk]))
        last = torch.from_numpy(np.ascontiguousarray(np.roll(p["last"], k)[:b])).cuda()
        alpha = 0.4 + 0.1 * (k % 3)
        tok, st = B.draft_block(head, lt, last, None, 1.0, alpha, 0.0, workspace=ws)
        fresh = B.draft_workspace(head, b, bk)
        tok2, st2 = B.draft_block(head, lt, last, None, 1.0, alpha, 0.0, workspace=fresh)
        torch.cuda.synchronize()
        assert B.workspace_error(ws) == 0 and B.workspace_error(fresh) == 0
        assert torch.equal(tok, tok2), (k, b, bk)
        assert torch.equal(st.view(torch.int32), st2.view(torch.int32)), (k, b, bk)
        # white-box: the set of 32-bit h words the next call will read is all zeros, whatever
        # this call was (narrow calls clear it too).  Layout: 256-byte header, 2 x 2 x 64 x 256
        # argmax keys of 8 bytes, then two sets of 2 x 64 x 4096 words of 4 bytes; the set is
        # the parity of the call epoch (the first uint32 of the header, advanced by each call)
        nxt = int(ws[0:4].view(torch.int32).item()) & 1
        off, size = 256 + 2 * 2 * 64 * 256 * 8, 2 * 64 * 4096 * 4
        assert int(ws[off + nxt * size: off + (nxt + 1) * size].count_nonzero().item()) == 0, (k, b, bk)


@pytest.mark.parametrize("shape", [0, 1, 3])
def test_exclusive_device_launch_same_bits(shape):
    """DLS_EXCLUSIVE_DEVICE (an ordinary instead of a cooperative dispatch of the persistent
    kernel) returns the cooperative launch's bits, call after call on one workspace."""
    p = _problem("qwen3-8b-b16", "stress", dtype="bf16", **SMALL[shape])
    head = _head(p, True)
    lt = B.as_tensor(p["long_h"])
    last = torch.from_numpy(p["last"]).cuda()
    prior = torch.from_numpy(p["prior"]).cuda()
    ws = B.draft_workspace(head, lt.shape[0], lt.shape[1])
    outs = []
    for i in range(6):
        tok, st = B.draft_block(head, lt, last, prior, 1.0, 0.5, 0.3, workspace=ws, exclusive_device=bool(i % 2))
        outs.append((tok.clone(), st.clone()))
    torch.cuda.synchronize()
    assert B.workspace_error(ws) == 0
    for tok, st in outs[1:]:
        assert torch.equal(tok, outs[0][0]) and torch.equal(st.view(torch.int32), outs[0][1].view(torch.int32))
    _check(p, 0.5, 0.3, with_prior=True, prepared=True, sequences=[0, p["wl"].batch - 1])


@pytest.mark.parametrize("name", ["tiny", "qwen3-4b-b1", "qwen3-8b-b16"])
def test_accept_len_on_drafts(name):
    """Targets agree with the oracle draft for a geometric prefix; the GPU acceptance length on its own
    draft equals the oracle's on that draft."""
    p = _problem(name, "stress")
    tok, _ = _draft(p, 0.5)
    seqs = list(range(min(p["wl"].batch, 4)))
    ref = O.draft_block(p["oracle"], p["long_h"], p["last"], None, 1.0, 0.5, 0.0, sequences=seqs)
    targets, k = W.make_targets(ref.tokens, p["wl"])
    acc = B.accept_len(torch.from_numpy(tok).cuda(), torch.from_numpy(targets).cuda())
    torch.cuda.synchronize()
    want = O.accept_len(tok, targets)
    assert np.array_equal(acc.cpu().numpy(), want)
    same = np.array_equal(tok[seqs], ref.tokens[seqs])
    if same:
        assert np.all(want[seqs] >= k[seqs])


def test_accept_len_cases():
    g = np.random.default_rng(3)
    for batch, Bk in [(1, 1), (5, 16), (300, 16), (7, 100), (3, 0), (64, 64), (2, 65)]:
        d = g.integers(0, 50, (batch, Bk)).astype(np.int32)
        t = d.copy()
        for b in range(batch):
            if Bk:
                k = int(g.integers(0, Bk + 1))
                if k < Bk:
                    t[b, k] += 1
        got = B.accept_len(torch.from_numpy(d).cuda(), torch.from_numpy(t).cuda())
        torch.cuda.synchronize()
        assert np.array_equal(got.cpu().numpy(), O.accept_len(d, t)), (batch, Bk)


@pytest.mark.parametrize("prepared", [False, True])
def test_draft_deterministic(prepared):
    p = _problem("qwen3-4b-b1", "stress")
    t0, s0 = _draft(p, 0.5, prepared=prepared)
    for _ in range(3):
        t1, s1 = _draft(p, 0.5, prepared=prepared)
        assert np.array_equal(t0, t1) and np.array_equal(s0.view(np.int32), s1.view(np.int32))
