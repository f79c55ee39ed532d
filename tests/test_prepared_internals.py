"""White-box GPU checks of the prepared head and of the persistent kernel's hand-off buffers.

* the folded input table T[u] = W_ih E[u] (float32 from exact bf16 products) against a
  float64 host product, relative error 1e-5;
* the operand-ordered copies of W_vocab and W_hh, bit-exact against a host rearrangement;
* after a one-position block: the published GRU state h_1 and rank vector rho_0 against
  the oracle's (the hand-off words are (tag << 32) | float bits).
"""
import numpy as np
import pytest
import torch

from oracle import dels_oracle as O
from paper_2607_07409_amd import binding as B
from paper_2607_07409_amd import workloads as W

pytestmark = pytest.mark.gpu

V, D, H, R = 5003, 96, 128, 128


def _layout():
    NT, KK = (V + 15) // 16, R // 32
    off_T = 256
    o = off_T + V * 3 * H * 4
    o = (o + 255) & ~255
    off_wv = o
    o += NT * KK * 1024
    off_whh = o
    return NT, KK, off_T, off_wv, off_whh


@pytest.fixture(scope="module")
def prob():
    wl = W.WORKLOADS["qwen3-8b-b16"].with_(V=V, d=D, H=H, r=R, B=1, batch=3, dtype="bf16")
    hw = W.make_head(wl, "stress")
    head = B.LocalHead.from_weights(hw).prepare()
    torch.cuda.synchronize()
    return wl, hw, head


def test_folded_input_table(prob):
    wl, hw, head = prob
    NT, KK, off_T, _, _ = _layout()
    T = head.prepared[off_T:off_T + V * 3 * H * 4].view(torch.float32).view(V, 3 * H).cpu().numpy()
    emb = np.asarray(hw.emb, np.float64)
    wih = np.asarray(hw.w_ih, np.float64)
    toks = np.arange(V)                        # every row: all row blocks, the ragged last one
    want = emb[toks] @ wih.T
    # float32 accumulation of exact products: |error| <= d * 2^-24 * sum |products| (plus slack)
    bound = D * 2.0 ** -24 * (np.abs(emb[toks]) @ np.abs(wih).T) + 1e-30
    err = np.abs(T[toks] - want)
    assert np.all(err <= 4 * bound), (err / bound).max()


@pytest.mark.parametrize("v,d,h", [(77, 8, 32), (300, 200, 96), (1000, 520, 160)])
def test_folded_input_table_shapes(v, d, h):
    """The fold's GEMM tiles (128 x 128 blocks, K steps of 64) at shapes that leave every edge
    ragged: rows past V, columns past 3H and K past d must read as zeros."""
    wl = W.WORKLOADS["qwen3-8b-b16"].with_(V=v, d=d, H=h, r=32, B=1, batch=1, dtype="bf16")
    hw = W.make_head(wl, "stress")
    head = B.LocalHead.from_weights(hw).prepare()
    torch.cuda.synchronize()
    T = head.prepared[256:256 + v * 3 * h * 4].view(torch.float32).view(v, 3 * h).cpu().numpy()
    emb = np.asarray(hw.emb, np.float64)
    wih = np.asarray(hw.w_ih, np.float64)
    want = emb @ wih.T
    bound = d * 2.0 ** -24 * (np.abs(emb) @ np.abs(wih).T) + 1e-30
    assert np.all(np.abs(T - want) <= 4 * bound), (np.abs(T - want) / bound).max()


def test_operand_order_copies(prob):
    wl, hw, head = prob
    NT, KK, _, off_wv, off_whh = _layout()
    wv = head.prepared[off_wv:off_wv + NT * KK * 1024].cpu().numpy().view(np.uint16).reshape(NT, KK, 64, 8)
    bits = np.zeros((NT * 16, R), np.uint16)
    bits[:V] = hw.w_vocab.bits
    for t in [0, 1, NT // 2, NT - 1]:
        for kk in range(KK):
            for l in range(64):
                row, col = 16 * t + l % 16, 32 * kk + 8 * (l // 16)
                assert np.array_equal(wv[t, kk, l], bits[row, col:col + 8]), (t, kk, l)
    KKH = H // 32
    whh = head.prepared[off_whh:off_whh + (H // 16) * 3 * KKH * 1024].cpu().numpy().view(np.uint16)
    whh = whh.reshape(H // 16, 3, KKH, 64, 8)
    hb = hw.w_hh.bits
    for g in [0, H // 16 - 1]:
        for q in range(3):
            for kk in range(KKH):
                for l in range(64):
                    row, col = q * H + 16 * g + l % 16, 32 * kk + 8 * (l // 16)
                    assert np.array_equal(whh[g, q, kk, l], hb[row, col:col + 8]), (g, q, kk, l)


def test_first_position_handoffs(prob):
    wl, hw, head = prob
    batch = wl.batch
    long_h = W.make_long_logits(wl)
    last = W.make_last_token(wl)
    assert head.path(batch, 1) == 1
    ws = B.draft_workspace(head, batch, 1)
    tok, st = B.draft_block(head, B.as_tensor(long_h), torch.from_numpy(last).cuda(), None, 1.0, 0.5, 0.0,
                            workspace=ws)
    torch.cuda.synchronize()
    assert B.workspace_error(ws) == 0
    # workspace layout: 256-byte header, argmax keys, the two sets of wide-batch h words
    # (2 x 2 x 64 x 4096 words of 4 bytes), then the 64-bit h and rho hand-off words
    off_h = 256 + 2 * 2 * 64 * 256 * 8 + 2 * 2 * 64 * 4096 * 4
    off_r = off_h + 2 * batch * H * 8
    words_h = ws[off_h:off_h + batch * H * 8].view(torch.int64).cpu().numpy()
    words_r = ws[off_r:off_r + batch * R * 8].view(torch.int64).cpu().numpy()
    h_gpu = (words_h & 0xffffffff).astype(np.uint32).view(np.float32).reshape(batch, H)
    r_gpu = (words_r & 0xffffffff).astype(np.uint32).view(np.float32).reshape(batch, R)
    oh = O.RnnHead.from_weights(hw)
    for b in range(batch):
        h1 = O.gru_cell(np.asarray(hw.emb[int(last[b])], np.float64), np.zeros(H), oh.w_ih, oh.w_hh)
        np.testing.assert_allclose(h_gpu[b], h1, atol=2e-5, err_msg=f"h_1 of sequence {b}")
        np.testing.assert_allclose(r_gpu[b], oh.rho(h1), atol=2e-5, err_msg=f"rho_0 of sequence {b}")
    ref = O.draft_block(oh, long_h, last, None, 1.0, 0.5, 0.0)
    gap_ok = ref.gap[:, 0] < 2e-2
    assert np.all((tok.cpu().numpy()[:, 0] == ref.tokens[:, 0]) | gap_ok)
