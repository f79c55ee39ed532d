"""Pins of the oracle's local heads (App. A) against library implementations.

The RNN head is a bias-free one-layer GRU over the frozen target embedding, a SiLU
low-rank projection and a vocabulary head.  torch.nn.GRU(bias=False), nn.Linear and
F.silu in float64 on the CPU are an independent implementation of exactly that, with the
(r, z, n) gate layout the oracle reads the weights in.  The greedy rollout of the head
alone is the w_long = 0 limit of the drafting loop.
"""
import math

import numpy as np
import pytest
import torch

from oracle import dels_oracle as O


def _weights(seed, V, d, H, r):
    g = np.random.default_rng(seed)
    return dict(emb=g.normal(0, 1, (V, d)), w_ih=g.normal(0, 2 / math.sqrt(d), (3 * H, d)),
                w_hh=g.normal(0, 2 / math.sqrt(H), (3 * H, H)),
                w_rank=g.normal(0, 1 / math.sqrt(H), (r, H)),
                w_vocab=g.normal(0, 3 / math.sqrt(r), (V, r)))


class TorchHead(torch.nn.Module):
    def __init__(self, w):
        super().__init__()
        V, d = w["emb"].shape
        H = w["w_hh"].shape[1]
        r = w["w_rank"].shape[0]
        self.emb = torch.nn.Embedding(V, d, dtype=torch.float64)
        self.gru = torch.nn.GRU(d, H, num_layers=1, bias=False, batch_first=True,
                                dtype=torch.float64)
        self.rank = torch.nn.Linear(H, r, bias=False, dtype=torch.float64)
        self.vocab = torch.nn.Linear(r, V, bias=False, dtype=torch.float64)
        with torch.no_grad():
            self.emb.weight.copy_(torch.from_numpy(w["emb"]))
            self.gru.weight_ih_l0.copy_(torch.from_numpy(w["w_ih"]))
            self.gru.weight_hh_l0.copy_(torch.from_numpy(w["w_hh"]))
            self.rank.weight.copy_(torch.from_numpy(w["w_rank"]))
            self.vocab.weight.copy_(torch.from_numpy(w["w_vocab"]))

    def forward(self, tokens):
        """short logits after each prefix token [T] -> [T, V]"""
        x = self.emb(torch.as_tensor(tokens).long())[None]
        hs, _ = self.gru(x)                      # h_0 = 0
        return self.vocab(torch.nn.functional.silu(self.rank(hs[0])))


@pytest.mark.parametrize("V,d,H,r", [(61, 12, 9, 5), (128, 32, 16, 8), (40, 7, 33, 64)])
def test_rnn_head_matches_torch_gru(V, d, H, r):
    w = _weights(V + d + H + r, V, d, H, r)
    head = O.RnnHead(**w)
    ref = TorchHead(w)
    toks = np.random.default_rng(0).integers(0, V, 9)
    with torch.no_grad():
        want = ref(toks).numpy()
    h = head.init_state()
    for t, tok in enumerate(toks):
        h, s = head.step(h, tok)
        np.testing.assert_allclose(s, want[t], rtol=1e-10, atol=1e-10)


def test_greedy_rollout_is_head_alone():
    """w_long = 0, beta = 0: the fused draft is the greedy rollout of the head itself,
    computed here with torch (the next input is the argmax of the previous short logits)."""
    V, d, H, r = 89, 16, 24, 12
    w = _weights(99, V, d, H, r)
    head = O.RnnHead(**w)
    ref = TorchHead(w)
    g = np.random.default_rng(5)
    L = g.normal(0, 3, (2, 8, V))
    last = [7, 50]
    res = O.draft_block(head, L, last, None, 0.0, 1.0, 0.0)
    for b in range(2):
        seq = [last[b]]
        for _ in range(8):
            with torch.no_grad():
                s = ref(seq)[-1]
            seq.append(int(torch.argmax(s.float())))
        assert res.tokens[b].tolist() == seq[1:]
    # and the oracle's own rollout helper agrees
    np.testing.assert_array_equal(O.head_rollout(head, last[0], 8), res.tokens[0])


def test_gru_single_step_from_zero_state():
    """From h_0 = 0 the recurrent term vanishes: h' = (1 - sigmoid(W_iz x)) * tanh(W_in x)."""
    g = np.random.default_rng(3)
    d, H = 10, 6
    w_ih = g.normal(0, 1, (3 * H, d))
    x = g.normal(0, 1, d)
    h1 = O.gru_cell(x, np.zeros(H), w_ih, g.normal(0, 1, (3 * H, H)))
    gru = torch.nn.GRUCell(d, H, bias=False, dtype=torch.float64)
    with torch.no_grad():
        gru.weight_ih.copy_(torch.from_numpy(w_ih))
        gru.weight_hh.zero_()
        want = gru(torch.from_numpy(x)[None], torch.zeros(1, H, dtype=torch.float64))[0].numpy()
    np.testing.assert_allclose(h1, want, rtol=1e-12, atol=1e-14)


def test_markov_head_matches_embedding_bag():
    """l_S = E_M(prev) W_M^T: compare with torch Embedding + Linear."""
    g = np.random.default_rng(4)
    V, dr = 33, 5
    em, wm = g.normal(0, 1, (V, dr)), g.normal(0, 1, (V, dr))
    head = O.MarkovHead(em, wm)
    E = torch.nn.Embedding(V, dr, dtype=torch.float64)
    Wl = torch.nn.Linear(dr, V, bias=False, dtype=torch.float64)
    with torch.no_grad():
        E.weight.copy_(torch.from_numpy(em))
        Wl.weight.copy_(torch.from_numpy(wm))
        for prev in [0, 5, 32]:
            _, s = head.step(None, prev)
            np.testing.assert_allclose(s, Wl(E(torch.tensor([prev])))[0].numpy(), rtol=1e-12)


def test_silu_sigmoid_library():
    x = np.linspace(-30, 30, 1001)
    np.testing.assert_allclose(O.silu(x), torch.nn.functional.silu(torch.from_numpy(x)).numpy(),
                               rtol=1e-12, atol=1e-300)
    np.testing.assert_allclose(O.logsumexp(x), torch.logsumexp(torch.from_numpy(x), 0).item(),
                               rtol=1e-14)
