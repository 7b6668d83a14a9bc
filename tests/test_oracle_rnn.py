"""Pins of the oracle's RNN-head draft block (no GPU).

The RNN head (the RNN-head item of the section on semi-autoregressive
generation, eq. rnn) feeds z_k = [s_{k-1}; W1[x_{k-1}]; h_k] through one
projection split into gate, candidate and output parts; the state is a gated
mix of the previous state and the candidate, and the transition bias is W2^T
applied to tanh of the output part.  The tests pin the oracle against what
the mathematics fixes, not against its own formula:

* zero weights give zero bias: every position is a library softmax of the
  scaled base logits, and the confidences equal the (separately pinned)
  Markov oracle's;
* an output part that reads only the embedding through a power-of-two
  multiple of the identity, alpha * I, is the Markov head with the projection
  scaled by alpha, up to tanh's cubic term, whatever the gate and candidate
  weights (the state must not leak into the bias);
* a gate saturated at 1 (sigmoid(1000) is 1 in fp64) keeps the state at zero,
  so the state columns of the projection cannot matter (bit-identical
  outputs); a swapped gate would fail it;
* a gate saturated at 0 makes the state the candidate: with a candidate that
  reads the embedding and an output that reads the state, position k + 1 is
  biased by the token two places back -- the Markov head one position
  later, through the anchor;
* with state weights the bias sees the whole prefix (two requests that share
  x_1 but not the anchor differ at position 2); without them they agree;
* a half-open gate (sigmoid(0) = 1/2) keeps half of the previous state: two
  requests that share x_1 and x_2 still differ at position 3 through the
  anchor, and agree once the gate is shut;
* requests are independent of each other.
"""
import numpy as np
from scipy.special import softmax

import oracle
from paper_2607_05147_amd import synth

bf16 = synth.f32_to_bf16_bits
widen = synth.bf16_bits_to_f32


def _inv_cdf(p, u):
    c = np.cumsum(p)
    return int(np.searchsorted(c, u * c[-1], side="right"))


def _base(rng, R, K, V, scale=3.0):
    return bf16((scale * rng.normal(size=(R * K, V))).astype(np.float32))


def _rand(rng, shape, scale=1.0):
    return bf16((scale * rng.normal(size=shape)).astype(np.float32))


def _blocks(rank, d, gate=None, cand=None, out=None):
    """Wrnn [3 rank, 2 rank + d] from per-part [rank, 2 rank + d] float blocks (None = 0)."""
    W = np.zeros((3 * rank, 2 * rank + d), np.float32)
    for i, b in enumerate((gate, cand, out)):
        if b is not None:
            W[i * rank:(i + 1) * rank] = b
    return bf16(W)


def test_zero_weights_are_an_independent_softmax():
    rng = np.random.default_rng(11)
    R, K, V, rank, d = 3, 4, 60, 8, 16
    W1 = _rand(rng, (V, rank))
    W2t = _rand(rng, (V, rank))
    Wr = np.zeros((3 * rank, 2 * rank + d), np.uint16)
    hid = _rand(rng, (R, K, d))
    wc = rng.normal(size=d + rank).astype(np.float32) * 0.2
    st = (1.0 + 0.1 * np.arange(K)).astype(np.float32)
    U = _base(rng, R, K, V)
    u = rng.random((R, K)).astype(np.float32)
    anc = rng.integers(0, V, R)
    tok, p, conf, _ = oracle.rnn_draft(anc, U, "bf16", W1, W2t, Wr, wc, u, K, V, hidden=hid,
                                       sts_temp=st, inv_temperature=0.9)
    itf = float(np.float32(0.9))
    Uf = widen(U).astype(np.float64)
    for r in range(R):
        for k in range(K):
            ref = softmax(itf * Uf[r * K + k])
            np.testing.assert_allclose(p[r, k], ref, rtol=1e-12, atol=0)
            assert tok[r, k] == _inv_cdf(ref, float(u[r, k]))
    # the same tokens through the Markov oracle with a zero projection: the
    # confidence path (backbone state, embedding of the previous token,
    # per-position temperature) must agree
    tm, pm, cm, _ = oracle.markov_draft(anc, U, "bf16", W1, np.zeros_like(W2t), wc, u, K, V,
                                        hidden=hid, sts_temp=st, inv_temperature=0.9)
    assert np.array_equal(tm, tok)
    np.testing.assert_allclose(pm, p, rtol=1e-13, atol=0)
    np.testing.assert_allclose(cm, conf, rtol=1e-13, atol=0)


def test_embedding_only_output_is_the_markov_head_with_a_scaled_projection():
    rng = np.random.default_rng(12)
    R, K, V, rank, d = 4, 5, 80, 8, 12
    alpha = 2.0 ** -10
    W1 = _rand(rng, (V, rank))
    W2t = _rand(rng, (V, rank), 256.0)
    n = 2 * rank + d
    # gate and candidate random (the state evolves), output = [0 | alpha I | 0]
    out = np.zeros((rank, n), np.float32)
    out[:, rank:2 * rank] = alpha * np.eye(rank)
    Wr = _blocks(rank, d, gate=rng.normal(size=(rank, n)), cand=rng.normal(size=(rank, n)),
                 out=out)
    hid = _rand(rng, (R, K, d))
    wc = rng.normal(size=d + rank).astype(np.float32) * 0.2
    U = _base(rng, R, K, V)
    u = rng.random((R, K)).astype(np.float32)
    anc = rng.integers(0, V, R)
    tok, p, conf, mg = oracle.rnn_draft(anc, U, "bf16", W1, W2t, Wr, wc, u, K, V, hidden=hid)
    # the Markov head with W2 scaled by alpha (exact in bf16: a power of two)
    W2s = bf16((widen(W2t) * alpha).astype(np.float32))
    assert np.array_equal(widen(W2s), widen(W2t) * np.float32(alpha))
    tm, pm, cm, mm = oracle.markov_draft(anc, U, "bf16", W1, W2s, wc, u, K, V, hidden=hid)
    # tanh(alpha e) = alpha e (1 - (alpha e)^2 / 3 + ...): the bias differs by
    # at most sum_j |W2| |alpha e_j|^3 / 3 (~1e-5 here), the probabilities by
    # about as much relatively
    e_max = float(np.abs(widen(W1)).max())
    w_max = float(np.abs(widen(W2t)).sum(axis=1).max())
    bound = w_max * (alpha * e_max) ** 3 / 3
    assert bound < 1e-4
    np.testing.assert_allclose(p, pm, rtol=3 * bound, atol=0)
    sure = (mg > 10 * bound) & (mm > 10 * bound)
    assert sure.mean() > 0.8
    assert np.array_equal(tok[sure], tm[sure])
    # the bias is not negligible: the same draws without it differ materially
    _, p0, _, _ = oracle.markov_draft(anc, U, "bf16", W1, np.zeros_like(W2t), wc, u, K, V,
                                      hidden=hid)
    assert np.abs(p - p0).max() > 100 * bound * p.max()
    np.testing.assert_allclose(conf, cm, rtol=1e-13, atol=0)


def test_gate_at_one_keeps_the_state_at_zero():
    rng = np.random.default_rng(13)
    R, K, V, rank, d = 3, 6, 40, 8, 10
    n = 2 * rank + d
    W1 = _rand(rng, (V, rank))
    W2t = _rand(rng, (V, rank), 2.0)
    hid = _rand(rng, (R, K, d), 0.3)
    hid[..., 0] = bf16(np.float32(1.0))  # a constant input
    gate = rng.normal(size=(rank, n)) * 0.1
    gate[:, 2 * rank] = 1000.0  # sigmoid(>= ~990) == 1.0 in fp64
    Wr = _blocks(rank, d, gate=gate, cand=rng.normal(size=(rank, n)),
                 out=rng.normal(size=(rank, n)) * 0.5)
    Wr_nos = Wr.copy().reshape(3 * rank, n)
    Wr_nos[:, :rank] = 0  # the state columns of every part
    wc = rng.normal(size=d + rank).astype(np.float32) * 0.2
    U = _base(rng, R, K, V)
    u = rng.random((R, K)).astype(np.float32)
    anc = rng.integers(0, V, R)
    a = oracle.rnn_draft(anc, U, "bf16", W1, W2t, Wr, wc, u, K, V, hidden=hid)
    b = oracle.rnn_draft(anc, U, "bf16", W1, W2t, Wr_nos, wc, u, K, V, hidden=hid)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
    # the same weights with the gate at 0 (the state is the candidate) do differ
    gate0 = gate.copy()
    gate0[:, 2 * rank] = -1000.0
    Wr0 = _blocks(rank, d, gate=gate0, cand=widen(Wr[rank:2 * rank]), out=widen(Wr[2 * rank:]))
    Wr0_nos = Wr0.copy()
    Wr0_nos[:, :rank] = 0
    c = oracle.rnn_draft(anc, U, "bf16", W1, W2t, Wr0, wc, u, K, V, hidden=hid)
    e = oracle.rnn_draft(anc, U, "bf16", W1, W2t, Wr0_nos, wc, u, K, V, hidden=hid)
    assert np.abs(c[1][:, 1:] - e[1][:, 1:]).max() > 1e-3
    # position 1 sees s_0 = 0 either way
    np.testing.assert_array_equal(c[1][:, 0], e[1][:, 0])


def test_gate_at_zero_carries_the_token_two_places_back():
    rng = np.random.default_rng(14)
    R, K, V, rank, d = 5, 4, 50, 8, 4
    n = 2 * rank + d
    a_c, a_o = 2.0 ** -8, 2.0 ** -8
    W1 = _rand(rng, (V, rank))
    W2t = _rand(rng, (V, rank), 256.0)
    hid = np.zeros((R, K, d), np.uint16)
    hid[..., 0] = bf16(np.float32(1.0))
    gate = np.zeros((rank, n))
    gate[:, 2 * rank] = -1000.0  # sigmoid == 0 exactly: s_k = tanh(candidate)
    cand = np.zeros((rank, n))
    cand[:, rank:2 * rank] = a_c * np.eye(rank)  # candidate = a_c * e_k
    out = np.zeros((rank, n))
    out[:, :rank] = a_o * np.eye(rank)  # output = a_o * s_{k-1}
    Wr = _blocks(rank, d, gate=gate, cand=cand, out=out)
    wc = np.zeros(d + rank, np.float32)
    U = _base(rng, R, K, V)
    u = rng.random((R, K)).astype(np.float32)
    anc = rng.integers(0, V, R)
    tok, p, _, _ = oracle.rnn_draft(anc, U, "bf16", W1, W2t, Wr, wc, u, K, V, hidden=hid)
    Uf = widen(U).astype(np.float64)
    # position 1: s_0 = 0, no bias
    for r in range(R):
        np.testing.assert_allclose(p[r, 0], softmax(Uf[r * K]), rtol=1e-12, atol=0)
    # position k >= 2: biased by W2^T (a_o a_c W1[x_{k-2}]) up to the cubic
    # terms: the Markov head with a scaled projection, run one position later
    # from the token two places back
    W2s = bf16((widen(W2t) * (a_c * a_o)).astype(np.float32))
    e_max = float(np.abs(widen(W1)).max())
    w_max = float(np.abs(widen(W2t)).sum(axis=1).max())
    bound = w_max * a_o * a_c * e_max * ((a_c * e_max) ** 2 + (a_o * a_c * e_max) ** 2)
    prev2 = np.concatenate([anc[:, None], tok], axis=1)  # x_0, x_1, ...
    for k in range(2, K + 1):
        Uk = U.reshape(R, K, V)[:, k - 1].copy()
        _, pm, _, _ = oracle.markov_draft(prev2[:, k - 2], Uk, "bf16", W1, W2s, wc,
                                          np.full((R, 1), 0.5, np.float32), 1, V)
        np.testing.assert_allclose(p[:, k - 1], pm[:, 0], rtol=3 * bound + 1e-12, atol=0)
        # and not the Markov head from the previous token (when it differs)
        _, pw, _, _ = oracle.markov_draft(prev2[:, k - 1], Uk, "bf16", W1, W2s, wc,
                                          np.full((R, 1), 0.5, np.float32), 1, V)
        differ = prev2[:, k - 2] != prev2[:, k - 1]
        assert differ.any()
        assert np.abs(p[differ, k - 1] - pw[differ, 0]).max() > 100 * bound * p.max()


def test_the_state_carries_the_whole_prefix():
    rng = np.random.default_rng(15)
    K, V, rank, d = 3, 30, 8, 6
    n = 2 * rank + d
    W1 = _rand(rng, (V, rank))
    W2t = _rand(rng, (V, rank), 2.0)
    # two requests, different anchors, x_1 forced to the same token by a spike
    anc = np.array([3, 17])
    U = np.zeros((2 * K, V), np.float32)
    U[:, :] = rng.normal(size=(2 * K, V))
    U[[0, K], 5] = 200.0  # position 1 of both requests: token 5
    U[K:] = U[:K]  # identical base logits for both requests
    hid = np.repeat(_rand(rng, (1, K, d)), 2, axis=0)  # identical backbone states
    wc = np.zeros(d + rank, np.float32)
    u = np.full((2, K), 0.5, np.float32)
    Wr = _blocks(rank, d, gate=rng.normal(size=(rank, n)), cand=rng.normal(size=(rank, n)),
                 out=rng.normal(size=(rank, n)))
    tok, p, _, _ = oracle.rnn_draft(anc, U, "f32", W1, W2t, Wr, wc, u, K, V, hidden=hid)
    assert tok[0, 0] == tok[1, 0] == 5
    assert np.abs(p[0, 1] - p[1, 1]).max() > 1e-3  # the anchor still matters at position 2
    Wn = Wr.copy()
    Wn[:, :rank] = 0  # no state columns: first order in the tokens
    tok, p, _, _ = oracle.rnn_draft(anc, U, "f32", W1, W2t, Wn, wc, u, K, V, hidden=hid)
    assert tok[0, 0] == tok[1, 0] == 5
    np.testing.assert_array_equal(p[0, 1], p[1, 1])


def test_a_half_open_gate_remembers_two_tokens_back():
    # gate weights zero: sigmoid(0) = 1/2 exactly, so s_k = (s_{k-1} + tanh(a_c)) / 2;
    # the candidate reads only the embedding, the output only the state.  Two
    # requests that share x_1 and x_2 but not the anchor must still differ at
    # position 3 (s_2 holds half of s_1, which came from the anchor); with the
    # gate at 0 the state forgets and they agree.
    rng = np.random.default_rng(17)
    K, V, rank, d = 3, 30, 8, 2
    n = 2 * rank + d
    W1 = _rand(rng, (V, rank))
    W2t = _rand(rng, (V, rank), 4.0)
    anc = np.array([2, 23])
    U = rng.normal(size=(K, V)).astype(np.float32)
    U[0, 5] = 200.0  # x_1 = 5
    U[1, 9] = 200.0  # x_2 = 9
    U = np.concatenate([U, U])
    hid = np.zeros((2, K, d), np.uint16)
    hid[..., 0] = bf16(np.float32(1.0))
    wc = np.zeros(d + rank, np.float32)
    u = np.full((2, K), 0.5, np.float32)
    cand = np.zeros((rank, n))
    cand[:, rank:2 * rank] = 0.5 * np.eye(rank)
    out = np.zeros((rank, n))
    out[:, :rank] = 2.0 * np.eye(rank)
    half = _blocks(rank, d, cand=cand, out=out)
    tok, p, _, _ = oracle.rnn_draft(anc, U, "f32", W1, W2t, half, wc, u, K, V, hidden=hid)
    assert (tok[:, :2] == [[5, 9], [5, 9]]).all()
    assert np.abs(p[0, 2] - p[1, 2]).max() > 1e-3
    gate = np.zeros((rank, n))
    gate[:, 2 * rank] = -1000.0
    shut = _blocks(rank, d, gate=gate, cand=cand, out=out)
    tok, p, _, _ = oracle.rnn_draft(anc, U, "f32", W1, W2t, shut, wc, u, K, V, hidden=hid)
    assert (tok[:, :2] == [[5, 9], [5, 9]]).all()
    np.testing.assert_array_equal(p[0, 2], p[1, 2])


def test_requests_are_independent():
    rng = np.random.default_rng(16)
    R, K, V, rank, d = 4, 3, 33, 8, 8
    n = 2 * rank + d
    W1 = _rand(rng, (V, rank))
    W2t = _rand(rng, (V, rank))
    Wr = _rand(rng, (3 * rank, n))
    hid = _rand(rng, (R, K, d))
    wc = rng.normal(size=d + rank).astype(np.float32) * 0.2
    U = _base(rng, R, K, V)
    u = rng.random((R, K)).astype(np.float32)
    anc = rng.integers(0, V, R)
    full = oracle.rnn_draft(anc, U, "bf16", W1, W2t, Wr, wc, u, K, V, hidden=hid)
    for r in range(R):
        one = oracle.rnn_draft(anc[r:r + 1], U[r * K:(r + 1) * K], "bf16", W1, W2t, Wr, wc,
                               u[r:r + 1], K, V, hidden=hid[r:r + 1])
        for x, y in zip(full, one):
            assert np.array_equal(x[r], y[0])
