"""Pins of the oracle's Markov-head draft block (no GPU).

The oracle follows the left-to-right factorisation of the semi-autoregressive
stage (eq. sequential-factorization) with the Markov head's low-rank
transition bias (eq. markov) and the confidence head (eq. confidence).  The
tests pin it against what the mathematics fixes, not against its own formula:

* a zero projection makes every position an independent softmax of the scaled
  base logits (a library softmax);
* an identity embedding with zero base logits turns the head into a
  first-order Markov chain whose transition rows are softmaxes of the
  projection; the measure of the uniforms that produce each token, found by
  bisection on the oracle as a black box, must equal those probabilities, and
  the second draw's measures must follow the first draw's token;
* a uniform distribution draws floor(u * V);
* one-hot confidence weights read single inputs through the sigmoid, which
  fixes the concatenation order, the indexing and the per-position
  temperature;
* requests are independent of each other.
"""
import math

import numpy as np
import pytest
from scipy.special import softmax

import oracle
from paper_2607_05147_amd import synth

bf16 = synth.f32_to_bf16_bits


def _weights(rng, V, rank, scale=1.0):
    W1 = bf16((rng.normal(size=(V, rank)) * scale).astype(np.float32))
    W2t = bf16((rng.normal(size=(V, rank)) * scale).astype(np.float32))
    return W1, W2t


def _inv_cdf(p, u):
    """Smallest v whose running mass exceeds u * total (numpy, fp64)."""
    c = np.cumsum(p)
    return int(np.searchsorted(c, u * c[-1], side="right"))


def test_zero_projection_is_an_independent_softmax():
    rng = np.random.default_rng(1)
    R, K, V, rank = 3, 4, 50, 8
    W1, _ = _weights(rng, V, rank)
    W2t = np.zeros((V, rank), dtype=np.uint16)  # bf16 +0
    U = bf16((4 * rng.normal(size=(R * K, V))).astype(np.float32))
    u = rng.random((R, K)).astype(np.float32)
    it = 0.7
    tok, p, _, _ = oracle.markov_draft(rng.integers(0, V, R), U, "bf16", W1, W2t,
                                       np.zeros(rank, np.float32), u, K, V, inv_temperature=it)
    Uf = synth.bf16_bits_to_f32(U).astype(np.float64)
    itf = float(np.float32(it))
    for r in range(R):
        for k in range(K):
            ref = softmax(itf * Uf[r * K + k])
            np.testing.assert_allclose(p[r, k], ref, rtol=1e-12, atol=0)
            assert tok[r, k] == _inv_cdf(ref, float(u[r, k]))


def _first_change(f, lo, hi, iters=60):
    """Smallest u in (lo, hi] with f(u) != f(lo), by bisection (f piecewise constant)."""
    a = f(lo)
    for _ in range(iters):
        mid = 0.5 * (lo + hi)
        if f(mid) == a:
            lo = mid
        else:
            hi = mid
    return hi


def _bucket_measures(f, V):
    """Lengths of the u-intervals of [0, 1) on which f takes each value."""
    meas = np.zeros(V)
    lo = 0.0
    while lo < 1.0:
        v = f(lo)
        hi = _first_change(f, lo, 1.0 - 1e-9) if f(1.0 - 1e-9) != v else 1.0
        meas[v] += hi - lo
        lo = hi
    return meas


def test_identity_embedding_is_a_markov_chain():
    # W1 = I, U = 0: the bias of position k is row x_{k-1} of the projection,
    # so the draft is a Markov chain with transitions P[a, :] = softmax(T[a, :])
    V = rank = 3
    T = np.array([[0.5, -1.25, 2.0], [1.5, 0.25, -0.75], [-2.0, 1.0, 0.125]], dtype=np.float32)
    W1 = bf16(np.eye(V, dtype=np.float32))
    W2t = bf16(np.ascontiguousarray(T.T))  # W2[j, v] = T[j, v]; rows of W2t are columns of W2
    U = np.zeros((2, V), dtype=np.float32)
    P = softmax(T.astype(np.float64), axis=1)
    x0 = 2

    def draw(u1, u2):
        tok, _, _, _ = oracle.markov_draft(np.array([x0]), U, "f32", W1, W2t,
                                           np.zeros(rank, np.float32),
                                           np.array([[u1, u2]], dtype=np.float64), 2, V,
                                           want_p=False)
        return tok[0]

    # the first draw follows row x0 (the anchor)
    m1 = _bucket_measures(lambda a: int(draw(a, 0.5)[0]), V)
    np.testing.assert_allclose(m1, P[x0], atol=1e-6)
    # the second draw follows the row of the first draw's token
    edges = np.concatenate([[0.0], np.cumsum(P[x0])])
    for a in range(V):
        u1 = 0.5 * (edges[a] + edges[a + 1])
        assert draw(u1, 0.5)[0] == a
        m2 = _bucket_measures(lambda b: int(draw(u1, b)[1]), V)
        np.testing.assert_allclose(m2, P[a], atol=1e-6)


def test_uniform_distribution_draws_floor_u_times_v():
    rng = np.random.default_rng(3)
    R, K, V, rank = 4, 5, 37, 8
    W1, _ = _weights(rng, V, rank)
    W2t = np.zeros((V, rank), dtype=np.uint16)
    U = np.zeros((R * K, V), dtype=np.float32)
    u = ((rng.integers(0, V, (R, K)) + rng.uniform(0.2, 0.8, (R, K))) / V).astype(np.float32)
    tok, p, _, mg = oracle.markov_draft(rng.integers(0, V, R), U, "f32", W1, W2t,
                                        np.zeros(rank, np.float32), u, K, V)
    uf = u.astype(np.float64)
    np.testing.assert_array_equal(tok, np.floor(uf * V).astype(np.int32))
    np.testing.assert_allclose(p, 1.0 / V, rtol=1e-14)
    frac = uf * V - np.floor(uf * V)
    np.testing.assert_allclose(mg, np.minimum(frac, 1 - frac) / V, rtol=1e-9)


def test_confidence_reads_hidden_then_embedding_with_position_temperature():
    rng = np.random.default_rng(4)
    R, K, V, rank, d = 3, 3, 20, 8, 6
    W1, W2t = _weights(rng, V, rank)
    U = bf16((4 * rng.normal(size=(R * K, V))).astype(np.float32))
    h = bf16(rng.normal(size=(R, K, d)).astype(np.float32))
    u = rng.random((R, K)).astype(np.float32)
    T = np.array([1.0, 2.0, 4.0], dtype=np.float32)
    anchor = rng.integers(0, V, R)
    sig = lambda x: 1.0 / (1.0 + math.exp(-x))

    # zero weights: one half, whatever the inputs
    _, _, c0, _ = oracle.markov_draft(anchor, U, "bf16", W1, W2t, np.zeros(d + rank, np.float32),
                                      u, K, V, hidden=h, sts_temp=T)
    np.testing.assert_array_equal(c0, 0.5)

    # one-hot on hidden dim i: sigmoid(h[r, k, i] / T_k)
    i = 4
    w = np.zeros(d + rank, np.float32)
    w[i] = 1.0
    _, _, ch, _ = oracle.markov_draft(anchor, U, "bf16", W1, W2t, w, u, K, V, hidden=h, sts_temp=T)
    hf = synth.bf16_bits_to_f32(h)
    for r in range(R):
        for k in range(K):
            assert ch[r, k] == pytest.approx(sig(float(hf[r, k, i]) / float(T[k])), rel=1e-14)

    # one-hot on embedding dim j: sigmoid(W1[x_{k-1}, j] / T_k), x_0 = anchor
    j = 5
    w = np.zeros(d + rank, np.float32)
    w[d + j] = 1.0
    tok, _, ce, _ = oracle.markov_draft(anchor, U, "bf16", W1, W2t, w, u, K, V, hidden=h,
                                        sts_temp=T)
    W1f = synth.bf16_bits_to_f32(W1)
    for r in range(R):
        prev = [int(anchor[r])] + [int(x) for x in tok[r, :-1]]
        for k in range(K):
            assert ce[r, k] == pytest.approx(sig(float(W1f[prev[k], j]) / float(T[k])), rel=1e-14)


def test_requests_are_independent():
    rng = np.random.default_rng(5)
    R, K, V, rank, d = 5, 4, 64, 16, 8
    W1, W2t = _weights(rng, V, rank, scale=0.5)
    U = bf16((4 * rng.normal(size=(R * K, V))).astype(np.float32))
    h = bf16(rng.normal(size=(R, K, d)).astype(np.float32))
    w = (rng.normal(size=d + rank) * 0.3).astype(np.float32)
    u = rng.random((R, K)).astype(np.float32)
    anchor = rng.integers(0, V, R)
    tok, p, c, _ = oracle.markov_draft(anchor, U, "bf16", W1, W2t, w, u, K, V, hidden=h)
    perm = rng.permutation(R)
    Up = U.reshape(R, K, V)[perm].reshape(R * K, V)
    tok2, p2, c2, _ = oracle.markov_draft(anchor[perm], Up, "bf16", W1, W2t, w, u[perm], K, V,
                                          hidden=h[perm])
    np.testing.assert_array_equal(tok2, tok[perm])
    np.testing.assert_array_equal(p2, p[perm])
    np.testing.assert_array_equal(c2, c[perm])
    np.testing.assert_allclose(p.sum(axis=-1), 1.0, rtol=1e-13)


def test_inverse_temperature_scales_base_logits_and_bias():
    # the temperature divides the whole logit U_k + B_k: halving both U and
    # the projection (exact, powers of two in fp32 and bf16) at temperature 1
    # must give bit for bit what inverse temperature 0.5 gives on the originals
    rng = np.random.default_rng(11)
    R, K, V, rank = 3, 4, 60, 8
    W1, W2t = _weights(rng, V, rank)
    U = (4 * rng.normal(size=(R * K, V))).astype(np.float32)
    u = rng.random((R, K)).astype(np.float32)
    anchor = rng.integers(0, V, R)
    wc = (rng.normal(size=rank) * 0.1).astype(np.float32)
    tok_a, p_a, c_a, _ = oracle.markov_draft(anchor, U, "f32", W1, W2t, wc, u, K, V,
                                             inv_temperature=0.5)
    W2h = bf16((synth.bf16_bits_to_f32(W2t) * np.float32(0.5)).astype(np.float32))
    assert np.array_equal(synth.bf16_bits_to_f32(W2h) * 2, synth.bf16_bits_to_f32(W2t))
    tok_b, p_b, c_b, _ = oracle.markov_draft(anchor, U * np.float32(0.5), "f32", W1, W2h, wc, u,
                                             K, V, inv_temperature=1.0)
    np.testing.assert_array_equal(tok_a, tok_b)
    np.testing.assert_array_equal(p_a, p_b)
    np.testing.assert_array_equal(c_a, c_b)
    # and the temperature matters: at 1.0 on the originals the distributions differ
    _, p_c, _, _ = oracle.markov_draft(anchor, U, "f32", W1, W2t, wc, u, K, V)
    assert np.abs(p_c - p_a).max() > 1e-3
