"""GPU parity of speculative acceptance against the oracle: accepted lengths and
emitted tokens bit-exact (greedy, and stochastic on guard-banded inputs), the
analytic acceptance rate within fp32 rounding, the sampler's output law by a
chi-square test, and edge cases."""
import numpy as np
import pytest
from scipy import stats
from scipy.special import softmax

import oracle
from oracle import guard
from paper_2607_05147_amd import synth

from gpu_helpers import gpu_accept, log, to_dev

pytestmark = pytest.mark.gpu


def _compare(case, label):
    acc, nxt, _ = gpu_accept(case.w, case.drafts, case.logits, case.cu_q)
    ok = np.ones(case.w.R, bool)
    ok[case.unguarded] = False
    log(f"[accept] {label}: R={case.w.R} total_q={case.total_q} unguarded={len(case.unguarded)} "
        f"mean accepted={case.accepted_len.mean():.2f}")
    assert ok.mean() > 0.9
    bad = np.nonzero(ok & ((acc != case.accepted_len) | (nxt != case.next_tok)))[0]
    assert bad.size == 0, (label, bad[:10], acc[bad[:10]], case.accepted_len[bad[:10]],
                           nxt[bad[:10]], case.next_tok[bad[:10]])


@pytest.mark.parametrize("name", synth.WORKLOAD_ORDER)
def test_workloads_full_size(name):
    w = synth.WORKLOADS[name]
    case = guard.build_case(w, 1, with_kv=False)
    _compare(case, name)


@pytest.mark.parametrize("name", ["tiny", "mid", "highconc"])
def test_reduced_sizes(name):
    # vocabularies that are not a multiple of the 4096-token chunk, several chunks
    w = synth.scaled(synth.WORKLOADS[name], R=24, V=20000 + 37)
    for seed in (2, 3):
        case = guard.build_case(w, seed, with_kv=False)
        _compare(case, f"{name}/V{w.V}/seed{seed}")


def test_accept_rate_matches_oracle():
    w = synth.scaled(synth.WORKLOADS["mid"], R=12, V=17000)
    case = guard.build_case(w, 4, with_kv=False)
    _, _, _, rate_o = oracle.accept(case.drafts.draft_tok, case.drafts.draft_p, case.logits,
                                    w.logit_dtype, case.cu_q, w.K, w.V, u=case.drafts.u,
                                    want_rate=True)
    acc, nxt, rate = gpu_accept(w, case.drafts, case.logits, case.cu_q, want_rate=True)
    total = case.total_q
    tested = rate_o[:total] >= 0
    assert np.array_equal(rate[:total] < 0, ~tested)
    np.testing.assert_allclose(rate[:total][tested], rate_o[:total][tested], atol=2e-5)


def test_identical_distributions_accept_all():
    rng = np.random.default_rng(3)
    R, K, V = 16, 6, 3000
    z = (rng.normal(size=(R * (K + 1), V)) * 4).astype(np.float32)
    cu = np.arange(R + 1, dtype=np.int32) * (K + 1)
    p = softmax(z.astype(np.float64), axis=1).astype(np.float32)
    dp = np.stack([p[cu[r]: cu[r] + K] for r in range(R)])
    tok = rng.integers(0, V, size=(R, K)).astype(np.int32)
    u = (rng.random((R, K + 1)) * 0.999).astype(np.float32)
    w = synth.scaled(synth.WORKLOADS["mid"], R=R, K=K, V=V)
    acc, nxt, _ = gpu_accept(w, synth.Drafts(tok, dp, u), z, cu)
    assert (acc == K).all()


def test_longest_block_accept_all_with_rate():
    """K = 64: 65 verified rows per request, the bonus draw from row 64, and
    every row's statistics written for the analytic rate (1 here)."""
    rng = np.random.default_rng(12)
    R, K, V = 6, 64, 2500
    z = (rng.normal(size=(R * (K + 1), V)) * 3).astype(np.float32)
    cu = np.arange(R + 1, dtype=np.int32) * (K + 1)
    p = softmax(z.astype(np.float64), axis=1).astype(np.float32)
    dp = np.stack([p[cu[r]: cu[r] + K] for r in range(R)])
    tok = rng.integers(0, V, size=(R, K)).astype(np.int32)
    u = (rng.random((R, K + 1)) * 0.999).astype(np.float32)
    w = synth.scaled(synth.WORKLOADS["mid"], R=R, K=K, V=V)
    acc, nxt, rate = gpu_accept(w, synth.Drafts(tok, dp, u), z, cu, want_rate=True)
    acc_o, nxt_o, mg, rate_o = oracle.accept(tok, dp, z, "f32", cu, K, V, u=u, want_rate=True)
    assert (acc == K).all() and (acc_o == K).all()
    ok = mg >= guard.ACCEPT_GUARD
    log(f"[accept] K=64 accept-all: {ok.sum()} of {R} requests guarded")
    assert ok.sum() >= R // 2
    assert np.array_equal(nxt[ok], nxt_o[ok])
    tested = rate_o >= 0
    assert np.array_equal(rate < 0, ~tested)
    np.testing.assert_allclose(rate[tested], rate_o[tested], atol=2e-5)


def test_wide_vocabulary_rows_one_at_a_time():
    # V = 300007: 74 chunks per row, more than one per lane, so the accept
    # tests fold each row's statistics on their own
    w = synth.scaled(synth.WORKLOADS["mid"], R=4, K=5, V=300007)
    case = guard.build_case(w, 9, with_kv=False)
    _compare(case, f"wide/V{w.V}")
    _, _, _, rate_o = oracle.accept(case.drafts.draft_tok, case.drafts.draft_p, case.logits,
                                    w.logit_dtype, case.cu_q, w.K, w.V, u=case.drafts.u,
                                    want_rate=True)
    _, _, rate = gpu_accept(w, case.drafts, case.logits, case.cu_q, want_rate=True)
    total = case.total_q
    tested = rate_o[:total] >= 0
    assert np.array_equal(rate[:total] < 0, ~tested)
    np.testing.assert_allclose(rate[:total][tested], rate_o[:total][tested], atol=2e-5)


def test_malformed_request_with_rate():
    """A request whose q_len exceeds K + 1 gets accepted_len = next_tok = -1
    and rate -1 on its rows; the others are unaffected (requests are
    independent), checked against the oracle on the unmodified batch."""
    w = synth.scaled(synth.WORKLOADS["mid"], R=6, V=9000)
    case = guard.build_case(w, 13, with_kv=False)
    acc_o, nxt_o, _, rate_o = oracle.accept(case.drafts.draft_tok, case.drafts.draft_p, case.logits,
                                            w.logit_dtype, case.cu_q, w.K, w.V, u=case.drafts.u,
                                            want_rate=True)
    bad = 2
    ql = np.diff(case.cu_q).astype(np.int64)
    ql_m = ql.copy()
    ql_m[bad] = w.K + 2
    cu_m = np.concatenate([[0], np.cumsum(ql_m)]).astype(np.int32)
    rng = np.random.default_rng(5)
    rows = []
    for r in range(w.R):
        if r == bad:
            rows.append((rng.normal(size=(w.K + 2, w.V)) * 4).astype(case.logits.dtype))
        else:
            rows.append(case.logits[case.cu_q[r]:case.cu_q[r + 1]])
    logits_m = np.concatenate(rows)
    acc, nxt, rate = gpu_accept(w, case.drafts, logits_m, cu_m, want_rate=True)
    assert acc[bad] == -1 and nxt[bad] == -1
    assert (rate[cu_m[bad]:cu_m[bad + 1]] == -1).all()
    ok = [r for r in range(w.R) if r != bad and r not in case.unguarded]
    assert np.array_equal(acc[ok], acc_o[ok]) and np.array_equal(nxt[ok], nxt_o[ok])
    for r in range(w.R):
        if r == bad:
            continue
        got = rate[cu_m[r]:cu_m[r + 1]]
        ref = rate_o[case.cu_q[r]:case.cu_q[r + 1]]
        assert np.array_equal(got < 0, ref < 0)
        np.testing.assert_allclose(got[ref >= 0], ref[ref >= 0], atol=2e-5)
    log(f"[accept] malformed request {bad}: -1 everywhere; {len(ok)} others exact")


def test_greedy_ties_and_rejections():
    rng = np.random.default_rng(8)
    R, K, V = 40, 4, 9000
    z = np.round(rng.normal(size=(R * (K + 1), V)) * 2).astype(np.float32)  # many ties
    cu = np.arange(R + 1, dtype=np.int32) * (K + 1)
    am = np.argmax(z, axis=1)
    tok = np.zeros((R, K), np.int32)
    for r in range(R):
        cut = r % (K + 1)
        for t in range(K):
            tok[r, t] = am[cu[r] + t] if t < cut else (am[cu[r] + t] + 1) % V
    w = synth.scaled(synth.WORKLOADS["tiny"], R=R, K=K, V=V)
    acc, nxt, _ = gpu_accept(w, synth.Drafts(tok, None, None), z, cu)
    acc_o, nxt_o, _, _ = oracle.accept(tok, None, z, "f32", cu, K, V)
    assert np.array_equal(acc, acc_o) and np.array_equal(nxt, nxt_o)


def test_zero_length_requests_and_bonus_only():
    """len = 0 for every request: only the bonus draw happens."""
    w = synth.scaled(synth.WORKLOADS["mid"], R=10, V=9000)
    case = guard.build_case(w, 5, with_kv=False)
    cu = np.arange(w.R + 1, dtype=np.int32)
    keys = [(r, 0) for r in range(w.R)]
    logits = synth.logit_rows(w, 5, keys)
    acc, nxt, _ = gpu_accept(w, case.drafts, logits, cu)
    acc_o, nxt_o, mg, _ = oracle.accept(case.drafts.draft_tok, case.drafts.draft_p, logits,
                                        w.logit_dtype, cu, w.K, w.V, u=case.drafts.u)
    ok = mg >= guard.ACCEPT_GUARD
    assert (acc == 0).all()
    assert np.array_equal(nxt[ok], nxt_o[ok])


def test_sampler_law_chi_square():
    """Emitted first token ~ target law (losslessness) on the GPU sampler."""
    rng = np.random.default_rng(11)
    V, L, N = 16, 2, 8192
    zrow = (rng.normal(size=(L + 1, V)) * 2).astype(np.float32)
    p_d = rng.dirichlet(np.ones(V), size=L).astype(np.float32)
    logits = np.tile(zrow, (N, 1))
    dp = np.ascontiguousarray(np.broadcast_to(p_d, (N, L, V)))
    tok = np.stack([[rng.choice(V, p=p_d[t] / p_d[t].sum()) for t in range(L)]
                    for _ in range(N)]).astype(np.int32)
    cu = np.arange(N + 1, dtype=np.int32) * (L + 1)
    p_t = softmax(zrow.astype(np.float64), axis=1)
    y = []
    for rep in range(6):
        u = rng.random((N, L + 1)).astype(np.float32)
        w = synth.scaled(synth.WORKLOADS["mid"], R=N, K=L, V=V)
        acc, nxt, _ = gpu_accept(w, synth.Drafts(tok, dp, u), logits, cu)
        y.append(np.where(acc >= 1, tok[:, 0], nxt))
    y = np.concatenate(y)
    obs = np.bincount(y, minlength=V)
    exp = p_t[0] * len(y)
    chi = ((obs - exp) ** 2 / exp).sum()
    assert stats.chi2.sf(chi, V - 1) > 1e-4, chi


def test_repeatable():
    w = synth.WORKLOADS["serving"]
    case = guard.build_case(synth.scaled(w, R=32), 6, with_kv=False)
    a1 = gpu_accept(case.w, case.drafts, case.logits, case.cu_q)
    a2 = gpu_accept(case.w, case.drafts, case.logits, case.cu_q)
    assert all(np.array_equal(x, y) for x, y in zip(a1[:2], a2[:2]))


@pytest.mark.parametrize("K,V,greedy", [(0, 1000, False), (0, 1000, True), (4, 1, False),
                                        (4, 1, True)])
def test_degenerate_shapes(K, V, greedy):
    """K = 0 (no drafts: the bonus draw only) and a single-token vocabulary
    (every draft is accepted and the emitted token is 0)."""
    rng = np.random.default_rng(17 + K + V)
    R = 5
    ln = rng.integers(0, K + 1, size=R)
    cu = oracle.cu_from_len(ln)
    z = (rng.normal(size=(int(cu[-1]), V)) * 3).astype(np.float32)
    tok = rng.integers(0, V, size=(R, K)).astype(np.int32)
    if greedy:
        dr = synth.Drafts(tok, None, None)
    else:
        dp = rng.dirichlet(np.ones(V), size=(R, K)).astype(np.float32).reshape(R, K, V)
        u = (rng.random((R, K + 1)) * 0.999).astype(np.float32)
        dr = synth.Drafts(tok, dp, u)
    w = synth.scaled(synth.WORKLOADS["mid"], R=R, K=K, V=V, greedy=greedy)
    acc, nxt, _ = gpu_accept(w, dr, z, cu)
    acc_o, nxt_o, mg, _ = oracle.accept(tok, dr.draft_p, z, "f32", cu, K, V, u=dr.u)
    ok = np.ones(R, bool) if greedy else mg >= guard.ACCEPT_GUARD
    log(f"[accept] K={K} V={V} greedy={greedy}: {ok.sum()} of {R} guarded")
    assert np.array_equal(acc, acc_o)
    assert np.array_equal(nxt[ok], nxt_o[ok])
    if V == 1:
        assert (acc == ln).all() and (nxt == 0).all()


def test_rows_past_the_batch_end():
    """Requests whose rows leave [0, cu_q[R]) get accepted_len = next_tok = -1
    (their rows were not covered by the row pass); the well-formed request is
    exact against the oracle."""
    w = synth.scaled(synth.WORKLOADS["mid"], R=4, V=9000)
    case = guard.build_case(w, 13, with_kv=False)
    ql = np.diff(case.cu_q)
    assert ql[1] >= 2 and not case.unguarded
    # request 0 as scheduled; requests 1 and 2 end past cu_q[R] = ql0 + 1;
    # request 3 runs backwards
    cu_m = np.array([0, ql[0], ql[0] + ql[1], ql[0] + ql[1] + ql[2], ql[0] + 1], np.int32)
    acc, nxt, rate = gpu_accept(w, case.drafts, case.logits, cu_m, want_rate=True)
    assert acc[0] == case.accepted_len[0] and nxt[0] == case.next_tok[0]
    assert acc[1:].tolist() == [-1, -1, -1] and nxt[1:].tolist() == [-1, -1, -1]
    # the one row past request 0 is owned by no well-formed request
    assert rate[ql[0]] == -1
    log("[accept] rows past cu_q[R]: requests 1-3 rejected, request 0 exact")
