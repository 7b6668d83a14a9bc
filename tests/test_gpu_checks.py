"""GPU tests of the input checks (dspark_check_*_inputs) through the C ABI.

Each case plants known rule breaks in otherwise valid inputs and expects the
exact first finding {code, request, index, value}: the smallest request, and
within a request the first rule in the documented order.  Batches of 600
requests take the checks over several rounds of 256 requests with a ragged
last round.  With DSPARK_DEBUG=1 the stage wrappers run the check first and
raise before any stage kernel sees the bad value.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import guard
from paper_2607_05147_amd import dspark, synth

from gpu_helpers import DevKV, dev, log, to_dev

pytestmark = pytest.mark.gpu

MAX_Q, PAGE, MAX_PAGES = 9, 16, 12


def _bits(x: float) -> int:
    return int(np.array([x], dtype=np.float32).view(np.int32)[0])


def _verify_case(R=600, seed=3):
    """Valid verify-attention metadata: q_len in 1..MAX_Q, kv_len in
    [q_len, MAX_PAGES*PAGE], pages handed out in a shuffled order; the
    block-table slots a request does not read hold -1 (never looked at)."""
    rng = np.random.default_rng(seed)
    q_len = rng.integers(1, MAX_Q + 1, R).astype(np.int32)
    kv_len = np.maximum(q_len, rng.integers(1, MAX_PAGES * PAGE + 1, R)).astype(np.int32)
    npg = (kv_len + PAGE - 1) // PAGE
    num_pages = int(npg.sum())
    perm = rng.permutation(num_pages).astype(np.int32)
    bt = np.full((R, MAX_PAGES), -1, np.int32)
    off = 0
    for r in range(R):
        bt[r, :npg[r]] = perm[off:off + npg[r]]
        off += npg[r]
    cu = np.concatenate([[0], np.cumsum(q_len)]).astype(np.int32)
    return bt, kv_len, cu, num_pages


def _check_verify(bt, kv_len, cu, num_pages, max_q=MAX_Q):
    found = dspark.check_verify_inputs(to_dev(bt), to_dev(kv_len), to_dev(cu), max_q, PAGE,
                                       num_pages)
    return None if found is None else found[:4]


def test_verify_valid_inputs_pass():
    bt, kv, cu, n = _verify_case()
    assert _check_verify(bt, kv, cu, n) is None
    bt, kv, cu, n = _verify_case(R=1, seed=4)
    assert _check_verify(bt, kv, cu, n) is None


def test_verify_block_table_entry_outside_cache():
    bt, kv, cu, n = _verify_case()
    r = 300
    npg = (int(kv[r]) + PAGE - 1) // PAGE
    bt[r, npg - 1] = n  # one past the last page
    assert _check_verify(bt, kv, cu, n) == (4, r, npg - 1, n)
    bt[r, npg - 1] = -5
    assert _check_verify(bt, kv, cu, n) == (4, r, npg - 1, -5)


def test_verify_unread_slots_are_not_checked():
    bt, kv, cu, n = _verify_case()
    short = [r for r in range(len(kv)) if (int(kv[r]) + PAGE - 1) // PAGE < MAX_PAGES]
    for r in short[:50]:
        bt[r, MAX_PAGES - 1] = 10 ** 9
    assert _check_verify(bt, kv, cu, n) is None


def test_verify_smallest_request_wins():
    bt, kv, cu, n = _verify_case()
    bt[590, 0] = n + 7  # last, ragged round
    assert _check_verify(bt, kv, cu, n) == (4, 590, 0, n + 7)
    kv[450] = MAX_PAGES * PAGE + 1  # third round
    assert _check_verify(bt, kv, cu, n) == (3, 450, 0, MAX_PAGES * PAGE + 1)
    bt[3, 0] = -1  # first round
    assert _check_verify(bt, kv, cu, n) == (4, 3, 0, -1)


def test_verify_rule_order_within_a_request():
    bt, kv, cu, n = _verify_case()
    r = 257
    q_len = np.diff(cu)
    bt[r, 0] = -2
    kv[r] = q_len[r] - 1  # breaks rule 3 as well as rule 4
    assert _check_verify(bt, kv, cu, n) == (3, r, 0, int(q_len[r]) - 1)


def test_verify_q_len_above_max_q():
    bt, kv, cu, n = _verify_case()
    q_len = np.diff(cu)
    r = int(np.argmin(q_len[100:]) + 100)  # keeps the total inside R*max_q
    q_len[r] = MAX_Q + 1
    kv[r] = max(int(kv[r]), MAX_Q + 1)
    npg = (int(kv[r]) + PAGE - 1) // PAGE
    bt[r, :npg] = np.arange(npg)
    cu2 = np.concatenate([[0], np.cumsum(q_len)]).astype(np.int32)
    assert int(cu2[-1]) <= len(kv) * MAX_Q
    assert _check_verify(bt, kv, cu2, n) == (2, r, 0, MAX_Q + 1)


def test_verify_row_offsets():
    bt, kv, cu, n = _verify_case()
    c = cu.copy()
    c[0] = -1
    assert _check_verify(bt, kv, c, n) == (1, 0, 0, -1)
    c = cu.copy()
    r = 411
    c[r + 1] = c[r] - 1  # decreasing
    assert _check_verify(bt, kv, c, n) == (1, r, 1, int(c[r]) - 1)
    # every request at max_q and the offsets shifted by one row: the last
    # request ends one row past R * max_q
    R = len(kv)
    kv2 = np.maximum(kv, MAX_Q).astype(np.int32)
    bt2 = bt.copy()
    for i in range(R):
        npg = (int(kv2[i]) + PAGE - 1) // PAGE
        bt2[i, :npg] = np.arange(npg)
    c = (np.arange(R + 1) * MAX_Q + 1).astype(np.int32)
    assert _check_verify(bt2, kv2, c, n) == (1, R - 1, 1, R * MAX_Q + 1)
    # cu_q[R] below cu_q[R-1]: request R-2 already ends past cu_q[R]
    c = cu.copy()
    c[R] = c[R - 1] - 1
    assert _check_verify(bt, kv, c, n) == (1, R - 2, 1, int(c[R - 1]))


def test_verify_on_a_schedule_and_cache():
    """The metadata of a scheduled tiny step and its KV pool pass."""
    w = synth.WORKLOADS["tiny"]
    case = guard.schedule_case(w, 0)
    kv = synth.paged_kv(w, 0)
    assert w.page == PAGE
    assert _check_verify(kv.block_table, kv.kv_len, case.cu_q, kv.pool_pages, max_q=w.max_q) is None


def _accept_case(R=600, K=8, seed=5):
    rng = np.random.default_rng(seed)
    ln = rng.integers(0, K + 1, R).astype(np.int32)
    u = rng.random((R, K + 1), dtype=np.float32)
    return oracle.cu_from_len(ln).astype(np.int32), u


def _check_accept(cu, u, K):
    found = dspark.check_accept_inputs(to_dev(cu), None if u is None else to_dev(u), K)
    return None if found is None else found[:4]


def test_accept_valid_inputs_pass():
    cu, u = _accept_case()
    assert _check_accept(cu, u, 8) is None
    assert _check_accept(cu, None, 8) is None
    u[:, 0] = 0.0
    u[:, 1] = np.nextafter(np.float32(1), np.float32(0))
    assert _check_accept(cu, u, 8) is None


def test_accept_uniform_outside_range():
    cu, u = _accept_case()
    u[520, 8] = 1.0
    assert _check_accept(cu, u, 8) == (3, 520, 8, _bits(1.0))
    u[201, 3] = -0.25
    assert _check_accept(cu, u, 8) == (3, 201, 3, _bits(-0.25))
    nan = np.float32("nan")
    u[2, 0] = nan
    assert _check_accept(cu, u, 8) == (3, 2, 0, int(np.array([nan]).view(np.int32)[0]))


def test_accept_length_outside_block():
    cu, u = _accept_case()
    ln = np.diff(cu) - 1
    r = int(np.argmin(ln[300:]) + 300)
    ln[r] = 9  # K + 1 drafts
    cu2 = oracle.cu_from_len(ln).astype(np.int32)
    assert int(cu2[-1]) <= 600 * 9
    assert _check_accept(cu2, u, 8) == (2, r, 0, 9)
    ln[r] = 0
    ln[77] = -1  # an empty row span (q_len 0)
    cu3 = np.concatenate([[0], np.cumsum(ln + 1)]).astype(np.int32)
    assert _check_accept(cu3, u, 8) == (2, 77, 0, -1)


def test_accept_row_offsets():
    cu, u = _accept_case()
    c = cu.copy()
    c[600] = 600 * 9 + 1
    assert _check_accept(c, None, 8) == (1, 599, 1, 600 * 9 + 1)


def test_accept_k_zero():
    cu = np.arange(301, dtype=np.int32)
    u = np.full((300, 1), 0.5, np.float32)
    assert _check_accept(cu, u, 0) is None
    u[299, 0] = 1.5
    assert _check_accept(cu, u, 0) == (3, 299, 0, _bits(1.5))


def test_schedule_confidences():
    w = synth.scaled(synth.WORKLOADS["highconc"], R=600)
    conf = synth.confidences(w, 2)
    assert dspark.check_schedule_inputs(to_dev(conf)) is None
    conf[10, 0], conf[11, 1] = 0.0, 1.0  # both ends are inside
    assert dspark.check_schedule_inputs(to_dev(conf)) is None
    conf[333, 5] = np.nextafter(np.float32(1), np.float32(2))
    assert dspark.check_schedule_inputs(to_dev(conf))[:4] == (1, 333, 5, _bits(conf[333, 5]))
    conf[40, 7] = np.float32("nan")
    assert dspark.check_schedule_inputs(to_dev(conf))[:4] == \
        (1, 40, 7, int(conf[40:41, 7].view(np.int32)[0]))
    empty = torch.empty((5, 0), dtype=torch.float32, device=dev())
    assert dspark.check_schedule_inputs(empty) is None


def test_debug_mode_raises_before_attention(monkeypatch):
    w = synth.WORKLOADS["tiny"]
    case = guard.schedule_case(w, 1)
    kv = synth.paged_kv(w, 1)
    qlen = np.diff(case.cu_q)
    q = to_dev(synth.query_rows(w, 1, synth.flat_keys(qlen)))
    dkv = DevKV(kv, False)
    cu = to_dev(case.cu_q)

    def run():
        return dspark.dspark_verify_attn(q, dkv.k, dkv.v, dkv.ks, dkv.vs, dkv.bt, dkv.kv_len, cu,
                                         w.max_q, w.Hkv, w.Dv, w.page, w.scale)

    ref, _ = run()
    monkeypatch.setenv("DSPARK_DEBUG", "1")
    out, _ = run()  # valid inputs: same result with the check in front
    torch.cuda.synchronize()
    assert torch.equal(out, ref)
    dkv.bt[2, 0] = kv.pool_pages  # one page past the cache
    log(f"[checks] debug verify: bad entry at request 2 page 0 -> {kv.pool_pages}")
    with pytest.raises(dspark.DSparkError, match="block-table entry outside the cache"):
        run()


def test_debug_mode_raises_before_accept_and_schedule(monkeypatch):
    monkeypatch.setenv("DSPARK_DEBUG", "1")
    R, K, V = 4, 8, 1024
    cu = to_dev(np.arange(R + 1, dtype=np.int32) * (K + 1))
    tok = torch.zeros((R, K), dtype=torch.int32, device=dev())
    logits = torch.zeros((R * (K + 1), V), dtype=torch.float32, device=dev())
    pd = torch.full((R, K, V), 1.0 / V, dtype=torch.float32, device=dev())
    u = torch.full((R, K + 1), 0.5, dtype=torch.float32, device=dev())
    dspark.dspark_accept(tok, logits, cu, draft_p=pd, u=u)
    u[3, 8] = 1.0
    with pytest.raises(dspark.DSparkError, match="uniform outside"):
        dspark.dspark_accept(tok, logits, cu, draft_p=pd, u=u)
    w = synth.WORKLOADS["tiny"]
    conf = synth.confidences(w, 0)
    conf[1, 2] = -0.5
    with pytest.raises(dspark.DSparkError, match="confidence outside"):
        dspark.dspark_schedule(to_dev(conf), to_dev(synth.sps_table(w)))


def test_draft_uniforms_and_temperatures():
    rng = np.random.default_rng(9)
    R, K = 600, 16
    u = rng.random((R, K), dtype=np.float32)
    temp = (1.0 + 0.05 * np.arange(1, K + 1)).astype(np.float32)
    assert dspark.check_draft_inputs(to_dev(u), to_dev(temp)) is None
    assert dspark.check_draft_inputs(to_dev(u)) is None  # no temperatures: all 1
    u[431, 15] = 1.0
    assert dspark.check_draft_inputs(to_dev(u), to_dev(temp))[:4] == (2, 431, 15, _bits(1.0))
    u[17, 3] = np.float32("inf")
    assert dspark.check_draft_inputs(to_dev(u), to_dev(temp))[:4] == (2, 17, 3, _bits(np.inf))
    temp[6] = 0.0  # a temperature is reported before any uniform
    assert dspark.check_draft_inputs(to_dev(u), to_dev(temp))[:4] == (1, -1, 6, _bits(0.0))


def test_debug_mode_raises_before_the_draft_block(monkeypatch):
    monkeypatch.setenv("DSPARK_DEBUG", "1")
    w = synth.scaled(synth.WORKLOADS["serving"], R=3, K=2, V=256)
    inp = synth.markov_inputs(w, 0, rank=32, d=8)
    args = [to_dev(inp.anchor), to_dev(inp.base), to_dev(inp.W1), to_dev(inp.W2t), to_dev(inp.w_conf)]
    u = to_dev(inp.u)
    dspark.dspark_markov_draft(*args, u, w.K, hidden=to_dev(inp.hidden), sts_temp=to_dev(inp.sts_temp))
    torch.cuda.synchronize()
    u[2, 1] = -0.5
    with pytest.raises(dspark.DSparkError, match="uniform outside"):
        dspark.dspark_markov_draft(*args, u, w.K, hidden=to_dev(inp.hidden), sts_temp=to_dev(inp.sts_temp))
