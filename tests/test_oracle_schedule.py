"""Pins for the oracle's Algorithm 1 (hardware-aware prefix scheduler).

Each check comes from outside the oracle: the numbers printed in the paper's
appendix counterexample, numpy's own cumulative product, exhaustive search
over every length vector on tiny batches, and special cases with a closed
answer.
"""
import itertools

import numpy as np
import pytest

import oracle
from paper_2607_05147_amd import synth


def _sps(vals):
    """Table with sps[B] = vals[B-1] (index 0 unused)."""
    return np.array([0.0] + list(vals), dtype=np.float64)


def test_appendix_with_break(appendix):
    sps = _sps([appendix["sps_1"], appendix["sps_2"], appendix["sps_3"]])
    for c2 in (appendix["case1_c2"], appendix["case2_c2"]):
        conf = np.array([[appendix["a_1"], c2]], dtype=np.float32)
        ln, theta, n_adm, _ = oracle.schedule(conf, sps, mode=0)
        assert ln.tolist() == [int(appendix["len_with_break"])]
        assert n_adm == 0
        assert theta == pytest.approx(appendix["theta_0"], abs=1e-12)


def test_appendix_without_break(appendix):
    sps = _sps([appendix["sps_1"], appendix["sps_2"], appendix["sps_3"]])
    conf = np.array([[appendix["a_1"], appendix["case1_c2"]]], dtype=np.float32)
    ln, theta, _, _ = oracle.schedule(conf, sps, mode=1)
    assert ln.tolist() == [int(appendix["case1_len_no_break"])]
    # fp32 confidences 0.8 / 0.9 are inexact: 1e-6 covers their rounding
    assert theta == pytest.approx(appendix["case1_theta_2"], abs=1e-6)
    a = oracle.survival(conf)[0]
    assert a[1] == pytest.approx(appendix["case1_a2"], abs=1e-7)

    conf = np.array([[appendix["a_1"], appendix["case2_c2"]]], dtype=np.float32)
    ln, theta, _, _ = oracle.schedule(conf, sps, mode=1)
    assert ln.tolist() == [int(appendix["case2_len_no_break"])]
    assert theta == pytest.approx(appendix["theta_0"], abs=1e-12)


def test_appendix_theta_values(appendix):
    """Theta_0 = 1.0, Theta_1 = 0.9, and Theta_2 = 1.134 (case 1) / 0.81 (case 2)."""
    sps = _sps([appendix["sps_1"], appendix["sps_2"], appendix["sps_3"]])
    conf = np.array([[appendix["a_1"], appendix["case1_c2"]]], dtype=np.float32)
    *_, tr = oracle.schedule(conf, sps, mode=1, trace=True)
    assert tr.tolist() == pytest.approx(
        [appendix["theta_0"], appendix["theta_1"], appendix["case1_theta_2"]], abs=1e-6)
    *_, tr0 = oracle.schedule(conf, sps, mode=0, trace=True)
    assert tr0.tolist() == pytest.approx([appendix["theta_0"], appendix["theta_1"]], abs=1e-6)
    # case 2: a_2 = 0 leaves the candidate space; a vanishing positive c_2 keeps
    # it in and reproduces the printed Theta_2 = 0.81
    conf = np.array([[appendix["a_1"], 1e-30]], dtype=np.float32)
    *_, tr = oracle.schedule(conf, sps, mode=1, trace=True)
    assert tr[2] == pytest.approx(appendix["case2_theta_2"], abs=1e-6)


def test_survival_is_numpy_cumprod_and_nonincreasing():
    rng = np.random.default_rng(5)
    conf = rng.uniform(0.0, 1.0, size=(64, 16)).astype(np.float32)
    conf[3, 5] = 0.0
    a = oracle.survival(conf)
    ref = np.cumprod(conf.astype(np.float64), axis=1)
    assert np.array_equal(a, ref)
    assert np.all(np.diff(a, axis=1) <= 0)
    assert np.all(a[3, 5:] == 0)


def test_invalid_confidences_are_clamped():
    conf = np.array([[0.5, np.nan, 0.9], [1.5, 0.5, -0.2]], dtype=np.float32)
    a = oracle.survival(conf)
    assert a[0].tolist() == [0.5, 0.0, 0.0]
    assert a[1].tolist() == [1.0, 0.5, 0.0]


def test_flat_profile_admits_everything():
    rng = np.random.default_rng(1)
    R, K = 7, 5
    conf = rng.uniform(0.05, 1.0, size=(R, K)).astype(np.float32)
    sps = np.ones(R * (K + 1) + 1)
    for mode in (0, 1):
        ln, _, n_adm, _ = oracle.schedule(conf, sps, mode)
        assert ln.tolist() == [K] * R
        assert n_adm == R * K


def test_zero_confidence_truncates():
    conf = np.array([[0.9, 0.0, 0.9, 0.9], [0.9, 0.9, 0.9, 0.9]], dtype=np.float32)
    sps = np.ones(2 * 5 + 1)
    ln, _, n_adm, _ = oracle.schedule(conf, sps, 1)
    assert ln.tolist() == [1, 4]
    assert n_adm == 5


def test_equal_throughput_stops():
    """An exact tie Theta_1 == Theta_0 is not an improvement (strict >)."""
    conf = np.array([[0.5, 0.5]], dtype=np.float32)
    sps = np.array([0.0, 1.5, 1.0, 0.5])  # Theta_0 = 1.5, Theta_1 = 1.5*1.0, Theta_2 = 0.875
    for mode in (0, 1):
        ln, theta, _, mm = oracle.schedule(conf, sps, mode)
        assert ln.tolist() == [0]
        assert theta == 1.5
        assert mm == 0.0


def _theta(a, ln, sps):
    R = a.shape[0]
    tau = R + sum(a[r, : ln[r]].sum() for r in range(R))
    return tau * sps[R + int(np.sum(ln))]


def _greedy_path(a):
    """Candidates in descending survival, ties by (r, j): numpy lexsort."""
    R, K = a.shape
    r_idx, j_idx = np.nonzero(a > 0)
    vals = a[r_idx, j_idx]
    order = np.lexsort((j_idx, r_idx, -vals))
    return r_idx[order], j_idx[order] + 1


@pytest.mark.parametrize("seed", range(40))
def test_brute_force_tiny(seed):
    rng = np.random.default_rng(seed)
    R = int(rng.integers(1, 4))
    K = int(rng.integers(1, 5))
    conf = rng.uniform(0.0, 1.0, size=(R, K)).astype(np.float32)
    if seed % 5 == 0:
        conf[0, -1] = 0.0
    # decreasing throughput with a random knee and jitter (not always unimodal)
    T = np.arange(R * (K + 1) + 1)
    knee = int(rng.integers(0, R * (K + 1)))
    sps = 1.0 / (1.0 + rng.uniform(0.02, 0.6) * np.maximum(0, T - knee))
    if seed % 3 == 0:
        sps = sps * (1.0 + 0.05 * rng.uniform(-1, 1, size=sps.shape))
    a = np.cumprod(conf.astype(np.float64), axis=1)

    # exhaustive search over every length vector with a consistent prefix
    best, best_set = -np.inf, []
    for ln in itertools.product(range(K + 1), repeat=R):
        if any(ln[r] > 0 and a[r, ln[r] - 1] <= 0 for r in range(R)):
            continue
        th = _theta(a, ln, sps)
        if th > best + 1e-12:
            best, best_set = th, [ln]
        elif abs(th - best) <= 1e-12:
            best_set.append(ln)

    ln1, th1, _, _ = oracle.schedule(conf, sps, 1)
    assert th1 == pytest.approx(best, rel=1e-12, abs=1e-12)
    assert tuple(ln1.tolist()) in best_set
    assert _theta(a, ln1, sps) == pytest.approx(th1, rel=1e-12)

    # the causal variant: strictly increasing Theta along the greedy path up
    # to its stop, which is the first non-improvement
    ln0, th0, n0, _ = oracle.schedule(conf, sps, 0)
    rs, js = _greedy_path(a)
    cur = np.zeros(R, dtype=int)
    thetas = [_theta(a, cur, sps)]
    for r, j in zip(rs, js):
        cur[r] = j
        thetas.append(_theta(a, cur, sps))
    thetas = np.array(thetas)
    stop = next((n for n in range(1, len(thetas)) if thetas[n] <= thetas[n - 1]), len(thetas))
    assert n0 == stop - 1
    assert th0 == pytest.approx(thetas[n0], rel=1e-12)
    expect = np.zeros(R, dtype=int)
    for r, j in zip(rs[:n0], js[:n0]):
        expect[r] = j
    assert ln0.tolist() == expect.tolist()
    # where Theta is unimodal along the path, the early stop finds the global optimum
    d = np.diff(thetas)
    if np.all(d[: n0] > 0) and np.all(d[n0:] <= 0):
        assert th0 == pytest.approx(best, rel=1e-12)


def test_admitted_set_is_a_threshold_set():
    w = synth.WORKLOADS["serving"]
    conf = synth.confidences(w, 3)
    sps = synth.sps_table(w)
    ln, _, n_adm, _ = oracle.schedule(conf, sps, 0)
    a = np.cumprod(conf.astype(np.float64), axis=1)
    K = w.K
    admitted = np.arange(K)[None, :] < ln[:, None]
    assert admitted.sum() == n_adm
    if admitted.any() and (~admitted & (a > 0)).any():
        assert a[admitted].min() >= a[~admitted & (a > 0)].max()
    assert np.all((ln >= 0) & (ln <= K))


@pytest.mark.parametrize("name", synth.WORKLOAD_ORDER)
def test_workload_schedules_are_sane(name):
    w = synth.WORKLOADS[name]
    conf = synth.confidences(w, 0)
    sps = synth.sps_table(w)
    ln0, th0, _, _ = oracle.schedule(conf, sps, 0)
    ln1, th1, _, _ = oracle.schedule(conf, sps, 1)
    assert np.all((ln0 >= 0) & (ln0 <= w.K))
    assert th1 >= th0  # the global search never does worse along the same path
    assert th0 > w.R * sps[w.R] or ln0.sum() == 0


def test_mode1_keeps_every_candidate_before_its_best_point():
    # two requests, one candidate each: admitting the first lowers Theta
    # (2.9 * 0.6 = 1.74 < 2.0), admitting the second raises it past the start
    # (3.7 * 0.6 = 2.22).  Mode 1 takes the best prefix of the path, so both
    # requests get their candidate; mode 0 stops at the first loss.
    conf = np.array([[0.9], [0.8]], np.float32)
    sps = np.array([0.0, 0.0, 1.0, 0.6, 0.6])
    ln1, th1, n1, _ = oracle.schedule(conf, sps, 1)
    a = conf.astype(np.float64)[:, 0]
    assert ln1.tolist() == [1, 1] and n1 == 2
    assert th1 == pytest.approx((2 + a[0] + a[1]) * 0.6, rel=1e-15)
    ln0, th0, n0, _ = oracle.schedule(conf, sps, 0)
    assert ln0.tolist() == [0, 0] and n0 == 0 and th0 == 2.0


# --------------------------------------------------------------------------
# the asynchronous scheduler: capacity from earlier confidences, then top-K
# admission of the current candidates (section on the scheduler in practice)
# --------------------------------------------------------------------------

def _leading_positive(conf):
    """Closed form of admitting every candidate: the run of confidences > 0
    at the start of each row (NaN, zero and negative end it)."""
    ok = np.nan_to_num(conf.astype(np.float64), nan=-1.0) > 0
    return np.where(ok.all(axis=1), conf.shape[1], np.argmin(ok, axis=1)).astype(np.int32)


def test_appendix_capacities(appendix):
    """The no-break search on the appendix's two realisations admits 2 and 0
    draft tokens: those are the capacities it hands to a later step."""
    sps = _sps([appendix["sps_1"], appendix["sps_2"], appendix["sps_3"]])
    for c2, expect in ((appendix["case1_c2"], appendix["case1_len_no_break"]),
                       (appendix["case2_c2"], appendix["case2_len_no_break"])):
        conf = np.array([[appendix["a_1"], c2]], dtype=np.float32)
        cap, _ = oracle.schedule_capacity(conf, sps)
        assert cap == int(expect)


def test_topk_capacity_extremes():
    rng = np.random.default_rng(11)
    R, K = 9, 6
    conf = rng.uniform(0.0, 1.0, size=(R, K)).astype(np.float32)
    conf[2, 0] = 0.0
    conf[4, 3] = np.nan
    conf[5, 1] = -0.5
    conf[6, 2] = 1.5
    n_pos = int(_leading_positive(conf).sum())
    for cap in (0, -1, -1000):
        ln, n = oracle.schedule_topk(conf, cap)
        assert ln.tolist() == [0] * R and n == 0
    for cap in (n_pos, n_pos + 1, R * K, 10 ** 9):
        ln, n = oracle.schedule_topk(conf, cap)
        assert ln.tolist() == _leading_positive(conf).tolist()
        assert n == n_pos


@pytest.mark.parametrize("seed", range(30))
def test_topk_is_the_first_capacity_candidates_brute_force(seed):
    """For every capacity, the admitted set is the first min(capacity, |E|)
    candidates of numpy's (-a, r, j) ranking; so it is a threshold set of the
    current a, and within a request a prefix."""
    rng = np.random.default_rng(100 + seed)
    R = int(rng.integers(1, 5))
    K = int(rng.integers(1, 6))
    conf = rng.uniform(0.0, 1.0, size=(R, K)).astype(np.float32)
    if seed % 3 == 0:
        conf[rng.integers(0, R), rng.integers(0, K)] = 1.0  # equal survival values
    if seed % 4 == 0:
        conf[:] = np.float32(0.5)  # ties everywhere
    if seed % 5 == 0:
        conf[0, rng.integers(0, K)] = 0.0
    a = np.cumprod(np.clip(conf.astype(np.float64), 0, 1), axis=1)
    rs, js = _greedy_path(a)
    for cap in range(0, R * K + 2):
        ln, n = oracle.schedule_topk(conf, cap)
        take = min(cap, len(rs))
        assert n == take
        expect = np.zeros(R, dtype=int)
        for r, j in zip(rs[:take], js[:take]):
            expect[r] = max(expect[r], j)
        assert ln.tolist() == expect.tolist()
        adm = np.arange(K)[None, :] < ln[:, None]
        assert adm.sum() == take
        rest = ~adm & (a > 0)
        if adm.any() and rest.any():
            assert a[adm].min() >= a[rest].max()


@pytest.mark.parametrize("name", synth.WORKLOAD_ORDER)
def test_topk_with_its_own_capacity_is_mode1(name):
    """With no change of confidences between the two steps, the capacity
    decided by the no-break search and the top-K admission together are the
    no-break search itself."""
    w = synth.WORKLOADS[name]
    sps = synth.sps_table(w)
    for seed in range(2):
        conf = synth.confidences(w, seed)
        cap, _ = oracle.schedule_capacity(conf, sps)
        ln1, _, n1, _ = oracle.schedule(conf, sps, 1)
        assert cap == n1 == int(ln1.sum())
        ln, n = oracle.schedule_topk(conf, cap)
        assert n == cap
        assert ln.tolist() == ln1.tolist()


@pytest.mark.parametrize("seed", range(20))
def test_capacity_is_the_brute_force_optimum_size(seed):
    """The capacity equals the number of draft tokens of the best length
    vector over [0, K]^R (exhaustive search) whenever that best is unique."""
    rng = np.random.default_rng(300 + seed)
    R = int(rng.integers(1, 4))
    K = int(rng.integers(1, 5))
    conf = rng.uniform(0.0, 1.0, size=(R, K)).astype(np.float32)
    T = np.arange(R * (K + 1) + 1)
    knee = int(rng.integers(0, R * (K + 1)))
    sps = 1.0 / (1.0 + rng.uniform(0.02, 0.6) * np.maximum(0, T - knee))
    a = np.cumprod(conf.astype(np.float64), axis=1)
    scored = []
    for ln in itertools.product(range(K + 1), repeat=R):
        scored.append((_theta(a, ln, sps), sum(ln)))
    scored.sort(reverse=True)
    if len(scored) > 1 and scored[0][0] - scored[1][0] <= 1e-12 * scored[0][0]:
        pytest.skip("tied optimum")
    cap, _ = oracle.schedule_capacity(conf, sps)
    assert cap == scored[0][1]


# --------------------------------------------------------------------------
# guard margins and the GPU's summation order
# --------------------------------------------------------------------------

def test_min_margin_is_relative_to_the_best_throughput(appendix):
    """The appendix's first comparison is Theta_1 = 0.9 against Theta_0 = 1.0,
    a relative margin of 0.1; with the table doubled the absolute gap doubles
    and the margin (relative) stays 0.1.  Mode 1 also compares Theta_2 = 1.134
    (margin 0.134), so its minimum is still the first comparison's."""
    base = [appendix["sps_1"], appendix["sps_2"], appendix["sps_3"]]
    conf = np.array([[appendix["a_1"], appendix["case1_c2"]]], dtype=np.float32)
    for scale in (1.0, 2.0, 0.25):
        sps = _sps([scale * v for v in base])
        for mode in (0, 1):
            _, _, _, mm = oracle.schedule(conf, sps, mode)
            assert mm == pytest.approx(0.1, abs=1e-7)
    _, mm = oracle.schedule_capacity(conf, _sps(base))
    assert mm == pytest.approx(0.1, abs=1e-7)


def _tau_in_gpu_order(a_flat, R):
    """tau_n as the scheduler kernel forms it: for candidate x, sixteen lanes
    s = 0..15 each add (in increasing flat index y, y = s mod 16) the a_y that
    come before x in the admission order, the sixteen partial sums are
    combined by a butterfly (offsets 8, 4, 2, 1), then tau = R + (sum + a_x).
    Sums are sequential fp64 additions (cumsum), one per element."""
    N = a_flat.size
    pad = (-N) % 16
    a = np.concatenate([a_flat, np.zeros(pad)])
    idx = np.arange(a.size)
    out = np.empty(N)
    for c0 in range(0, N, 256):
        xs = np.arange(c0, min(N, c0 + 256))
        ax = a_flat[xs][:, None]
        before = np.where(idx[None, :] < xs[:, None], a[None, :] >= ax, a[None, :] > ax)
        v = np.where(before & (idx[None, :] < N), a[None, :], 0.0)
        lanes = np.cumsum(v.reshape(len(xs), -1, 16), axis=1)[:, -1, :]  # [x, 16]
        for o in (8, 4, 2, 1):
            lanes = lanes + lanes[:, np.arange(16) ^ o]
        out[xs - c0 + c0] = R + (lanes[:, 0] + a_flat[xs])
    return out


def test_gpu_summation_order_stays_inside_the_guard_band():
    """The guard band of the scheduler's parity cases (1e-9 relative) rests on
    the GPU's summation order changing Theta by far less.  Recompute tau in
    that order at the largest size (R*K = 8192) and compare every Theta_n
    with the oracle's sequential one."""
    from oracle import guard
    w = synth.scaled(synth.WORKLOADS["highconc"], R=1024, K=8, knee=1536)
    conf = synth.confidences(w, 7)
    sps = synth.sps_table(w)
    a = np.cumprod(np.clip(conf.astype(np.float64), 0, 1), axis=1).reshape(-1)
    tau = _tau_in_gpu_order(a, w.R)
    # position of each candidate in the admission order
    order = np.lexsort((np.arange(a.size), -a))
    order = order[a[order] > 0]
    *_, trace = oracle.schedule(conf, sps, 1, trace=True)
    n = np.arange(len(order))
    theta_gpu = tau[order] * sps[w.R + n + 1]
    rel = np.abs(theta_gpu - trace[1:]) / trace[1:]
    assert len(order) == a.size == 8192
    assert rel.max() <= 1e-11, rel.max()
    assert rel.max() < guard.SCHED_GUARD / 100
