"""GPU parity of the scheduler kernel against the oracle (bit-exact lengths,
cu_q and token -> request marker) on every workload and on edge cases."""
import numpy as np
import pytest

import oracle
from oracle import guard
from paper_2607_05147_amd import synth

from gpu_helpers import gpu_schedule, log

pytestmark = pytest.mark.gpu


def _check(conf, sps, mode, label):
    ln_o, _, _, mm = oracle.schedule(conf, sps, mode)
    R, K = conf.shape
    log(f"[schedule] {label} R={R} K={K} mode={mode} margin={mm:.3g}")
    ln_g, cu_g, tok_g = gpu_schedule(conf, sps, mode)
    assert np.array_equal(ln_g, ln_o), (label, np.nonzero(ln_g != ln_o))
    cu_o = oracle.cu_from_len(ln_o)
    assert np.array_equal(cu_g, cu_o)
    tok_o = np.full(R * (K + 1), -1, np.int32)
    for r in range(R):
        tok_o[cu_o[r]:cu_o[r + 1]] = r
    assert np.array_equal(tok_g, tok_o)
    return mm


@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("name", synth.WORKLOAD_ORDER)
def test_workloads(name, mode):
    w = synth.WORKLOADS[name]
    for seed in range(3):
        case = guard.schedule_case(w, seed, mode=mode)
        assert case.sched_guarded
        _check(case.conf, case.sps, mode, f"{name}/seed{seed}")


def test_appendix_counterexample(appendix):
    sps = np.array([0.0, appendix["sps_1"], appendix["sps_2"], appendix["sps_3"]])
    for c2, mode, expect in ((0.9, 0, 0), (0.0, 0, 0), (0.9, 1, 2), (0.0, 1, 0)):
        conf = np.array([[appendix["a_1"], c2]], np.float32)
        ln, _, _ = gpu_schedule(conf, sps, mode)
        assert ln.tolist() == [expect]


def test_edge_cases():
    rng = np.random.default_rng(0)
    # K = 0: nothing to schedule
    conf = np.zeros((5, 0), np.float32)
    _check(conf, np.ones(6), 0, "K=0")
    # a single request
    conf = rng.uniform(0.3, 1, (1, 16)).astype(np.float32)
    _check(conf, 1.0 / (1 + 0.05 * np.arange(18)), 0, "R=1")
    # all-zero / NaN / negative / >1 confidences
    conf = rng.uniform(0.2, 1, (6, 8)).astype(np.float32)
    conf[0] = 0.0
    conf[1, 3] = np.nan
    conf[2, 0] = -0.5
    conf[3, 2] = 1.7
    sps = 1.0 / (1 + 0.02 * np.maximum(0, np.arange(6 * 9 + 1) - 10))
    _check(conf, sps, 0, "invalid conf")
    _check(conf, sps, 1, "invalid conf")
    # flat profile admits every positive candidate
    conf = rng.uniform(0.05, 1, (7, 5)).astype(np.float32)
    ln, _, _ = gpu_schedule(conf, np.ones(7 * 6 + 1), 0)
    assert ln.tolist() == [5] * 7
    # equal confidences everywhere: ties broken by request, then position
    conf = np.full((64, 8), 0.75, np.float32)
    sps = 1.0 / (1 + np.maximum(0, np.arange(64 * 9 + 1) - 100) / 128.0)
    _check(conf, sps, 0, "ties")
    _check(conf, sps, 1, "ties")


@pytest.mark.parametrize("R,K", [(512, 16), (8192, 1), (1024, 8), (33, 7)])
def test_sizes(R, K):
    """Largest candidate counts (R*K = 8192) and ragged, non-power-of-two sizes."""
    w = synth.scaled(synth.WORKLOADS["highconc"], R=R, K=K, knee=R + R // 2)
    for mode in (0, 1):
        case = guard.schedule_case(w, 7, mode=mode)
        if not case.sched_guarded:
            pytest.skip("no guarded draw")
        _check(case.conf, case.sps, mode, f"R{R}K{K}")


def test_mode1_keeps_the_prefix_before_its_best_point():
    # the first admission loses throughput, the second gains past the start:
    # mode 1 admits both requests, mode 0 neither (the oracle's pin, on the GPU)
    conf = np.array([[0.9], [0.8]], np.float32)
    sps = np.array([0.0, 0.0, 1.0, 0.6, 0.6])
    assert gpu_schedule(conf, sps, 1)[0].tolist() == [1, 1]
    assert gpu_schedule(conf, sps, 0)[0].tolist() == [0, 0]
    _check(conf, sps, 1, "dip then gain")


# --------------------------------------------------------------------------
# asynchronous scheduler: capacity from earlier confidences, top-K admission
# --------------------------------------------------------------------------

def _check_topk(conf, capacity, label):
    from gpu_helpers import gpu_topk
    ln_o, n_o = oracle.schedule_topk(conf, int(capacity))
    R, K = conf.shape
    log(f"[schedule-topk] {label} R={R} K={K} capacity={int(capacity)} admitted={n_o}")
    ln_g, cu_g, tok_g = gpu_topk(conf, capacity)
    assert np.array_equal(ln_g, ln_o), (label, np.nonzero(ln_g != ln_o))
    cu_o = oracle.cu_from_len(ln_o)
    assert np.array_equal(cu_g, cu_o)
    tok_o = np.full(R * (K + 1), -1, np.int32)
    for r in range(R):
        tok_o[cu_o[r]:cu_o[r + 1]] = r
    assert np.array_equal(tok_g, tok_o)


@pytest.mark.parametrize("name", synth.WORKLOAD_ORDER)
def test_capacity_then_topk_workloads(name):
    """The device capacity (no-break search on earlier confidences) is exact,
    and the top-K admission that reads it on the device gives exact lengths,
    cu_q and token markers, on every workload and 3 seeds."""
    from gpu_helpers import gpu_capacity, gpu_topk
    w = synth.WORKLOADS[name]
    for seed in range(3):
        case = guard.capacity_case(w, seed)
        assert case.guarded
        log(f"[schedule-capacity] {name}/seed{seed} capacity={case.capacity} "
            f"margin={case.margin:.3g}")
        cap_d = gpu_capacity(case.conf_prev, case.sps)
        ln_g, cu_g, tok_g = gpu_topk(case.conf, cap_d)  # reads the capacity on the device
        assert int(cap_d.item()) == case.capacity
        assert np.array_equal(ln_g, case.len)
        assert np.array_equal(cu_g, case.cu_q)
        R, K = case.conf.shape
        tok_o = np.full(R * (K + 1), -1, np.int32)
        for r in range(R):
            tok_o[case.cu_q[r]:case.cu_q[r + 1]] = r
        assert np.array_equal(tok_g, tok_o)


@pytest.mark.parametrize("name", synth.WORKLOAD_ORDER)
def test_capacity_on_the_current_confidences_is_mode1(name):
    from gpu_helpers import gpu_capacity, gpu_topk
    w = synth.WORKLOADS[name]
    case = guard.schedule_case(w, 0, mode=1)
    assert case.sched_guarded
    ln_g, cu_g, _ = gpu_topk(case.conf, gpu_capacity(case.conf, case.sps))
    assert np.array_equal(ln_g, case.len)
    assert np.array_equal(cu_g, case.cu_q)


def test_capacity_appendix(appendix):
    from gpu_helpers import gpu_capacity
    sps = np.array([0.0, appendix["sps_1"], appendix["sps_2"], appendix["sps_3"]])
    for c2, expect in ((appendix["case1_c2"], 2), (appendix["case2_c2"], 0)):
        conf = np.array([[appendix["a_1"], c2]], np.float32)
        assert int(gpu_capacity(conf, sps).item()) == expect


def test_topk_edge_cases():
    rng = np.random.default_rng(3)
    conf = rng.uniform(0.0, 1.0, (37, 9)).astype(np.float32)
    conf[1] = 0.0
    conf[2, 4] = np.nan
    conf[3, 0] = -1.0
    conf[4, 5] = 1.5
    n_pos = oracle.schedule_topk(conf, 10 ** 6)[1]
    for cap in (0, -5, 1, 17, n_pos - 1, n_pos, n_pos + 1, 37 * 9, 2 ** 31 - 1):
        _check_topk(conf, cap, f"capacity {cap}")
    # ties everywhere: admission by request, then position
    _check_topk(np.full((64, 8), 0.75, np.float32), 100, "ties")
    # K = 0
    _check_topk(np.zeros((5, 0), np.float32), 3, "K=0")


@pytest.mark.parametrize("R,K", [(512, 16), (8192, 1), (1024, 8), (33, 7)])
def test_topk_sizes(R, K):
    """Largest candidate counts (R*K = 8192) and ragged sizes, at capacities
    spread over the candidate count."""
    w = synth.scaled(synth.WORKLOADS["highconc"], R=R, K=K, knee=R + R // 2)
    conf = synth.confidences(w, 5)
    for frac in (0.0, 0.1, 0.5, 0.97, 1.2):
        _check_topk(conf, int(frac * R * K), f"R{R}K{K}")
