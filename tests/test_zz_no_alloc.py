"""GPU test of dspark_schedule_noalloc, the scheduler entry point that takes
its workspace from the library's fixed device array instead of an argument.

Its outputs must equal dspark_schedule's bit for bit (and the oracle's) on
consecutive calls whose sizes shrink, so that what the array holds from the
previous call cannot leak into the next; both modes are covered.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import guard
from paper_2607_05147_amd import dspark, synth

from gpu_helpers import dev, log, to_dev

pytestmark = pytest.mark.gpu


def _noalloc(conf, sps, mode):
    R, K = conf.shape
    ln = torch.full((R,), -7, dtype=torch.int32, device=dev())
    cu = torch.full((R + 1,), -7, dtype=torch.int32, device=dev())
    tok = torch.full((R * (K + 1),), -7, dtype=torch.int32, device=dev())
    dspark.dspark_schedule_noalloc(to_dev(conf), to_dev(sps), mode, ln, cu, tok)
    torch.cuda.synchronize()
    return ln.cpu().numpy(), cu.cpu().numpy(), tok.cpu().numpy()


def _with_workspace(conf, sps, mode):
    ln, cu, tok = dspark.dspark_schedule(to_dev(conf), to_dev(sps), mode, want_tok_req=True)
    torch.cuda.synchronize()
    return ln.cpu().numpy(), cu.cpu().numpy(), tok.cpu().numpy()


def _cases():
    big = synth.scaled(synth.WORKLOADS["highconc"], R=1024, K=8, knee=1536)  # R*K = 8192
    for w, seed in ((big, 7), (synth.WORKLOADS["serving"], 1), (synth.WORKLOADS["tiny"], 2)):
        yield w, seed


@pytest.mark.parametrize("mode", [0, 1])
def test_noalloc_matches_the_workspace_entry_point_on_shrinking_calls(mode):
    for w, seed in _cases():
        case = guard.schedule_case(w, seed, mode=mode)
        assert case.sched_guarded
        log(f"[noalloc] mode={mode} R={w.R} K={w.K} seed={seed}")
        got = _noalloc(case.conf, case.sps, mode)
        ref = _with_workspace(case.conf, case.sps, mode)
        for g, r in zip(got, ref):
            assert np.array_equal(g, r)
        assert np.array_equal(got[0], case.len)
        assert np.array_equal(got[1], case.cu_q)


def test_noalloc_rejects_bad_arguments():
    conf = to_dev(np.full((4, 8), 0.5, np.float32))
    sps = to_dev(np.ones(4 * 9 + 1))
    ln = torch.empty(4, dtype=torch.int32, device=dev())
    cu = torch.empty(5, dtype=torch.int32, device=dev())
    with pytest.raises(dspark.DSparkError):
        dspark.dspark_schedule_noalloc(conf, sps, 2, ln, cu)
    with pytest.raises(dspark.DSparkError):
        dspark.dspark_schedule_noalloc(conf, sps[:30], 0, ln, cu)
    # after a rejected call the next valid one still matches
    got = dspark.dspark_schedule_noalloc(conf, sps, 0, ln, cu)
    torch.cuda.synchronize()
    assert got[0].cpu().tolist() == [8, 8, 8, 8]
