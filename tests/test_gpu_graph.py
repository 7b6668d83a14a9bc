"""The verify step (schedule -> attention -> acceptance) captured in a HIP
graph and replayed.

The eager step is checked against the fp64 oracle first (scheduled lengths,
accepted lengths and emitted tokens exact on guarded inputs; GQA attention
rows within the bf16 tolerance), so the replays are compared with a step
known to be right.

The library enqueues kernels only: no memset, allocation or synchronisation.
Its persistent kernels' work counters are reset by their plan kernels on
every call, so a captured step can be replayed as it is.  Each replay follows
eager work and a synchronisation, after the outputs have been overwritten,
and must reproduce the eager step bit for bit.  This holds because the split
merges combine in split order and every other stage is deterministic."""
import numpy as np
import pytest
import torch

import oracle
from oracle import guard
from paper_2607_05147_amd import dspark, synth

from gpu_helpers import DevKV, log, to_dev

pytestmark = pytest.mark.gpu

CASES = {
    # GQA with several splits per context and stochastic acceptance
    "serving": dict(R=8, kv_dist=("uniform", 5000, 13000)),
    # latent attention (V aliases K) with several 4096-key splits
    "mla": dict(R=2, kv_dist=("uniform", 9000, 20000)),
    # greedy acceptance
    "highconc": dict(R=24, kv_dist=("uniform", 600, 3000)),
}


def _step_setup(name, seed=3):
    """Device inputs, outputs and workspaces of one verify step, and a closure
    that enqueues it on the current stream."""
    w = synth.scaled(synth.WORKLOADS[name], **CASES[name])
    case = guard.build_case(w, seed)
    bf16 = w.dtype == "bf16"
    dkv = DevKV(case.kv, bf16)
    dev = torch.device("cuda:0")
    conf, sps = to_dev(case.conf), to_dev(case.sps)
    q = to_dev(case.q, bf16)
    logits = to_dev(case.logits, w.logit_dtype == "bf16")
    tok = to_dev(case.drafts.draft_tok)
    dp = None if case.drafts.draft_p is None else to_dev(case.drafts.draft_p)
    u = None if case.drafts.u is None else to_dev(case.drafts.u)
    R, K = w.R, w.K
    ln = torch.empty(R, dtype=torch.int32, device=dev)
    cu = torch.empty(R + 1, dtype=torch.int32, device=dev)
    out = torch.empty((q.shape[0], w.Hq, w.Dv), dtype=q.dtype, device=dev)
    acc = torch.empty(R, dtype=torch.int32, device=dev)
    nxt = torch.empty(R, dtype=torch.int32, device=dev)
    u8 = torch.uint8
    ws_s = torch.empty(max(dspark.dspark_schedule_workspace_size(R, K), 1), dtype=u8, device=dev)
    ws_a = torch.empty(dspark.dspark_verify_attn_workspace_size(
        R, w.max_q, w.Hq, w.Hkv, w.Dqk, w.Dv, dkv.bt.shape[1], w.page, q.dtype), dtype=u8, device=dev)
    ws_c = torch.empty(dspark.dspark_accept_workspace_size(R, K, w.V), dtype=u8, device=dev)

    def step():
        dspark.dspark_schedule(conf, sps, 0, len_out=ln, cu_q=cu, ws=ws_s)
        dspark.dspark_verify_attn(q, dkv.k, dkv.v, dkv.ks, dkv.vs, dkv.bt, dkv.kv_len, cu, w.max_q,
                                  w.Hkv, w.Dv, w.page, w.scale, out=out, ws=ws_a)
        dspark.dspark_accept(tok, logits, cu, draft_p=dp, u=u, accepted_len=acc, next_tok=nxt,
                             ws=ws_c)

    return w, case, q, step, (ln, cu, out, acc, nxt)


def _check_against_oracle(w, case, outs):
    ln, cu, out, acc, nxt = (t.cpu() for t in outs)
    assert np.array_equal(ln.numpy(), case.len)
    assert np.array_equal(cu.numpy(), case.cu_q)
    ok = np.ones(w.R, bool)
    ok[case.unguarded] = False
    assert np.array_equal(acc.numpy()[ok], case.accepted_len[ok])
    assert np.array_equal(nxt.numpy()[ok], case.next_tok[ok])
    if not w.mla:  # (the latent case's attention is compared in test_gpu_attention.py)
        ref, _ = oracle.verify_attn(case.q, case.kv.k, case.kv.v, case.kv.k_strides, case.kv.v_strides,
                                    case.kv.block_table, case.kv.kv_len, case.cu_q, w.Hq, w.Hkv, w.Dqk,
                                    w.Dv, w.page, w.scale, w.dtype)
        o = out.float().numpy().astype(np.float64)
        err = (np.linalg.norm((o - ref).reshape(-1, w.Dv), axis=1) /
               np.linalg.norm(ref.reshape(-1, w.Dv), axis=1)).max()
        log(f"[graph] {w.name} eager step: attention max row rel err {err:.3g}, "
            f"{int(ok.sum())} of {w.R} requests' acceptance compared")
        assert err <= 2e-2


@pytest.mark.parametrize("name", sorted(CASES))
def test_verify_step_graph_replays(name):
    w, case, q, step, outs = _step_setup(name)
    dev = q.device
    step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in outs]
    _check_against_oracle(w, case, ref)

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    x = torch.randn(256, 256, device=dev)
    for rep in range(3):
        for t in outs:
            t.zero_()
        y = float((x @ x).sum())  # eager work (and a synchronisation) between replays
        g.replay()
        torch.cuda.synchronize()
        same = [torch.equal(t, r) for t, r in zip(outs, ref)]
        log(f"[graph] {name} R={w.R} rows={q.shape[0]} replay {rep}: identical {same} ({y:.1f})")
        assert all(same)


def test_two_steps_on_two_streams_at_once():
    # the library keeps no state between calls: two steps with their own
    # buffers, enqueued on two streams at the same time (default priority),
    # give what each gives alone
    a = _step_setup("serving", 3)
    b = _step_setup("mla", 4)
    refs = []
    for _, _, _, step, outs in (a, b):
        step()
        torch.cuda.synchronize()
        refs.append([t.clone() for t in outs])
    for rep in range(3):
        for _, _, _, _, outs in (a, b):
            for t in outs:
                t.zero_()
        torch.cuda.synchronize()
        s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
        with torch.cuda.stream(s1):
            a[3]()
        with torch.cuda.stream(s2):
            b[3]()
        torch.cuda.synchronize()
        same = [[torch.equal(t, r) for t, r in zip(x[4], ref)] for x, ref in zip((a, b), refs)]
        log(f"[streams] rep {rep}: identical {same}")
        assert all(all(v) for v in same)
