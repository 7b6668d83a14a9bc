"""GPU parity of ragged paged verify attention against the fp64 oracle.

Tolerance: per (token, head) row, ||o - o_ref|| / ||o_ref|| <= 1e-5 for fp32
and <= 2e-2 for bf16 inputs (outputs are rounded to the input type).  Reduced
cases are compared in full; the full-size serving and high-concurrency
workloads are compared on sampled rows that cover every request.  Page tails
and unused block-table slots hold NaN, so any read past a context shows up.
"""
import numpy as np
import pytest

import oracle
from oracle import guard
from paper_2607_05147_amd import synth

from gpu_helpers import DevKV, gpu_attention, log, row_rel_err, to_f64

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 2e-2}


def _scale_keys_after(kv, first, factor):
    """Multiplies every cached key (and aliased value) of each request except
    its first `first` tokens by `factor`, a power of two (exact in bf16)."""
    P = kv.k.shape[2]
    for r in range(len(kv.kv_len)):
        npg = (int(kv.kv_len[r]) + P - 1) // P
        for i in range(npg):
            lo = max(0, first - i * P)
            if lo >= P:
                continue
            pg = kv.block_table[r, i]
            for arr in {id(kv.k): kv.k, id(kv.v): kv.v}.values():
                blk = arr[pg, :, lo:, :]
                if arr.dtype == np.uint16:
                    f = (blk.astype(np.uint32) << 16).view(np.float32) * np.float32(factor)
                    arr[pg, :, lo:, :] = (f.view(np.uint32) >> 16).astype(np.uint16)
                else:
                    arr[pg, :, lo:, :] = blk * np.float32(factor)


def _full_compare(w, seed, q_len=None, label="", kv_fn=None):
    if q_len is None:
        case = guard.schedule_case(w, seed)
        cu = case.cu_q
    else:
        cu = oracle.cu_from_len(np.asarray(q_len) - 1)
    qlen = np.diff(cu)
    kv = synth.paged_kv(w, seed)
    if kv_fn is not None:
        kv_fn(kv)
    q = synth.query_rows(w, seed, synth.flat_keys(qlen))
    log(f"[attn] {label} {w.name} R={w.R} Hq={w.Hq}/{w.Hkv} D={w.Dqk}/{w.Dv} "
        f"total_q={int(cu[-1])} kv={int(kv.kv_len.min())}..{int(kv.kv_len.max())}")
    ref, ref_lse = oracle.verify_attn(q, kv.k, kv.v, kv.k_strides, kv.v_strides, kv.block_table,
                                      kv.kv_len, cu, w.Hq, w.Hkv, w.Dqk, w.Dv, w.page, w.scale,
                                      w.dtype)
    out, lse = gpu_attention(w, DevKV(kv, w.dtype == "bf16"), q, cu)
    o = to_f64(out)
    assert np.isfinite(o).all()
    err = row_rel_err(o, ref)
    log(f"[attn]   max row rel err {err.max():.3g}, max |lse err| "
        f"{np.abs(to_f64(lse) - ref_lse).max():.3g}")
    assert err.max() <= TOL[w.dtype]
    np.testing.assert_allclose(to_f64(lse), ref_lse, rtol=0, atol=1e-4 if w.dtype == "bf16" else 1e-5)


def test_tiny_fp32():
    for seed in range(3):
        _full_compare(synth.WORKLOADS["tiny"], seed, label=f"seed{seed}")


@pytest.mark.parametrize("name", ["mid", "serving", "highconc"])
def test_bf16_reduced(name):
    # a few requests with short contexts: several splits, ragged page tails,
    # every q_len from 1 to K+1
    base = synth.WORKLOADS[name]
    w = synth.scaled(base, R=6, kv_dist=("uniform", base.K + 1, 5000))
    q_len = [1, 2, base.K + 1, 5, 3, base.K // 2 + 1]
    _full_compare(w, 21, q_len=q_len, label="reduced")


def test_bf16_long_split_contexts():
    base = synth.WORKLOADS["serving"]
    w = synth.scaled(base, R=3, kv_dist=("uniform", 9000, 16384))
    _full_compare(w, 4, q_len=[17, 1, 9], label="long")


def test_mla_reduced():
    base = synth.WORKLOADS["mla"]
    w = synth.scaled(base, R=2, Hq=16, kv_dist=("uniform", 300, 3000))
    _full_compare(w, 5, q_len=[3, 17], label="mla-small")


def test_mla_split_contexts():
    # several 8192-key splits per row block, ragged row blocks, partial last steps
    base = synth.WORKLOADS["mla"]
    w = synth.scaled(base, R=2, Hq=32, kv_dist=("uniform", 8200, 17000))
    _full_compare(w, 7, q_len=[5, 2], label="mla-splits")


def test_mla_reference_rerun():
    # keys past each request's first 32 score about 16x higher, far above the
    # first step's maximum (the per-row softmax reference) plus 2^32, so every
    # row block, including both splits of the long request, runs again with
    # the observed maxima
    base = synth.WORKLOADS["mla"]
    w = synth.scaled(base, R=2, Hq=16, kv_dist=("uniform", 200, 9000))
    seed, first = 0, 32
    assert synth.kv_lengths(w, seed).max() > 8192  # two splits

    def scale_and_check(kv):
        _scale_keys_after(kv, first, 16.0)
        # precondition: request 1's last query, head 0, scores (log2 units)
        # past the first step exceed the first step's maximum by more than 32
        cu = oracle.cu_from_len(np.array([3, 8]))
        qb = synth.query_rows(w, seed, synth.flat_keys(np.diff(cu)))[int(cu[2]) - 1, 0]
        q = synth.bf16_bits_to_f32(qb).astype(np.float64)
        n = int(kv.kv_len[1])
        keys = np.stack([synth.bf16_bits_to_f32(kv.k[kv.block_table[1, j // w.page], 0, j % w.page])
                         for j in range(n)]).astype(np.float64)
        s2 = keys @ q * w.scale / np.log(2.0)
        assert s2[first:].max() > s2[:first].max() + 32

    _full_compare(w, seed, q_len=[4, 9], label="mla-rerun", kv_fn=scale_and_check)


def test_mla_reference_rerun_one_row():
    # One key of request 1 is set to 160 times the unit direction of one query
    # row (token 6, head 5: row 5 of its 16-row tile, not the tile's first).
    # Only that row's score leaves its reference by more than 2^128 (exp2 would
    # overflow), so the rerun has to be triggered by that row alone.
    base = synth.WORKLOADS["mla"]
    w = synth.scaled(base, R=2, Hq=16, kv_dist=("uniform", 200, 3000))
    seed, q_len, t_star, h_star, j_key = 3, [4, 9], 6, 5, 100
    cu = oracle.cu_from_len(np.array(q_len) - 1)

    def plant(kv):
        assert int(kv.kv_len[1]) - q_len[1] + t_star >= j_key  # the key is visible to the row
        qb = synth.query_rows(w, seed, synth.flat_keys(np.diff(cu)))[int(cu[1]) + t_star, h_star]
        q = synth.bf16_bits_to_f32(qb).astype(np.float64)
        kvec = synth.f32_to_bf16_bits((160.0 * q / np.linalg.norm(q)).astype(np.float32))
        kv.k[kv.block_table[1, j_key // w.page], 0, j_key % w.page] = kvec
        keys = np.stack([synth.bf16_bits_to_f32(kv.k[kv.block_table[1, j // w.page], 0, j % w.page])
                         for j in range(64)]).astype(np.float64)
        s2 = keys @ q * w.scale / np.log(2.0)
        k_star = synth.bf16_bits_to_f32(kvec).astype(np.float64)
        assert (k_star @ q) * w.scale / np.log(2.0) > s2[:32].max() + 128

    _full_compare(w, seed, q_len=q_len, label="mla-rerun-row", kv_fn=plant)


def test_fp32_other_head_dims():
    base = synth.WORKLOADS["tiny"]
    for D, group in ((128, 8), (72, 1), (64, 16)):
        w = synth.scaled(base, Dqk=D, Dv=D, Hq=2 * group, Hkv=2, R=3)
        _full_compare(w, 6, q_len=[1, 4, 9], label=f"D{D}g{group}")


def _sampled_compare(name, seed, n_per_req=3):
    w = synth.WORKLOADS[name]
    case = guard.schedule_case(w, seed)
    cu = case.cu_q
    qlen = np.diff(cu)
    kv = synth.paged_kv(w, seed)
    q = synth.query_rows(w, seed, synth.flat_keys(qlen))
    log(f"[attn] full {name}: total_q={int(cu[-1])} KV {kv.k.nbytes * 2 / 1e9:.2f} GB")
    out, lse = gpu_attention(w, DevKV(kv, True), q, cu)
    rng = np.random.default_rng(seed)
    rows = []
    for r in range(w.R):
        for _ in range(n_per_req):
            rows.append((int(cu[r] + rng.integers(0, qlen[r])), int(rng.integers(0, w.Hq))))
        rows.append((int(cu[r + 1] - 1), int(rng.integers(0, w.Hq))))  # last query of r
    ref, ref_lse = oracle.verify_attn(q, kv.k, kv.v, kv.k_strides, kv.v_strides, kv.block_table,
                                      kv.kv_len, cu, w.Hq, w.Hkv, w.Dqk, w.Dv, w.page, w.scale,
                                      w.dtype, rows=rows)
    o = to_f64(out)
    l = to_f64(lse)
    got = np.stack([o[t, h] for t, h in rows])
    got_lse = np.array([l[t, h] for t, h in rows])
    err = row_rel_err(got, ref)
    log(f"[attn]   {len(rows)} sampled rows, max row rel err {err.max():.3g}")
    assert np.isfinite(o[: int(cu[-1])]).all()
    assert err.max() <= TOL["bf16"]
    np.testing.assert_allclose(got_lse, ref_lse, rtol=0, atol=1e-4)


def test_serving_full_size_sampled():
    _sampled_compare("serving", 0)


def test_mid_full_size_sampled():
    # the mid workload at its full size (32 requests, fp32 logits upstream,
    # bf16 attention): every context fits one split
    _sampled_compare("mid", 0, n_per_req=4)


def test_highconc_full_size_sampled():
    _sampled_compare("highconc", 0, n_per_req=1)


def test_mla_full_size_sampled():
    _sampled_compare("mla", 0, n_per_req=2)


def test_repeatable_bitwise():
    base = synth.WORKLOADS["serving"]
    w = synth.scaled(base, R=8, kv_dist=("uniform", 2000, 9000))
    case = guard.schedule_case(w, 3)
    kv = synth.paged_kv(w, 3)
    q = synth.query_rows(w, 3, synth.flat_keys(case.q_len))
    dkv = DevKV(kv, True)
    o1, l1 = gpu_attention(w, dkv, q, case.cu_q)
    o2, l2 = gpu_attention(w, dkv, q, case.cu_q)
    import torch
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(l1.view(torch.int32), l2.view(torch.int32))


@pytest.mark.parametrize("name", ["tiny", "mid", "mla"])
def test_invalid_requests_left_unwritten(name):
    """A request whose kv_len is shorter than its q_len, or longer than its
    block table covers, is skipped: its output and LSE rows keep what was
    there, and every other request is unaffected (generic, GQA and latent
    paths)."""
    import torch
    from paper_2607_05147_amd import dspark
    from gpu_helpers import to_dev
    over = dict(R=4)
    if name == "mla":
        over = dict(R=3, kv_dist=("uniform", 5000, 12000))
    w = synth.scaled(synth.WORKLOADS[name], **over)
    q_len = [3, 2, 4, 1][: w.R]
    cu = oracle.cu_from_len(np.asarray(q_len) - 1)
    kv = synth.paged_kv(w, 21)
    q = synth.query_rows(w, 21, synth.flat_keys(np.diff(cu)))
    ref, ref_lse = oracle.verify_attn(q, kv.k, kv.v, kv.k_strides, kv.v_strides, kv.block_table,
                                      kv.kv_len, cu, w.Hq, w.Hkv, w.Dqk, w.Dv, w.page, w.scale,
                                      w.dtype)
    bf16 = w.dtype == "bf16"
    dkv = DevKV(kv, bf16)
    kv_bad = kv.kv_len.copy()
    kv_bad[0] = q_len[0] - 1                                 # fewer keys than verify tokens
    kv_bad[2] = kv.block_table.shape[1] * w.page + 1         # beyond the block table
    dkv.kv_len = to_dev(kv_bad)
    qd = to_dev(q, bf16)
    sentinel = 7.0
    out = torch.full((q.shape[0], w.Hq, w.Dv), sentinel, dtype=qd.dtype, device=qd.device)
    lse = torch.full((q.shape[0], w.Hq), sentinel, dtype=torch.float32, device=qd.device)
    dspark.dspark_verify_attn(qd, dkv.k, dkv.v, dkv.ks, dkv.vs, dkv.bt, dkv.kv_len, to_dev(cu),
                              w.max_q, w.Hkv, w.Dv, w.page, w.scale, out=out, lse=lse)
    torch.cuda.synchronize()
    o, l = to_f64(out), to_f64(lse)
    for r in range(w.R):
        rows = slice(cu[r], cu[r + 1])
        if r in (0, 2):
            assert (o[rows] == sentinel).all() and (l[rows] == sentinel).all(), r
        else:
            err = row_rel_err(o[rows], ref[rows])
            assert err.max() <= TOL[w.dtype], (r, err.max())
            np.testing.assert_allclose(l[rows], ref_lse[rows], rtol=0,
                                       atol=1e-4 if bf16 else 1e-5)
    log(f"[attn] invalid requests skipped: {name} R={w.R}, requests 0 and 2 untouched")


@pytest.mark.parametrize("name", ["tiny", "mid", "mla"])
def test_rows_outside_the_batch_left_unwritten(name):
    """Requests whose row range leaves [0, cu_q[R]) -- a negative start, or an
    end past cu_q[R] -- are skipped on every path: their rows, and every row
    past cu_q[R] of buffers sized for R * max_q rows, keep what was there;
    the well-formed requests match the oracle."""
    import torch
    from paper_2607_05147_amd import dspark
    from gpu_helpers import to_dev
    over = dict(R=5)
    if name == "mla":
        over = dict(R=5, kv_dist=("uniform", 5000, 9000))
    w = synth.scaled(synth.WORKLOADS[name], **over)
    kv = synth.paged_kv(w, 23)
    bf16 = w.dtype == "bf16"
    # request 0: rows 0..2; request 1: rows 3..10, past cu_q[R] = 6;
    # request 2: 11 -> 4 (negative length); request 3: rows 4..5; request 4:
    # rows 6..5 (empty, q_len 0)
    cu = np.array([0, 3, 11, 4, 6, 6], np.int32)
    good = {0: (0, 3), 3: (4, 2)}
    rows_total = w.R * w.max_q
    q = synth.query_rows(w, 23, [(0, t) for t in range(rows_total)])
    dkv = DevKV(kv, bf16)
    qd = to_dev(q, bf16)
    sentinel = 7.0
    out = torch.full((rows_total, w.Hq, w.Dv), sentinel, dtype=qd.dtype, device=qd.device)
    lse = torch.full((rows_total, w.Hq), sentinel, dtype=torch.float32, device=qd.device)
    dspark.dspark_verify_attn(qd, dkv.k, dkv.v, dkv.ks, dkv.vs, dkv.bt, dkv.kv_len, to_dev(cu),
                              w.max_q, w.Hkv, w.Dv, w.page, w.scale, out=out, lse=lse)
    torch.cuda.synchronize()
    o, l = to_f64(out), to_f64(lse)
    written = np.zeros(rows_total, bool)
    for r, (q0, ql) in good.items():
        written[q0:q0 + ql] = True
        ref, ref_lse = oracle.verify_attn(q[q0:q0 + ql], kv.k, kv.v, kv.k_strides, kv.v_strides,
                                          kv.block_table[r:r + 1], kv.kv_len[r:r + 1],
                                          np.array([0, ql], np.int32), w.Hq, w.Hkv, w.Dqk, w.Dv,
                                          w.page, w.scale, w.dtype)
        err = row_rel_err(o[q0:q0 + ql], ref)
        assert err.max() <= TOL[w.dtype], (r, err.max())
        np.testing.assert_allclose(l[q0:q0 + ql], ref_lse, rtol=0, atol=1e-4 if bf16 else 1e-5)
    assert (o[~written] == sentinel).all() and (l[~written] == sentinel).all()
    log(f"[attn] rows outside the batch skipped: {name}, only requests 0 and 3 written")


@pytest.mark.parametrize("name,Hq,Hkv,q_len,kv_len", [
    # one query head per KV head; every context exactly its verify block (the
    # first query sees a single key)
    ("mid", 8, 8, [1, 2, 5], [1, 2, 5]),
    # contexts one key past a page, and one key past a 4096-key split
    ("mid", 32, 8, [1, 3, 17], [64, 65, 4097]),
    # latent: a single key; 4097 keys (one split, a partial last step)
    ("mla", 128, 1, [1, 2], [1, 4097]),
    # latent: one key past an 8192-key split, and a last split whose first key
    # some verify rows cannot see (their partials are empty)
    ("mla", 128, 1, [1, 6, 9], [8193, 16385, 8196]),
])
def test_edge_context_lengths(name, Hq, Hkv, q_len, kv_len):
    w = synth.scaled(synth.WORKLOADS[name], R=len(q_len), Hq=Hq, Hkv=Hkv)
    cu = oracle.cu_from_len(np.asarray(q_len) - 1)
    kv = synth.paged_kv(w, 31, kv_len=np.asarray(kv_len, np.int32))
    q = synth.query_rows(w, 31, synth.flat_keys(np.diff(cu)))
    ref, ref_lse = oracle.verify_attn(q, kv.k, kv.v, kv.k_strides, kv.v_strides, kv.block_table,
                                      kv.kv_len, cu, w.Hq, w.Hkv, w.Dqk, w.Dv, w.page, w.scale,
                                      w.dtype)
    out, lse = gpu_attention(w, DevKV(kv, w.dtype == "bf16"), q, cu)
    o = to_f64(out)
    assert np.isfinite(o).all()
    err = row_rel_err(o, ref)
    log(f"[attn] edge lengths {name} Hq={Hq}/{Hkv} q_len={q_len} kv={kv_len}: "
        f"max row rel err {err.max():.3g}")
    assert err.max() <= TOL[w.dtype]
    np.testing.assert_allclose(to_f64(lse), ref_lse, rtol=0, atol=1e-4)
