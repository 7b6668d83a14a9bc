"""GPU parity of the Markov-head draft block against the fp64 oracle.

Draft tokens are compared exactly, on uniforms guarded so that every draw is
at least 1e-4 of the total mass from its bucket's edges (a draw is a
floating-point decision; the guard is far above the fp32 error of the masses).

Distributions: the transition bias is a sum of ``rank`` products of bf16
values, each exact in fp32, accumulated in fp32, so its error is at most
rank * 2^-24 * sum_j |e_j W2[j, v]| -- about 1.5e-4 at rank 256 with the
synthetic weights (sum ~ 10), typically ~1e-6.  p = exp(z - M) / S carries
that error relatively (plus a few fp32 roundings of exp, the max and the sum),
so entries of p are compared with relative tolerance P_RTOL = 2e-4.
Confidences: c = sigmoid(s / T) moves by at most |ds| / 4; s is an fp32 sum of
d + rank products, compared at C_ATOL = 2e-5.
"""
import numpy as np
import pytest
import torch

from oracle import guard
from paper_2607_05147_amd import dspark, synth

from gpu_helpers import log, to_dev

pytestmark = pytest.mark.gpu

P_RTOL = 2e-4
C_ATOL = 2e-5


# requests of the full-size case that the oracle checks in full: 16 of 128,
# spread over the batch (both ends included)
FULL_SIZE_REQS = [int(x) for x in np.linspace(0, 127, 16).round()]

def _run_gpu(w, case, rank, d, inv_temperature=1.0, anchor=None):
    inp = case.inp
    tok, p, conf = dspark.dspark_markov_draft(
        to_dev(inp.anchor if anchor is None else anchor), to_dev(inp.base), to_dev(inp.W1),
        to_dev(inp.W2t), to_dev(inp.w_conf), to_dev(inp.u), w.K,
        hidden=None if d == 0 else to_dev(inp.hidden), sts_temp=to_dev(inp.sts_temp),
        inv_temperature=inv_temperature)
    torch.cuda.synchronize()
    return tok, p, conf


def _compare(w, case, tok, p, conf, label):
    reqs = [r for r in case.reqs if r not in case.unguarded]
    idx = [case.reqs.index(r) for r in reqs]
    got_tok = tok[reqs].cpu().numpy()
    np.testing.assert_array_equal(got_tok, case.tok[idx])
    got_p = p[reqs].double().cpu().numpy()
    ref_p = case.p[idx]
    rel = np.abs(got_p - ref_p) / np.maximum(ref_p, 1e-300)
    rel[ref_p < 1e-30] = 0.0  # far below anything a draw or the acceptance can see
    got_c = conf[reqs].double().cpu().numpy()
    cerr = np.abs(got_c - case.conf[idx]).max()
    log(f"[draft] {label}: R={w.R} K={w.K} V={w.V} | {len(reqs)} requests compared, "
        f"{len(case.unguarded)} unguarded, min margin {case.margin.min():.2e}; "
        f"max p rel err {rel.max():.2e}, max conf err {cerr:.2e}")
    assert rel.max() <= P_RTOL
    assert cerr <= C_ATOL
    np.testing.assert_allclose(got_p.sum(axis=-1), 1.0, rtol=0, atol=1e-5)


def test_draft_reduced_unaligned_vocabulary():
    # V not a multiple of 4 (one entry at a time), a ragged last tile, rank 64,
    # hidden states and per-position temperatures, bf16 base logits
    w = synth.scaled(synth.WORKLOADS["serving"], R=6, K=4, V=3001)
    case = guard.draft_case(w, 1, rank=64, d=40)
    tok, p, conf = _run_gpu(w, case, 64, 40)
    _compare(w, case, tok, p, conf, "reduced")


def test_draft_vector_path_fp32_base_and_temperature():
    # V and ld multiples of 4 (four entries at a time), fp32 base logits,
    # rank 256, no hidden part, inverse temperature 0.8
    w = synth.scaled(synth.WORKLOADS["mid"], R=5, K=3, V=4096)
    case = guard.draft_case(w, 2, rank=256, d=0, inv_temperature=0.8)
    tok, p, conf = _run_gpu(w, case, 256, 0, inv_temperature=0.8)
    _compare(w, case, tok, p, conf, "vector fp32")


@pytest.mark.parametrize("rank", [32, 128])
def test_draft_other_ranks(rank):
    w = synth.scaled(synth.WORKLOADS["serving"], R=3, K=2, V=1000)
    case = guard.draft_case(w, 3, rank=rank, d=16)
    tok, p, conf = _run_gpu(w, case, rank, 16)
    _compare(w, case, tok, p, conf, f"rank {rank}")


@pytest.mark.parametrize("R,K", [(150, 2), (300, 3)])
def test_draft_several_request_chunks(R, K):
    # more requests than one cooperative launch takes: groups of 128 (the last
    # partial), one launch per group and position, their grid barriers
    # numbered across the block (three groups x three positions: nine launches)
    w = synth.scaled(synth.WORKLOADS["serving"], R=R, K=K, V=1024)
    case = guard.draft_case(w, 4, rank=64, d=8)
    tok, p, conf = _run_gpu(w, case, 64, 8)
    _compare(w, case, tok, p, conf, f"{R} requests")


def test_draft_wide_vocabulary():
    # 1563 vocabulary tiles: the per-request statistics take 32 tiles per lane
    # (the serving vocabulary has 1010 tiles, 16 per lane)
    w = synth.scaled(synth.WORKLOADS["serving"], R=3, K=2, V=200003)
    case = guard.draft_case(w, 9, rank=64, d=16)
    tok, p, conf = _run_gpu(w, case, 64, 16)
    _compare(w, case, tok, p, conf, "wide vocabulary")


def test_draft_wide_aligned_vocabulary():
    # bf16 base logits and V % 4 == 0 but 1094 tiles: more than one
    # cooperative grid holds, so each position takes the three-launch form
    w = synth.scaled(synth.WORKLOADS["serving"], R=5, K=2, V=140000)
    case = guard.draft_case(w, 10, rank=128, d=16)
    tok, p, conf = _run_gpu(w, case, 128, 16)
    _compare(w, case, tok, p, conf, "wide aligned vocabulary")


def test_draft_invalid_anchor():
    # anchors outside [0, V) mark their requests: tokens -1, confidences NaN;
    # the other requests are unaffected
    w = synth.scaled(synth.WORKLOADS["serving"], R=5, K=3, V=777)
    case = guard.draft_case(w, 5, rank=64, d=8)
    anchor = case.inp.anchor.copy()
    anchor[1], anchor[3] = -1, w.V
    tok, p, conf = _run_gpu(w, case, 64, 8, anchor=anchor)
    t = tok.cpu().numpy()
    c = conf.cpu().numpy()
    assert (t[[1, 3]] == -1).all() and np.isnan(c[[1, 3]]).all()
    assert np.isfinite(p[[1, 3]].cpu().numpy()).all()
    keep = [0, 2, 4]
    np.testing.assert_array_equal(t[keep], case.tok[keep])
    assert np.abs(c[keep] - case.conf[keep]).max() <= C_ATOL


def test_draft_full_size_sampled():
    # the serving shape: 128 requests, 16 positions, V = 129280, rank 256,
    # 4096-wide hidden states; the oracle checks 16 requests spread over the batch in full
    w = synth.WORKLOADS["serving"]
    case = guard.draft_case(w, 0, rank=256, d=4096, reqs=FULL_SIZE_REQS)
    tok, p, conf = _run_gpu(w, case, 256, 4096)
    _compare(w, case, tok, p, conf, "full size")
    assert ((tok >= 0) & (tok < w.V)).all().item()
    c = conf.cpu().numpy()
    assert ((c > 0) & (c < 1)).all()


@pytest.mark.parametrize("R,K,V", [(1, 1, 700), (3, 1, 129), (2, 5, 5), (2, 3, 1), (2, 64, 300)])
def test_draft_degenerate_shapes(R, K, V):
    # one request; one position (no next embedding to gather); a vocabulary
    # smaller than one tile, down to a single token; the longest block
    w = synth.scaled(synth.WORKLOADS["serving"], R=R, K=K, V=V)
    case = guard.draft_case(w, 8, rank=64, d=16)
    tok, p, conf = _run_gpu(w, case, 64, 16)
    _compare(w, case, tok, p, conf, f"R={R} K={K} V={V}")
    if V == 1:
        assert (tok == 0).all().item() and torch.equal(p, torch.ones_like(p))
