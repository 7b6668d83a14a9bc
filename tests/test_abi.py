"""C ABI checks that need no GPU.

The library must load on a host without a GPU, export every function that
include/dspark.h declares, and reject bad arguments with the documented
status before it touches HIP (every call here fails validation, so nothing is
launched).
"""
import ctypes as C
import os
import re

import pytest

from paper_2607_05147_amd import dspark

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dspark.h")

EINVAL, ESHAPE, EDTYPE, EUNSUPPORTED, EWORKSPACE = 1, 2, 3, 4, 5
FAKE = C.c_void_p(1 << 20)  # aligned, never dereferenced: validation fails first


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(dspark.LIB_PATH):
        from paper_2607_05147_amd import build
        build.build()
    return dspark.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dspark_[a-z_]+)\s*\(", text)))


def test_header_declares_the_three_stages():
    names = declared_functions()
    for n in ("dspark_schedule", "dspark_verify_attn", "dspark_accept", "dspark_abi_version",
              "dspark_last_error"):
        assert n in names


def test_library_exports_every_declared_symbol(L):
    for name in declared_functions():
        assert hasattr(L, name), name


def test_abi_version_matches_header(L):
    m = re.search(r"#define DSPARK_ABI_VERSION (\d+)", open(HEADER).read())
    assert L.dspark_abi_version() == int(m.group(1))


def _sched(L, conf=FAKE, R=4, K=8, sps=FAKE, sps_len=100, mode=0, ln=FAKE, ws=FAKE,
           ws_bytes=None):
    if ws_bytes is None:
        ws_bytes = L.dspark_schedule_workspace_size(R, K)
    return L.dspark_schedule(conf, R, K, sps, sps_len, mode, ln, None, None, ws, ws_bytes, None)


def test_schedule_validation(L):
    assert _sched(L, conf=None) == EINVAL
    assert _sched(L, sps=None) == EINVAL
    assert _sched(L, ln=None) == EINVAL
    assert _sched(L, R=0) == EINVAL
    assert _sched(L, K=65) == EINVAL
    assert _sched(L, K=-1) == EINVAL
    assert _sched(L, mode=2) == EINVAL
    assert _sched(L, sps_len=36) == ESHAPE  # must exceed R*(K+1) = 36
    assert _sched(L, R=8192, K=2, sps_len=10**6) == EUNSUPPORTED
    assert _sched(L, conf=C.c_void_p((1 << 20) + 2)) == EINVAL  # misaligned


def test_schedule_noalloc_validation(L):
    def na(conf=FAKE, R=4, K=8, sps=FAKE, sps_len=100, mode=0, ln=FAKE):
        return L.dspark_schedule_noalloc(conf, R, K, sps, sps_len, mode, ln, None, None, None)

    assert na(conf=None) == EINVAL
    assert na(sps=None) == EINVAL
    assert na(ln=None) == EINVAL
    assert na(R=0) == EINVAL
    assert na(K=65) == EINVAL
    assert na(mode=2) == EINVAL
    assert na(sps_len=36) == ESHAPE
    assert na(R=8192, K=2, sps_len=10**6) == EUNSUPPORTED
    assert na(ln=C.c_void_p((1 << 20) + 2)) == EINVAL


def test_schedule_capacity_validation(L):
    need = L.dspark_schedule_workspace_size(4, 8)

    def cap(conf=FAKE, R=4, K=8, sps=FAKE, sps_len=100, out=FAKE, ws=FAKE, ws_bytes=need):
        return L.dspark_schedule_capacity(conf, R, K, sps, sps_len, out, ws, ws_bytes, None)

    assert cap(conf=None) == EINVAL
    assert cap(sps=None) == EINVAL
    assert cap(out=None) == EINVAL
    assert cap(R=0) == EINVAL
    assert cap(K=65) == EINVAL
    assert cap(sps_len=36) == ESHAPE
    assert cap(R=8192, K=2, sps_len=10**6) == EUNSUPPORTED
    assert cap(out=C.c_void_p((1 << 20) + 2)) == EINVAL
    assert cap(ws=None) == EWORKSPACE
    assert cap(ws_bytes=need - 1) == EWORKSPACE


def test_schedule_topk_validation(L):
    need = L.dspark_schedule_workspace_size(4, 8)

    def topk(conf=FAKE, R=4, K=8, capacity=FAKE, ln=FAKE, ws=FAKE, ws_bytes=need):
        return L.dspark_schedule_topk(conf, R, K, capacity, ln, None, None, ws, ws_bytes, None)

    assert topk(conf=None) == EINVAL
    assert topk(capacity=None) == EINVAL
    assert topk(ln=None) == EINVAL
    assert topk(R=0) == EINVAL
    assert topk(K=-1) == EINVAL
    assert topk(R=8192, K=2) == EUNSUPPORTED
    assert topk(capacity=C.c_void_p((1 << 20) + 1)) == EINVAL
    assert topk(ws=C.c_void_p((1 << 20) + 64)) == EWORKSPACE
    assert topk(ws_bytes=need - 1) == EWORKSPACE


def test_schedule_workspace(L):
    need = L.dspark_schedule_workspace_size(4, 8)
    assert need >= 16 + 12 * 32 and need % 256 == 0
    assert L.dspark_schedule_workspace_size(0, 8) == 0
    assert _sched(L, ws=None) == EWORKSPACE
    assert _sched(L, ws_bytes=need - 1) == EWORKSPACE
    assert _sched(L, ws=C.c_void_p((1 << 20) + 64)) == EWORKSPACE  # not 256-aligned


def test_last_error_describes_failure(L):
    assert _sched(L, sps_len=36) == ESHAPE
    assert "sps_len" in L.dspark_last_error().decode()


def _attn(L, **kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, ks=(C.c_int64 * 3)(8 * 64 * 128, 64 * 128, 128),
             vs=(C.c_int64 * 3)(8 * 64 * 128, 64 * 128, 128), bt=FAKE, max_pages=4, kv=FAKE,
             cu=FAKE, R=4, max_q=9, Hq=32, Hkv=8, Dqk=128, Dv=128, page=64, scale=0.1, dt=1,
             out=FAKE, lse=None, ws=FAKE, ws_bytes=0)
    a.update(kw)
    return L.dspark_verify_attn(a["q"], a["k"], a["v"], a["ks"], a["vs"], a["bt"], a["max_pages"],
                                a["kv"], a["cu"], a["R"], a["max_q"], a["Hq"], a["Hkv"], a["Dqk"],
                                a["Dv"], a["page"], a["scale"], a["dt"], a["out"], a["lse"],
                                a["ws"], a["ws_bytes"], None)


def test_verify_attn_validation(L):
    assert _attn(L, q=None) == EINVAL
    assert _attn(L, bt=None) == EINVAL
    assert _attn(L, ks=None) == EINVAL
    assert _attn(L, dt=7) == EDTYPE
    assert _attn(L, Hq=30) == ESHAPE  # not a multiple of Hkv
    assert _attn(L, Dqk=100) == EUNSUPPORTED
    assert _attn(L, Dv=1024) == EUNSUPPORTED
    assert _attn(L, page=24) == EUNSUPPORTED
    assert _attn(L, max_q=0) == EINVAL
    assert _attn(L, R=0) == EINVAL
    assert _attn(L, ks=(C.c_int64 * 3)(1, 1, 64)) == ESHAPE  # token stride < Dqk
    assert _attn(L, scale=float("nan")) == EINVAL
    assert _attn(L, scale=0.0) == EINVAL
    assert _attn(L, scale=-0.1) == EINVAL
    assert _attn(L, scale=float("inf")) == EINVAL
    assert _attn(L, q=C.c_void_p((1 << 20) + 1)) == EINVAL
    assert _attn(L, ws_bytes=16) == EWORKSPACE  # far too small


def test_verify_attn_workspace_sizes(L):
    f = L.dspark_verify_attn_workspace_size
    mfma = f(128, 17, 64, 8, 128, 128, 256, 64, 1)
    assert mfma > 0
    assert f(4, 9, 8, 2, 64, 64, 8, 16, 0) > 0  # fp32 vector path
    assert f(0, 9, 8, 2, 64, 64, 8, 16, 0) == 0  # invalid shape -> 0


def _acc(L, **kw):
    a = dict(tok=FAKE, dp=FAKE, logits=FAKE, dt=1, ld=1024, u=FAKE, cu=FAKE, R=4, K=8, V=1024,
             it=1.0, acc=FAKE, nxt=FAKE, rate=None, ws=FAKE, ws_bytes=0)
    a.update(kw)
    return L.dspark_accept(a["tok"], a["dp"], a["logits"], a["dt"], a["ld"], a["u"], a["cu"],
                           a["R"], a["K"], a["V"], a["it"], a["acc"], a["nxt"], a["rate"], a["ws"],
                           a["ws_bytes"], None)


def test_accept_validation(L):
    assert _acc(L, dt=5) == EDTYPE
    assert _acc(L, ld=1000) == ESHAPE
    assert _acc(L, it=0.0) == EINVAL
    assert _acc(L, it=float("inf")) == EINVAL
    assert _acc(L, dp=None) == EINVAL  # u without draft_p
    # with K = 0 there is no draft distribution: u alone selects stochastic
    # mode (the call gets as far as the workspace check)
    assert _acc(L, K=0, tok=None, dp=None, ws_bytes=8) == EWORKSPACE
    assert _acc(L, u=None) == EINVAL
    assert _acc(L, dp=None, u=None, rate=FAKE) == EINVAL  # rate needs stochastic mode
    assert _acc(L, logits=None) == EINVAL
    assert _acc(L, K=65) == EINVAL
    assert _acc(L, V=0) == EINVAL
    assert _acc(L, R=0) == EINVAL
    assert _acc(L, ws_bytes=8) == EWORKSPACE
    assert _acc(L, logits=C.c_void_p((1 << 20) + 1)) == EINVAL


def test_input_check_validation(L):
    def cv(bt=FAKE, mp=8, kv=FAKE, cu=FAKE, R=4, mq=9, ps=16, n=100, rep=FAKE):
        return L.dspark_check_verify_inputs(bt, mp, kv, cu, R, mq, ps, n, rep, None)

    assert cv(R=0) == EINVAL
    assert cv(R=8193) == EINVAL
    assert cv(mq=0) == EINVAL
    assert cv(n=0) == EINVAL
    assert cv(ps=0) == EINVAL
    assert cv(mp=1 << 20, ps=1 << 12) == EUNSUPPORTED  # context bound past int32
    assert cv(bt=None) == EINVAL
    assert cv(rep=None) == EINVAL
    assert cv(kv=C.c_void_p((1 << 20) + 2)) == EINVAL

    def ca(cu=FAKE, u=FAKE, R=4, K=8, rep=FAKE):
        return L.dspark_check_accept_inputs(cu, u, R, K, rep, None)

    assert ca(R=0) == EINVAL
    assert ca(K=-1) == EINVAL
    assert ca(K=65) == EINVAL
    assert ca(cu=None) == EINVAL
    assert ca(rep=None) == EINVAL
    assert ca(u=C.c_void_p((1 << 20) + 1)) == EINVAL

    def cs(conf=FAKE, R=4, K=8, rep=FAKE):
        return L.dspark_check_schedule_inputs(conf, R, K, rep, None)

    assert cs(conf=None) == EINVAL  # conf is needed when K > 0
    assert cs(R=8193) == EINVAL
    assert cs(K=65) == EINVAL
    assert cs(rep=None) == EINVAL
    assert cs(rep=C.c_void_p((1 << 20) + 3)) == EINVAL

    def cd(u=FAKE, t=FAKE, R=4, K=8, rep=FAKE):
        return L.dspark_check_draft_inputs(u, t, R, K, rep, None)

    assert cd(u=None) == EINVAL
    assert cd(K=0) == EINVAL  # a draft block has at least one position
    assert cd(R=0) == EINVAL
    assert cd(rep=None) == EINVAL
    assert cd(t=C.c_void_p((1 << 20) + 2)) == EINVAL


def test_accept_workspace_size(L):
    assert L.dspark_accept_workspace_size(128, 16, 129280) > 0
    assert L.dspark_accept_workspace_size(0, 16, 129280) == 0


def _draft(L, **kw):
    a = dict(anchor=FAKE, base=FAKE, dt=1, ld=1024, W1=FAKE, W2t=FAKE, rank=256, hidden=FAKE,
             wc=FAKE, d=64, sts=None, u=FAKE, it=1.0, R=4, K=8, V=1024, tok=FAKE, dp=FAKE,
             conf=FAKE, ws=FAKE, ws_bytes=0)
    a.update(kw)
    return L.dspark_markov_draft(a["anchor"], a["base"], a["dt"], a["ld"], a["W1"], a["W2t"],
                                 a["rank"], a["hidden"], a["wc"], a["d"], a["sts"], a["u"],
                                 a["it"], a["R"], a["K"], a["V"], a["tok"], a["dp"], a["conf"],
                                 a["ws"], a["ws_bytes"], None)


def test_markov_draft_validation(L):
    assert _draft(L, dt=7) == EDTYPE
    assert _draft(L, K=0) == EINVAL
    assert _draft(L, R=0) == EINVAL
    assert _draft(L, V=0) == EINVAL
    assert _draft(L, ld=1000) == ESHAPE
    assert _draft(L, rank=96) == EUNSUPPORTED
    assert _draft(L, V=262145, ld=262145) == EUNSUPPORTED  # tile statistics of a row fit one workgroup
    assert _draft(L, d=-1) == EINVAL
    assert _draft(L, it=0.0) == EINVAL
    assert _draft(L, it=float("inf")) == EINVAL
    assert _draft(L, hidden=None) == EINVAL  # d > 0 needs the hidden states
    assert _draft(L, dp=None) == EINVAL
    assert _draft(L, W2t=C.c_void_p((1 << 20) + 8)) == EUNSUPPORTED  # not 16-byte aligned
    assert _draft(L) == EWORKSPACE  # every argument valid, no workspace
    assert _draft(L, hidden=None, d=0) == EWORKSPACE


def test_markov_draft_workspace_size(L):
    n = L.dspark_markov_draft_workspace_size(128, 16, 129280, 256)
    # two embedding buffers, per-tile statistics (1010 tiles of 128 entries),
    # per-row state, the hidden part of every confidence logit
    assert n >= 2 * 128 * 256 * 2 + 128 * 1010 * 8 + 128 * 24 + 128 * 16 * 4
    assert L.dspark_markov_draft_workspace_size(128, 16, 129280, 96) == 0


def _rnn(L, **kw):
    a = dict(anchor=FAKE, base=FAKE, dt=1, ld=1024, W1=FAKE, W2t=FAKE, Wr=FAKE, rank=256,
             hidden=FAKE, wc=FAKE, d=64, sts=None, u=FAKE, it=1.0, R=4, K=8, V=1024, tok=FAKE,
             dp=FAKE, conf=FAKE, ws=FAKE, ws_bytes=0)
    a.update(kw)
    return L.dspark_rnn_draft(a["anchor"], a["base"], a["dt"], a["ld"], a["W1"], a["W2t"], a["Wr"],
                              a["rank"], a["hidden"], a["wc"], a["d"], a["sts"], a["u"], a["it"],
                              a["R"], a["K"], a["V"], a["tok"], a["dp"], a["conf"], a["ws"],
                              a["ws_bytes"], None)


def test_rnn_draft_validation(L):
    assert _rnn(L, dt=7) == EDTYPE
    assert _rnn(L, K=0) == EINVAL
    assert _rnn(L, R=0) == EINVAL
    assert _rnn(L, V=0) == EINVAL
    assert _rnn(L, ld=1000) == ESHAPE
    assert _rnn(L, rank=96) == EUNSUPPORTED
    assert _rnn(L, d=-1) == EINVAL
    assert _rnn(L, d=60) == EUNSUPPORTED  # the hidden projection reads 8 inputs at a time
    assert _rnn(L, it=0.0) == EINVAL
    assert _rnn(L, Wr=None) == EINVAL
    assert _rnn(L, hidden=None) == EINVAL
    assert _rnn(L, Wr=C.c_void_p((1 << 20) + 8)) == EUNSUPPORTED  # not 16-byte aligned
    assert _rnn(L, hidden=C.c_void_p((1 << 20) + 8)) == EUNSUPPORTED
    assert _rnn(L) == EWORKSPACE
    need = L.dspark_rnn_draft_workspace_size(4, 8, 1024, 256)
    assert _rnn(L, ws_bytes=need - 1) == EWORKSPACE
    assert _rnn(L, hidden=None, d=0, ws=C.c_void_p((1 << 20) + 64), ws_bytes=need) == EWORKSPACE


def test_rnn_draft_workspace_size(L):
    n = L.dspark_rnn_draft_workspace_size(128, 16, 129280, 256)
    # the Markov head's buffers plus the two-term output, two states and the
    # hidden part of the projection for every position
    assert n >= L.dspark_markov_draft_workspace_size(128, 16, 129280, 256) + 128 * 16 * 768 * 4
    assert L.dspark_rnn_draft_workspace_size(128, 16, 129280, 96) == 0


def test_binding_rejects_host_tensors():
    import torch
    with pytest.raises(dspark.DSparkError):
        dspark.dspark_schedule(torch.zeros(2, 3), torch.ones(20, dtype=torch.float64))
