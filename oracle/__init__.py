"""fp64 CPU oracle for DSpark's verification step -- TEST INFRASTRUCTURE ONLY.

Only the test suite, the smoke check and the CPU-baseline leg of the
benchmark import this package.  The GPU library never loads it and shares no
code with it.  ``oracle.c`` holds the arithmetic; this module marshals numpy
arrays into it.  ``guard`` builds parity inputs whose decisions sit at least a
stated distance from any tie.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from typing import Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

_lib = None


def build(force: bool = True) -> str:
    """Compile oracle.c with gcc (fp64, no FMA contraction, OpenMP)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call([
            "gcc", "-O2", "-std=c11", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
            "-Wall", "-Wextra", "-shared", "-fPIC", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        # ORACLE_LIB: a prebuilt copy to load instead (the planted-mistake
        # tests compile mutated copies of oracle.c and run the pins on them)
        override = os.environ.get("ORACLE_LIB")
        if override:
            lib = C.CDLL(override)
        else:
            if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
                build(force=True)
            lib = C.CDLL(_LIB)
        p = C.c_void_p
        i32, i64, f64 = C.c_int, C.c_int64, C.c_double
        lib.oracle_survival.argtypes = [p, i32, i32, p]
        lib.oracle_schedule.argtypes = [p, i32, i32, p, i64, i32, p, p, p, p, p, p]
        lib.oracle_schedule_capacity.argtypes = [p, i32, i32, p, i64, p, p]
        lib.oracle_schedule_topk.argtypes = [p, i32, i32, i64, p, p]
        lib.oracle_verify_attn.argtypes = [p, p, p, p, p, p, i32, p, p, i32, i32, i32, i32, i32,
                                           i32, f64, i32, p, i64, p, p]
        lib.oracle_accept.argtypes = [p, p, p, i32, i64, p, p, i32, i32, i32, f64, p, p, p, p]
        lib.oracle_markov_draft.argtypes = [p, p, i32, i64, p, p, i32, p, p, i32, p, p, f64, i32,
                                            i32, i32, p, p, p, p]
        lib.oracle_rnn_draft.argtypes = [p, p, i32, i64, p, p, p, i32, p, p, i32, p, p, f64, i32,
                                         i32, i32, p, p, p, p]
        lib.oracle_threads.argtypes = []
        lib.oracle_set_threads.argtypes = [i32]
        lib.oracle_set_threads.restype = None
        for f in (lib.oracle_survival, lib.oracle_schedule, lib.oracle_schedule_capacity,
                  lib.oracle_schedule_topk, lib.oracle_verify_attn,
                  lib.oracle_accept, lib.oracle_markov_draft, lib.oracle_rnn_draft,
                  lib.oracle_threads):
            f.restype = C.c_int
        _lib = lib
    return _lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


class OracleError(RuntimeError):
    pass


def _check(rc: int, what: str) -> None:
    if rc != 0:
        raise OracleError(f"{what}: invalid arguments (code {rc})")


def threads() -> int:
    return int(_load().oracle_threads())


def set_threads(n: int) -> None:
    """OpenMP threads for the oracle's later calls (timing baselines)."""
    _load().oracle_set_threads(int(n))


def survival(conf: np.ndarray) -> np.ndarray:
    conf = _c(conf, np.float32)
    R, K = conf.shape
    a = np.empty((R, K), dtype=np.float64)
    _check(_load().oracle_survival(_ptr(conf), R, K, _ptr(a)), "survival")
    return a


def schedule(conf: np.ndarray, sps: np.ndarray, mode: int = 0, trace: bool = False):
    """Algorithm 1.  Returns (len[R] int32, theta_best, n_admitted, min_margin),
    plus the evaluated Theta values when ``trace``."""
    conf = _c(conf, np.float32)
    sps = _c(sps, np.float64)
    R, K = conf.shape
    ln = np.zeros(R, dtype=np.int32)
    tb = C.c_double()
    na = C.c_int32()
    mm = C.c_double()
    tr = np.zeros(R * K + 1, dtype=np.float64) if trace else None
    nt = C.c_int64()
    rc = _load().oracle_schedule(_ptr(conf), R, K, _ptr(sps), sps.size, mode, _ptr(ln),
                                 C.byref(tb), C.byref(na), C.byref(mm), _ptr(tr), C.byref(nt))
    _check(rc, "schedule")
    if trace:
        return ln, tb.value, na.value, mm.value, tr[: nt.value]
    return ln, tb.value, na.value, mm.value


def schedule_capacity(conf_prev: np.ndarray, sps: np.ndarray):
    """Capacity of the asynchronous scheduler: the number of draft tokens the
    no-break search admits on earlier confidences.  Returns (capacity,
    min_margin of its throughput comparisons)."""
    conf_prev = _c(conf_prev, np.float32)
    sps = _c(sps, np.float64)
    R, K = conf_prev.shape
    cap = C.c_int32()
    mm = C.c_double()
    rc = _load().oracle_schedule_capacity(_ptr(conf_prev), R, K, _ptr(sps), sps.size,
                                          C.byref(cap), C.byref(mm))
    _check(rc, "schedule_capacity")
    return cap.value, mm.value


def schedule_topk(conf: np.ndarray, capacity: int):
    """Dynamic top-K admission of the current candidates.  Returns
    (len[R] int32, n_admitted)."""
    conf = _c(conf, np.float32)
    R, K = conf.shape
    ln = np.zeros(R, dtype=np.int32)
    na = C.c_int32()
    rc = _load().oracle_schedule_topk(_ptr(conf), R, K, int(capacity), _ptr(ln), C.byref(na))
    _check(rc, "schedule_topk")
    return ln, na.value


def cu_from_len(ln: np.ndarray) -> np.ndarray:
    cu = np.zeros(len(ln) + 1, dtype=np.int32)
    cu[1:] = np.cumsum(1 + ln.astype(np.int64))
    return cu


def verify_attn(q, k_cache, v_cache, k_strides, v_strides, block_table, kv_len, cu_q,
                Hq: int, Hkv: int, Dqk: int, Dv: int, page_size: int, scale: float,
                dtype: str, rows: Optional[Sequence[Tuple[int, int]]] = None):
    """Returns (out fp64, lse fp64): [total_q, Hq, Dv] / [total_q, Hq], or
    [n, Dv] / [n] for an explicit list of (token, head) rows."""
    dt = 0 if dtype == "f32" else 1
    store = np.float32 if dt == 0 else np.uint16
    q = _c(q, store)
    if not (k_cache.dtype == store and k_cache.flags.c_contiguous):
        raise OracleError("k_cache must be a contiguous array of the input dtype")
    if not (v_cache.dtype == store and v_cache.flags.c_contiguous):
        raise OracleError("v_cache must be a contiguous array of the input dtype")
    bt = _c(block_table, np.int32)
    kv = _c(kv_len, np.int32)
    cu = _c(cu_q, np.int32)
    ks = _c(k_strides, np.int64)
    vs = _c(v_strides, np.int64)
    R = len(kv)
    total = int(cu[-1])
    if rows is None:
        rr = None
        n = total * Hq
        out = np.empty((total, Hq, Dv), dtype=np.float64)
        lse = np.empty((total, Hq), dtype=np.float64)
    else:
        rr = _c(np.asarray(rows, dtype=np.int32).reshape(-1, 2), np.int32)
        n = rr.shape[0]
        out = np.empty((n, Dv), dtype=np.float64)
        lse = np.empty((n,), dtype=np.float64)
    rc = _load().oracle_verify_attn(_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(ks), _ptr(vs),
                                    _ptr(bt), bt.shape[1], _ptr(kv), _ptr(cu), R, Hq, Hkv, Dqk,
                                    Dv, page_size, float(scale), dt, _ptr(rr), n, _ptr(out),
                                    _ptr(lse))
    _check(rc, "verify_attn")
    return out, lse


def accept(draft_tok, draft_p, logits, logit_dtype: str, cu_q, K: int, V: int,
           u=None, inv_temperature: float = 1.0, ld: Optional[int] = None,
           want_rate: bool = False):
    """Returns (accepted_len int32[R], next_tok int32[R], margin f64[R], rate f64[total_q]|None)."""
    dt = 0 if logit_dtype == "f32" else 1
    store = np.float32 if dt == 0 else np.uint16
    logits = _c(logits, store)
    if ld is None:
        ld = logits.shape[-1]
    tok = _c(draft_tok, np.int32)
    dp = None if draft_p is None else _c(draft_p, np.float32)
    uu = None if u is None else _c(u, np.float32)
    cu = _c(cu_q, np.int32)
    R = len(cu) - 1
    acc = np.zeros(R, dtype=np.int32)
    nxt = np.zeros(R, dtype=np.int32)
    mg = np.zeros(R, dtype=np.float64)
    rate = np.zeros(int(cu[-1]), dtype=np.float64) if want_rate else None
    # inv_temperature is an fp32 argument on the GPU side; widen the same value
    it = float(np.float32(inv_temperature))
    rc = _load().oracle_accept(_ptr(tok), _ptr(dp), _ptr(logits), dt, ld, _ptr(uu), _ptr(cu),
                               R, K, V, it, _ptr(acc), _ptr(nxt), _ptr(mg), _ptr(rate))
    _check(rc, "accept")
    return acc, nxt, mg, rate


def markov_draft(anchor, U, u_dtype: str, W1, W2t, w_conf, u, K: int, V: int,
                 hidden=None, sts_temp=None, inv_temperature: float = 1.0,
                 ld: Optional[int] = None, want_p: bool = True):
    """Markov-head draft block.  U: [R*K, >=V] rows (fp32 or bf16 bits), W1 /
    W2t: [V, rank] bf16 bits, hidden: [R, K, d] bf16 bits or None, w_conf:
    [d + rank] fp32, sts_temp: [K] or None, u: [R, K].  Returns (draft_tok
    int32[R, K], draft_p f64[R, K, V] or None, conf f64[R, K], margin f64[R, K]:
    each draw's distance from its bucket's edges in units of the total mass)."""
    dt = 0 if u_dtype == "f32" else 1
    store = np.float32 if dt == 0 else np.uint16
    U = _c(U, store)
    if ld is None:
        ld = U.shape[-1]
    anc = _c(anchor, np.int32)
    R = len(anc)
    W1 = _c(W1, np.uint16)
    W2t = _c(W2t, np.uint16)
    rank = W1.shape[1]
    hid = None if hidden is None else _c(hidden, np.uint16)
    d = 0 if hid is None else hid.shape[-1]
    wc = _c(w_conf, np.float32)
    st = None if sts_temp is None else _c(sts_temp, np.float32)
    uu = _c(u, np.float32)
    tok = np.zeros((R, K), dtype=np.int32)
    dp = np.empty((R, K, V), dtype=np.float64) if want_p else None
    conf = np.zeros((R, K), dtype=np.float64)
    mg = np.zeros((R, K), dtype=np.float64)
    it = float(np.float32(inv_temperature))
    rc = _load().oracle_markov_draft(_ptr(anc), _ptr(U), dt, ld, _ptr(W1), _ptr(W2t), rank,
                                     _ptr(hid), _ptr(wc), d, _ptr(st), _ptr(uu), it, R, K, V,
                                     _ptr(tok), _ptr(dp), _ptr(conf), _ptr(mg))
    _check(rc, "markov_draft")
    return tok, dp, conf, mg


def rnn_draft(anchor, U, u_dtype: str, W1, W2t, Wrnn, w_conf, u, K: int, V: int,
              hidden=None, sts_temp=None, inv_temperature: float = 1.0,
              ld: Optional[int] = None, want_p: bool = True):
    """RNN-head draft block.  As markov_draft, plus Wrnn: [3 rank, 2 rank + d]
    bf16 bits (gate, candidate and output rows; columns [s; e; h]).  Returns
    (draft_tok int32[R, K], draft_p f64[R, K, V] or None, conf f64[R, K],
    margin f64[R, K])."""
    dt = 0 if u_dtype == "f32" else 1
    store = np.float32 if dt == 0 else np.uint16
    U = _c(U, store)
    if ld is None:
        ld = U.shape[-1]
    anc = _c(anchor, np.int32)
    R = len(anc)
    W1 = _c(W1, np.uint16)
    W2t = _c(W2t, np.uint16)
    Wr = _c(Wrnn, np.uint16)
    rank = W1.shape[1]
    hid = None if hidden is None else _c(hidden, np.uint16)
    d = 0 if hid is None else hid.shape[-1]
    if Wr.shape != (3 * rank, 2 * rank + d):
        raise ValueError(f"Wrnn must be [{3 * rank}, {2 * rank + d}], got {Wr.shape}")
    wc = _c(w_conf, np.float32)
    st = None if sts_temp is None else _c(sts_temp, np.float32)
    uu = _c(u, np.float32)
    tok = np.zeros((R, K), dtype=np.int32)
    dp = np.empty((R, K, V), dtype=np.float64) if want_p else None
    conf = np.zeros((R, K), dtype=np.float64)
    mg = np.zeros((R, K), dtype=np.float64)
    it = float(np.float32(inv_temperature))
    rc = _load().oracle_rnn_draft(_ptr(anc), _ptr(U), dt, ld, _ptr(W1), _ptr(W2t), _ptr(Wr), rank,
                                  _ptr(hid), _ptr(wc), d, _ptr(st), _ptr(uu), it, R, K, V,
                                  _ptr(tok), _ptr(dp), _ptr(conf), _ptr(mg))
    _check(rc, "rnn_draft")
    return tok, dp, conf, mg
