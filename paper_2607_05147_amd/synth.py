"""Seeded synthetic workloads for the DSpark verification step.

This module only *constructs inputs*: confidences, the engine throughput
table, paged KV caches, verify queries, target logits, draft tokens, draft
distributions and uniforms.  It holds none of the verification step's own
arithmetic (no survival products, no scheduling, no attention, no acceptance
test), so it can feed both the GPU path and the CPU reference.

Every array is a pure function of ``(workload, seed, stream, key...)``: each
piece draws from its own counter-keyed ``numpy`` generator
(``SeedSequence([seed, stream, *key])``), so a row, a page or a request can be
generated on its own and comes out identical to the same piece of a full
generation.  Large arrays are generated in fixed-size chunks on a thread pool.

The shapes and distributions follow the five workloads the verification step
is evaluated on: a tiny fp32 case, a mid-sized bf16 case, a 128-request
serving case, a 512-request high-concurrency case and a long-context
absorbed-latent (MLA-style) case.  Where a workload description leaves a
parameter open, the reading used is stated on the field.
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

# Sub-stream identifiers.  Fixed forever: changing one changes every input.
_STREAM = {
    "conf": 1,
    "kv_len": 2,
    "pages": 3,
    "q": 4,
    "k": 5,
    "v": 6,
    "logits": 7,
    "draft_tok": 8,
    "draft_p": 9,
    "uniform": 10,
    "mk_anchor": 11,
    "mk_base": 12,
    "mk_w1": 13,
    "mk_w2": 14,
    "mk_hidden": 15,
    "mk_wconf": 16,
    "mk_uniform": 17,
    "rnn_w": 18,
    "conf_prev": 19,
}

_KV_CHUNK_PAGES = 64  # pages per generator chunk of the KV pool


def _rng(seed: int, stream: str, *key: int) -> np.random.Generator:
    ss = np.random.SeedSequence([int(seed), _STREAM[stream]] + [int(k) for k in key])
    return np.random.Generator(np.random.PCG64(ss))


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bfloat16 (round to nearest even); returns uint16 bit patterns."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    out = ((u + (((u >> 16) & np.uint32(1)) + np.uint32(0x7FFF))) >> 16).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = np.uint16(0x7FC0)
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to fp32."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


BF16_NAN = np.uint16(0x7FC0)


@dataclass(frozen=True)
class Workload:
    """Shape and distribution recipe of one verification-step workload."""

    name: str
    R: int  # active requests
    Hq: int  # query heads
    Hkv: int  # KV heads (1 shared latent head for the MLA-style case)
    Dqk: int  # query/key head dim
    Dv: int  # value head dim
    page: int  # tokens per KV page
    dtype: str  # "f32" or "bf16" for Q/K/V/out
    kv_dist: Tuple  # ("uniform", lo, hi) or ("lognormal", median, sigma, lo, hi)
    K: int  # draft block length (the paper's gamma)
    conf_beta: Tuple[float, float]  # Beta(a, b) per-position confidence
    conf_decay: float  # per-position multiplicative decay (1.0 = none)
    knee: int  # step_time(T) = 1 + slope * max(0, T - knee)
    slope: float
    V: int  # vocabulary
    logit_dtype: str  # "f32" or "bf16"
    logit_scale: float  # target logits ~ logit_scale * N(0, 1)
    greedy: bool  # greedy match (True) or stochastic rejection sampling
    mla: bool = False  # V aliases the first Dv dims of the shared latent K row
    pd_temperature: float = 0.8  # draft distribution: target softmax at this temperature ...
    pd_mix: float = 0.8  # ... mixed pd_mix / (1 - pd_mix) with ...
    pd_dirichlet: float = 0.1  # ... a Dirichlet(pd_dirichlet) perturbation

    @property
    def group(self) -> int:
        return self.Hq // self.Hkv

    @property
    def max_q(self) -> int:
        return self.K + 1

    @property
    def sps_len(self) -> int:
        return self.R * (self.K + 1) + 1

    @property
    def scale(self) -> float:
        return float(np.float32(1.0 / math.sqrt(self.Dqk)))

    @property
    def kv_elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    @property
    def logit_elem_bytes(self) -> int:
        return 4 if self.logit_dtype == "f32" else 2


# The five workloads.  Readings where the description is silent:
#  * step_time knee/slope for mid (64, 1/256), serving (256, 1/1024),
#    high-concurrency (512, 1/1024), latent (64, 1/128);
#  * log-normal contexts use sigma 0.5 in log space, then clip and round;
#  * Q/K/V ~ N(0,1); logits 4*N(0,1) where unstated; mid uses fp32 logits;
#  * draft distributions for the stochastic cases follow the mid recipe;
#  * greedy draft tokens equal the target argmax with probability equal to
#    their confidence, otherwise uniform over the vocabulary.
WORKLOADS: Dict[str, Workload] = {
    "tiny": Workload(
        name="tiny", R=4, Hq=8, Hkv=2, Dqk=64, Dv=64, page=16, dtype="f32",
        kv_dist=("uniform", 32, 128), K=8, conf_beta=(4.0, 1.0), conf_decay=1.0,
        knee=16, slope=0.01, V=1024, logit_dtype="f32", logit_scale=3.0, greedy=True),
    "mid": Workload(
        name="mid", R=32, Hq=32, Hkv=8, Dqk=128, Dv=128, page=64, dtype="bf16",
        kv_dist=("uniform", 1024, 4096), K=16, conf_beta=(3.0, 1.0), conf_decay=0.97,
        knee=64, slope=1.0 / 256, V=32768, logit_dtype="f32", logit_scale=4.0, greedy=False),
    "serving": Workload(
        name="serving", R=128, Hq=64, Hkv=8, Dqk=128, Dv=128, page=64, dtype="bf16",
        kv_dist=("lognormal", 4096, 0.5, 2048, 16384), K=16, conf_beta=(4.0, 1.5),
        conf_decay=1.0, knee=256, slope=1.0 / 1024, V=129280, logit_dtype="bf16",
        logit_scale=4.0, greedy=False),
    "highconc": Workload(
        name="highconc", R=512, Hq=32, Hkv=4, Dqk=128, Dv=128, page=64, dtype="bf16",
        kv_dist=("lognormal", 2048, 0.5, 512, 8192), K=8, conf_beta=(2.0, 1.0),
        conf_decay=1.0, knee=512, slope=1.0 / 1024, V=129280, logit_dtype="bf16",
        logit_scale=4.0, greedy=True),
    "mla": Workload(
        name="mla", R=16, Hq=128, Hkv=1, Dqk=576, Dv=512, page=64, dtype="bf16",
        kv_dist=("uniform", 32768, 131072), K=16, conf_beta=(5.0, 1.0), conf_decay=1.0,
        knee=64, slope=1.0 / 128, V=129280, logit_dtype="bf16", logit_scale=4.0,
        greedy=False, mla=True),
}

WORKLOAD_ORDER = ["tiny", "mid", "serving", "highconc", "mla"]


def scaled(w: Workload, **over) -> Workload:
    """A copy of ``w`` with some fields replaced (small parity cases)."""
    d = dict(w.__dict__)
    d.update(over)
    return Workload(**d)


# --------------------------------------------------------------------------
# scheduling inputs
# --------------------------------------------------------------------------

def confidences(w: Workload, seed: int, attempt: int = 0) -> np.ndarray:
    """Per-position draft confidences c[r, j], fp32 [R, K]."""
    g = _rng(seed, "conf", attempt)
    c = g.beta(w.conf_beta[0], w.conf_beta[1], size=(w.R, w.K))
    if w.conf_decay != 1.0:
        c = c * (w.conf_decay ** np.arange(w.K, dtype=np.float64))[None, :]
    return np.ascontiguousarray(c.astype(np.float32))


def previous_confidences(w: Workload, seed: int, attempt: int = 0) -> np.ndarray:
    """Confidences of an earlier step for the same requests (same law as
    ``confidences``, an independent sub-stream): the input from which the
    asynchronous scheduler decides its capacity."""
    g = _rng(seed, "conf_prev", attempt)
    c = g.beta(w.conf_beta[0], w.conf_beta[1], size=(w.R, w.K))
    if w.conf_decay != 1.0:
        c = c * (w.conf_decay ** np.arange(w.K, dtype=np.float64))[None, :]
    return np.ascontiguousarray(c.astype(np.float32))


def sps_table(w: Workload) -> np.ndarray:
    """Engine steps/s versus total verify tokens T, fp64 [R*(K+1)+1].

    The workload states a step-time profile; the table holds its reciprocal."""
    T = np.arange(w.sps_len, dtype=np.float64)
    step_time = 1.0 + w.slope * np.maximum(0.0, T - w.knee)
    return 1.0 / step_time


# --------------------------------------------------------------------------
# KV cache
# --------------------------------------------------------------------------

def kv_lengths(w: Workload, seed: int) -> np.ndarray:
    g = _rng(seed, "kv_len")
    d = w.kv_dist
    if d[0] == "uniform":
        kv = g.integers(d[1], d[2] + 1, size=w.R)
    elif d[0] == "lognormal":
        _, med, sig, lo, hi = d
        x = np.exp(g.normal(math.log(med), sig, size=w.R))
        kv = np.rint(np.clip(x, lo, hi))
    else:  # pragma: no cover
        raise ValueError(d)
    return kv.astype(np.int32)


@dataclass
class PagedKV:
    """A paged KV pool and the per-request block table.

    ``k``/``v`` have shape [pool_pages, Hkv, page, D] (fp32, or uint16 bf16
    bits).  For the latent workload ``v`` is ``k`` itself and only its first
    ``Dv`` dims are values.  The last pool page is a poison page (NaN) that
    every unused block-table slot points at; slots of a request's last page
    past its context are also NaN."""

    kv_len: np.ndarray
    block_table: np.ndarray  # int32 [R, max_pages]
    n_pages: int  # pages in use (excludes the poison page)
    k: np.ndarray
    v: np.ndarray
    k_strides: Tuple[int, int, int]  # element strides (page, head, token)
    v_strides: Tuple[int, int, int]

    @property
    def max_pages(self) -> int:
        return int(self.block_table.shape[1])

    @property
    def pool_pages(self) -> int:
        return int(self.k.shape[0])


def _normal_fill(w: Workload, seed: int, stream: str, out: np.ndarray, chunk_rows: int) -> None:
    """Fill ``out`` (first axis chunked) with N(0,1) in the workload dtype."""
    n = out.shape[0]
    inner = out.shape[1:]

    def job(ci: int) -> None:
        lo = ci * chunk_rows
        hi = min(n, lo + chunk_rows)
        x = _rng(seed, stream, ci).standard_normal((hi - lo,) + inner, dtype=np.float32)
        out[lo:hi] = x if w.dtype == "f32" else f32_to_bf16_bits(x)

    nchunks = (n + chunk_rows - 1) // chunk_rows
    with ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(job, range(nchunks)))


def paged_kv(w: Workload, seed: int, kv_len: Optional[np.ndarray] = None,
             poison: bool = True) -> PagedKV:
    if kv_len is None:
        kv_len = kv_lengths(w, seed)
    P = w.page
    npg = (kv_len.astype(np.int64) + P - 1) // P
    total = int(npg.sum())
    max_pages = int(npg.max())
    pool = total + 1  # + poison page
    perm = _rng(seed, "pages").permutation(total).astype(np.int32)
    bt = np.full((w.R, max_pages), total, dtype=np.int32)
    off = 0
    for r in range(w.R):
        bt[r, : npg[r]] = perm[off: off + npg[r]]
        off += int(npg[r])
    store = np.float32 if w.dtype == "f32" else np.uint16
    nan = np.float32(np.nan) if w.dtype == "f32" else BF16_NAN
    k = np.empty((pool, w.Hkv, P, w.Dqk), dtype=store)
    _normal_fill(w, seed, "k", k[:total], _KV_CHUNK_PAGES)
    k[total] = nan
    if w.mla:
        v = k
    else:
        v = np.empty((pool, w.Hkv, P, w.Dv), dtype=store)
        _normal_fill(w, seed, "v", v[:total], _KV_CHUNK_PAGES)
        v[total] = nan
    if poison:
        for r in range(w.R):
            tail = int(kv_len[r]) - (int(npg[r]) - 1) * P
            if tail < P:
                pg = bt[r, npg[r] - 1]
                k[pg, :, tail:, :] = nan
                if not w.mla:
                    v[pg, :, tail:, :] = nan
    ks = (w.Hkv * P * w.Dqk, P * w.Dqk, w.Dqk)
    vs = ks if w.mla else (w.Hkv * P * w.Dv, P * w.Dv, w.Dv)
    return PagedKV(kv_len=kv_len, block_table=bt, n_pages=total, k=k, v=v,
                   k_strides=ks, v_strides=vs)


# --------------------------------------------------------------------------
# verify queries and target logits: one row per (request r, verify slot t)
# --------------------------------------------------------------------------

def _rows_parallel(fn, keys: Sequence[Tuple[int, int]], out: np.ndarray) -> None:
    def job(i: int) -> None:
        out[i] = fn(*keys[i])

    if len(keys) == 0:
        return
    with ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(job, range(len(keys))))


def query_rows(w: Workload, seed: int, keys: Sequence[Tuple[int, int]]) -> np.ndarray:
    """Q rows [n, Hq, Dqk] for the (r, t) keys, in the given order."""
    store = np.float32 if w.dtype == "f32" else np.uint16
    out = np.empty((len(keys), w.Hq, w.Dqk), dtype=store)

    def one(r: int, t: int) -> np.ndarray:
        x = _rng(seed, "q", r, t).standard_normal((w.Hq, w.Dqk), dtype=np.float32)
        return x if w.dtype == "f32" else f32_to_bf16_bits(x)

    _rows_parallel(one, keys, out)
    return out


def _logit_row_f32(w: Workload, seed: int, r: int, t: int) -> np.ndarray:
    """Target logits of slot t of request r as the stored dtype, widened to fp32."""
    x = _rng(seed, "logits", r, t).standard_normal(w.V, dtype=np.float32) * np.float32(w.logit_scale)
    if w.logit_dtype == "bf16":
        x = bf16_bits_to_f32(f32_to_bf16_bits(x))
    return x


def logit_rows(w: Workload, seed: int, keys: Sequence[Tuple[int, int]]) -> np.ndarray:
    """Target logit rows [n, V] (fp32, or uint16 bf16 bits) for the (r, t) keys."""
    store = np.float32 if w.logit_dtype == "f32" else np.uint16
    out = np.empty((len(keys), w.V), dtype=store)

    def one(r: int, t: int) -> np.ndarray:
        x = _logit_row_f32(w, seed, r, t)
        return x if w.logit_dtype == "f32" else f32_to_bf16_bits(x)

    _rows_parallel(one, keys, out)
    return out


def flat_keys(q_len: np.ndarray) -> List[Tuple[int, int]]:
    """(r, t) keys in flattened verify order for per-request query counts."""
    return [(r, t) for r in range(len(q_len)) for t in range(int(q_len[r]))]


# --------------------------------------------------------------------------
# drafts
# --------------------------------------------------------------------------

@dataclass
class Drafts:
    draft_tok: np.ndarray  # int32 [R, K]; draft_tok[r, t] is the draft for slot t+1
    draft_p: Optional[np.ndarray]  # fp32 [R, K, V] draft distribution (stochastic only)
    u: Optional[np.ndarray]  # fp32 [R, K+1] uniforms (stochastic only)


def _draft_dist(w: Workload, seed: int, r: int, t: int) -> np.ndarray:
    """Draft distribution for draft slot t+1 of request r (fp32 [V])."""
    z = _logit_row_f32(w, seed, r, t).astype(np.float64)
    y = z / w.pd_temperature
    y = np.exp(y - y.max())
    tgt = y / y.sum()
    gam = _rng(seed, "draft_p", r, t).standard_gamma(w.pd_dirichlet, size=w.V)
    s = gam.sum()
    dirich = gam / s if s > 0 else np.full(w.V, 1.0 / w.V)
    return (w.pd_mix * tgt + (1.0 - w.pd_mix) * dirich).astype(np.float32)


def _sample_index(p: np.ndarray, x: float) -> int:
    c = np.cumsum(p.astype(np.float64))
    i = int(np.searchsorted(c, x * c[-1], side="right"))
    return min(i, len(p) - 1)


def uniforms(w: Workload, seed: int, r: int, attempt: int = 0) -> np.ndarray:
    """Uniforms u[r, 0..K] in [0, 1) for request r (redraw index ``attempt``)."""
    return _rng(seed, "uniform", r, attempt).random(w.K + 1, dtype=np.float32)


def drafts(w: Workload, seed: int, conf: np.ndarray,
           needed: Optional[np.ndarray] = None,
           u_attempts: Optional[np.ndarray] = None) -> Drafts:
    """Draft tokens (and, when stochastic, draft distributions and uniforms).

    ``needed`` (bool [R, K]) marks draft slots whose token/distribution is
    consumed; other slots get token 0 and a NaN draft row, which the
    verification step never reads.  ``u_attempts`` (int [R]) picks the redraw
    index of each request's uniforms."""
    R, K, V = w.R, w.K, w.V
    if needed is None:
        needed = np.ones((R, K), dtype=bool)
    keys = [(r, t) for r in range(R) for t in range(K) if needed[r, t]]
    tok = np.zeros((R, K), dtype=np.int32)
    if w.greedy:
        def one(r: int, t: int) -> int:
            g = _rng(seed, "draft_tok", r, t)
            hit, alt = g.random(), int(g.integers(0, V))
            if hit < float(conf[r, t]):
                return int(np.argmax(_logit_row_f32(w, seed, r, t)))
            return alt

        vals = np.zeros(len(keys), dtype=np.int64)
        _rows_parallel(one, keys, vals)
        for (r, t), x in zip(keys, vals):
            tok[r, t] = x
        return Drafts(draft_tok=tok, draft_p=None, u=None)

    dp = np.empty((R, K, V), dtype=np.float32)
    dp[~needed] = np.nan

    def one_row(i: int) -> None:
        r, t = keys[i]
        p = _draft_dist(w, seed, r, t)
        dp[r, t] = p
        tok[r, t] = _sample_index(p, _rng(seed, "draft_tok", r, t).random())

    if keys:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(one_row, range(len(keys))))
    if u_attempts is None:
        u_attempts = np.zeros(R, dtype=np.int64)
    u = np.stack([uniforms(w, seed, r, int(u_attempts[r])) for r in range(R)])
    return Drafts(draft_tok=tok, draft_p=dp, u=np.ascontiguousarray(u))


# --------------------------------------------------------------------------
# Markov-head draft block inputs (the drafter's sequential stage)
# --------------------------------------------------------------------------

MARKOV_RANK = 256  # the paper's default low rank of the transition bias
MARKOV_HIDDEN = 4096  # width of the backbone state the confidence head reads


@dataclass
class MarkovInputs:
    anchor: np.ndarray  # int32 [R] x_0
    base: np.ndarray  # [R * K, V] base logits U_k (fp32, or uint16 bf16 bits)
    W1: np.ndarray  # uint16 bf16 bits [V, rank]: embedding rows
    W2t: np.ndarray  # uint16 bf16 bits [V, rank]: row v holds W2[:, v]
    hidden: np.ndarray  # uint16 bf16 bits [R, K, d]
    w_conf: np.ndarray  # fp32 [d + rank]
    sts_temp: np.ndarray  # fp32 [K] per-position temperatures
    u: np.ndarray  # fp32 [R, K] uniforms of the draws
    Wrnn: Optional[np.ndarray] = None  # uint16 bf16 bits [3 rank, 2 rank + d] (RNN head only)


def markov_uniforms(seed: int, r: int, K: int, attempt: int = 0) -> np.ndarray:
    """Uniforms of request r's K draws (redraw index ``attempt``)."""
    return _rng(seed, "mk_uniform", r, attempt).random(K, dtype=np.float32)


def rnn_weights(seed: int, rank: int, d: int) -> np.ndarray:
    """Seeded RNN-head projection [3 rank, 2 rank + d] (bf16 bits): rows are
    gate, candidate and output; columns [s; e; h].  Column blocks ~ N(0, 1/rank),
    N(0, 1) and N(0, 1/d) for the state, the unit-norm embedding and the
    N(0, 1) hidden state, so each pre-activation is about N(0, 2); the output
    rows are scaled by 1/sqrt(rank), which keeps tanh near linear and the bias
    W2^T o about N(0, 2), like the Markov head's."""
    g = _rng(seed, "rnn_w").standard_normal((3 * rank, 2 * rank + d), dtype=np.float32)
    col = np.concatenate([np.full(rank, 1.0 / math.sqrt(rank)), np.ones(rank),
                          np.full(d, 1.0 / math.sqrt(max(d, 1)))]).astype(np.float32)
    row = np.concatenate([np.ones(2 * rank), np.full(rank, 1.0 / math.sqrt(rank))]).astype(np.float32)
    return f32_to_bf16_bits(g * col[None, :] * row[:, None])


def markov_inputs(w: Workload, seed: int, rank: int = MARKOV_RANK, d: int = MARKOV_HIDDEN,
                  u_attempts: Optional[np.ndarray] = None, rnn: bool = False) -> MarkovInputs:
    """Seeded synthetic inputs of the Markov-head draft block for workload w:
    base logits logit_scale * N(0, 1) in the logit dtype; W1 ~ N(0, 1/rank)
    (unit-norm embeddings) and W2 ~ N(0, 1), so the transition bias is about
    N(0, 1); hidden ~ N(0, 1); w_conf ~ N(0, 1/(d + rank)); temperatures
    1 + 0.05 k; anchors uniform over the vocabulary."""
    R, K, V = w.R, w.K, w.V
    anchor = _rng(seed, "mk_anchor").integers(0, V, R).astype(np.int32)
    store = np.float32 if w.logit_dtype == "f32" else np.uint16
    base = np.empty((R * K, V), dtype=store)

    def base_row(i: int) -> None:
        x = _rng(seed, "mk_base", i).standard_normal(V, dtype=np.float32) * np.float32(w.logit_scale)
        base[i] = x if w.logit_dtype == "f32" else f32_to_bf16_bits(x)

    with ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(base_row, range(R * K)))
    g1 = _rng(seed, "mk_w1").standard_normal((V, rank), dtype=np.float32) * np.float32(1.0 / math.sqrt(rank))
    g2 = _rng(seed, "mk_w2").standard_normal((V, rank), dtype=np.float32)
    hidden = f32_to_bf16_bits(_rng(seed, "mk_hidden").standard_normal((R, K, d), dtype=np.float32))
    w_conf = (_rng(seed, "mk_wconf").standard_normal(d + rank) / math.sqrt(d + rank)).astype(np.float32)
    sts = (1.0 + 0.05 * np.arange(1, K + 1)).astype(np.float32)
    if u_attempts is None:
        u_attempts = np.zeros(R, dtype=np.int64)
    u = np.stack([markov_uniforms(seed, r, K, int(u_attempts[r])) for r in range(R)])
    return MarkovInputs(anchor=anchor, base=base, W1=f32_to_bf16_bits(g1), W2t=f32_to_bf16_bits(g2),
                        hidden=hidden, w_conf=w_conf, sts_temp=sts, u=np.ascontiguousarray(u),
                        Wrnn=rnn_weights(seed, rank, d) if rnn else None)
