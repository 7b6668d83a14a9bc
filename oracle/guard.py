"""Guard-banded parity cases -- TEST INFRASTRUCTURE ONLY.

Builds one verification step's inputs from the seeded generator and runs the
oracle on them, redrawing inputs until every discrete decision the oracle
takes sits at least a stated distance from a tie:

* scheduler: every throughput comparison made satisfies
  |Theta - Theta_best| >= SCHED_GUARD * Theta_best.  The GPU sums the
  survival probabilities in a different order than the oracle's sequential
  loop; for at most 8192 positive fp64 terms each order's relative error is
  below 8192 * 2^-53 (about 9.1e-13), so the two differ by less than 2e-12,
  and recomputing tau in the GPU's order at 8192 candidates measures 3.5e-15
  (tests/test_oracle_schedule.py).  A 1e-9 band makes equal decisions
  certain.  (A
  1e-4 band is unreachable here: the greedy stop happens exactly where the
  marginal throughput gain crosses zero, typically 1e-6..1e-9 from a tie.)
* acceptance test: |u - min(1, p_t(x) / p_d(x))| >= ACCEPT_GUARD;
* final draw: u * mass at least ACCEPT_GUARD (in units of the total mass)
  from both edges of the chosen token's bucket.

Redraws use fresh sub-streams of the generator (confidences as a whole,
uniforms per request), at most ``max_tries`` times; requests still inside the
band are listed in ``unguarded`` and left out of exact comparisons.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

import oracle
from paper_2607_05147_amd import synth

SCHED_GUARD = 1e-9
ACCEPT_GUARD = 1e-4


@dataclass
class StepCase:
    w: synth.Workload
    seed: int
    conf: np.ndarray
    sps: np.ndarray
    len: np.ndarray  # oracle schedule
    cu_q: np.ndarray
    sched_margin: float
    sched_guarded: bool
    kv: Optional[synth.PagedKV] = None
    q: Optional[np.ndarray] = None  # [total_q, Hq, Dqk]
    logits: Optional[np.ndarray] = None  # [total_q, V]
    drafts: Optional[synth.Drafts] = None
    accepted_len: Optional[np.ndarray] = None  # oracle acceptance
    next_tok: Optional[np.ndarray] = None
    accept_margin: Optional[np.ndarray] = None
    unguarded: List[int] = field(default_factory=list)

    @property
    def total_q(self) -> int:
        return int(self.cu_q[-1])

    @property
    def q_len(self) -> np.ndarray:
        return np.diff(self.cu_q)


def schedule_case(w: synth.Workload, seed: int, mode: int = 0, max_tries: int = 64,
                  guard: float = SCHED_GUARD) -> StepCase:
    sps = synth.sps_table(w)
    best = None
    for attempt in range(max_tries):
        conf = synth.confidences(w, seed, attempt)
        ln, _, _, mm = oracle.schedule(conf, sps, mode)
        if best is None or mm > best[3]:
            best = (conf, ln, attempt, mm)
        if mm >= guard:
            break
    conf, ln, _, mm = best
    return StepCase(w=w, seed=seed, conf=conf, sps=sps, len=ln, cu_q=oracle.cu_from_len(ln),
                    sched_margin=mm, sched_guarded=mm >= guard)


@dataclass
class CapacityCase:
    conf_prev: np.ndarray  # earlier step's confidences (capacity decided on them)
    conf: np.ndarray  # current confidences (ranked)
    sps: np.ndarray
    capacity: int  # oracle capacity
    len: np.ndarray  # oracle top-K lengths
    cu_q: np.ndarray
    margin: float  # min margin of the capacity search's throughput comparisons
    guarded: bool


def capacity_case(w: synth.Workload, seed: int, max_tries: int = 64,
                  guard: float = SCHED_GUARD) -> CapacityCase:
    """Asynchronous scheduler inputs: the earlier confidences are redrawn until
    the no-break search's comparisons are all outside the guard band; the
    top-K admission itself takes no floating-point decision that can tie
    (equal survival values are ordered by index)."""
    sps = synth.sps_table(w)
    best = None
    for attempt in range(max_tries):
        prev = synth.previous_confidences(w, seed, attempt)
        cap, mm = oracle.schedule_capacity(prev, sps)
        if best is None or mm > best[2]:
            best = (prev, cap, mm)
        if mm >= guard:
            break
    prev, cap, mm = best
    conf = synth.confidences(w, seed)
    ln, _ = oracle.schedule_topk(conf, cap)
    return CapacityCase(conf_prev=prev, conf=conf, sps=sps, capacity=cap, len=ln,
                        cu_q=oracle.cu_from_len(ln), margin=mm, guarded=mm >= guard)


def _accept_subset(case: StepCase, reqs: List[int], u: np.ndarray):
    """Oracle acceptance for a subset of requests (rows gathered)."""
    w = case.w
    cu = case.cu_q
    rows = np.concatenate([np.arange(cu[r], cu[r + 1]) for r in reqs])
    sub_cu = oracle.cu_from_len(case.len[reqs])
    dr = case.drafts
    acc, nxt, mg, _ = oracle.accept(
        dr.draft_tok[reqs], None if dr.draft_p is None else dr.draft_p[reqs],
        case.logits[rows], w.logit_dtype, sub_cu, w.K, w.V,
        u=None if u is None else u[reqs])
    return acc, nxt, mg


def build_case(w: synth.Workload, seed: int, mode: int = 0, with_kv: bool = True,
               with_accept: bool = True, max_tries: int = 64,
               guard: float = ACCEPT_GUARD) -> StepCase:
    """Schedule (guarded), then KV/queries and logits/drafts (guarded)."""
    case = schedule_case(w, seed, mode=mode, max_tries=max_tries)
    keys = synth.flat_keys(case.q_len)
    if with_kv:
        case.kv = synth.paged_kv(w, seed)
        case.q = synth.query_rows(w, seed, keys)
    if not with_accept:
        return case
    case.logits = synth.logit_rows(w, seed, keys)
    needed = np.arange(w.K)[None, :] < case.len[:, None]
    attempts = np.zeros(w.R, dtype=np.int64)
    case.drafts = synth.drafts(w, seed, case.conf, needed=needed, u_attempts=attempts)
    R = w.R
    acc = np.zeros(R, np.int32)
    nxt = np.zeros(R, np.int32)
    mg = np.full(R, np.inf)
    todo = list(range(R))
    u = case.drafts.u
    for _ in range(max_tries):
        a, n, m = _accept_subset(case, todo, u)
        acc[todo], nxt[todo], mg[todo] = a, n, m
        todo = [r for r in todo if mg[r] < guard]
        if not todo or w.greedy:
            break
        for r in todo:
            attempts[r] += 1
            u[r] = synth.uniforms(w, seed, r, int(attempts[r]))
    case.accepted_len, case.next_tok, case.accept_margin = acc, nxt, mg
    case.unguarded = [] if w.greedy else [r for r in range(R) if mg[r] < guard]
    return case


# --------------------------------------------------------------------------
# Markov-head draft block
# --------------------------------------------------------------------------

@dataclass
class DraftCase:
    inp: "synth.MarkovInputs"
    tok: np.ndarray  # oracle draft tokens [n, K] of the requests in ``reqs``
    p: Optional[np.ndarray]  # oracle draft distributions [n, K, V] (fp64) or None
    conf: np.ndarray  # oracle confidences [n, K]
    margin: np.ndarray  # per-draw margins [n, K]
    reqs: List[int]
    unguarded: List[int] = field(default_factory=list)


def draft_case(w: synth.Workload, seed: int, rank: int, d: int, reqs: Optional[List[int]] = None,
               inv_temperature: float = 1.0, want_p: bool = True, max_tries: int = 64,
               head: str = "markov") -> DraftCase:
    """Inputs of the draft block and the oracle's outputs for ``reqs`` (all by
    default), with each request's uniforms redrawn draw by draw, left to right,
    until every draw is at least ACCEPT_GUARD (units of the total mass) from
    its bucket's edges.  A redraw of draw k takes element k of the request's
    next uniform sub-stream and changes every later draw, which is checked
    again."""
    inp = synth.markov_inputs(w, seed, rank=rank, d=d, rnn=head == "rnn")
    R, K, V = w.R, w.K, w.V
    reqs = list(range(R)) if reqs is None else list(reqs)
    tries = {r: np.zeros(K, dtype=np.int64) for r in reqs}
    sub = np.array(reqs, dtype=np.int64)
    unguarded: List[int] = []

    def run(want):
        base = inp.base.reshape(R, K, -1)[sub].reshape(len(sub) * K, -1)
        hid = None if d == 0 else inp.hidden[sub]
        if head == "rnn":
            return oracle.rnn_draft(inp.anchor[sub], base, w.logit_dtype, inp.W1, inp.W2t,
                                    inp.Wrnn, inp.w_conf, inp.u[sub], K, V, hidden=hid,
                                    sts_temp=inp.sts_temp, inv_temperature=inv_temperature,
                                    want_p=want)
        return oracle.markov_draft(inp.anchor[sub], base, w.logit_dtype, inp.W1, inp.W2t,
                                   inp.w_conf, inp.u[sub], K, V, hidden=hid,
                                   sts_temp=inp.sts_temp, inv_temperature=inv_temperature,
                                   want_p=want)

    for _ in range(max_tries * K):
        tok, _, _, mg = run(False)
        bad = False
        for i, r in enumerate(reqs):
            ks = np.nonzero(mg[i] < ACCEPT_GUARD)[0]
            if len(ks) == 0 or r in unguarded:
                continue
            k = int(ks[0])
            tries[r][k] += 1
            if tries[r][k] > max_tries:
                unguarded.append(r)
                continue
            inp.u[r, k] = synth.markov_uniforms(seed, r, K, int(tries[r][k]))[k]
            bad = True
        if not bad:
            break
    tok, p, conf, mg = run(want_p)
    return DraftCase(inp=inp, tok=tok, p=p, conf=conf, margin=mg, reqs=reqs, unguarded=unguarded)
