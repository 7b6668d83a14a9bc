"""Python binding of the C ABI in include/dspark.h (argument marshalling only).

Every function takes torch tensors that live on a ROCm device, checks their
dtype/shape/contiguity, passes raw pointers to ``libdspark.so`` and raises
``DSparkError`` with the library's message when a call fails.  Outputs that are
not supplied are allocated with torch (device memory plumbing); all
computation happens in the library's HIP kernels, enqueued on the current
torch stream unless ``stream`` is given.  There is no fallback: without the
built library every call raises.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional, Sequence, Tuple

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdspark.so")

DSPARK_F32 = 0
DSPARK_BF16 = 1
STATUS = {0: "OK", 1: "EINVAL", 2: "ESHAPE", 3: "EDTYPE", 4: "EUNSUPPORTED", 5: "EWORKSPACE",
          6: "EHIP"}


class DSparkError(RuntimeError):
    def __init__(self, msg: str, status: int = -1):
        super().__init__(msg)
        self.status = status


_lib = None


def lib():
    """The loaded C library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        # DSPARK_LIB: another build of the same library to load instead (the
        # host-sanitizer test builds an instrumented copy)
        path = os.environ.get("DSPARK_LIB") or LIB_PATH
        if not os.path.exists(path):
            raise DSparkError(f"{path} is missing: build it with "
                              "`python -m paper_2607_05147_amd.build` (no fallback path exists)")
        L = C.CDLL(path)
        p, i32, i64, sz, f32 = C.c_void_p, C.c_int, C.c_int64, C.c_size_t, C.c_float
        L.dspark_abi_version.restype = i32
        L.dspark_abi_version.argtypes = []
        L.dspark_last_error.restype = C.c_char_p
        L.dspark_last_error.argtypes = []
        L.dspark_schedule_workspace_size.restype = sz
        L.dspark_schedule_workspace_size.argtypes = [i32, i32]
        L.dspark_schedule.restype = i32
        L.dspark_schedule.argtypes = [p, i32, i32, p, i64, i32, p, p, p, p, sz, p]
        L.dspark_schedule_noalloc.restype = i32
        L.dspark_schedule_noalloc.argtypes = [p, i32, i32, p, i64, i32, p, p, p, p]
        L.dspark_schedule_capacity.restype = i32
        L.dspark_schedule_capacity.argtypes = [p, i32, i32, p, i64, p, p, sz, p]
        L.dspark_schedule_topk.restype = i32
        L.dspark_schedule_topk.argtypes = [p, i32, i32, p, p, p, p, p, sz, p]
        L.dspark_verify_attn_workspace_size.restype = sz
        L.dspark_verify_attn_workspace_size.argtypes = [i32] * 8 + [i32]
        L.dspark_verify_attn.restype = i32
        L.dspark_verify_attn.argtypes = [p, p, p, p, p, p, i32, p, p, i32, i32, i32, i32, i32, i32,
                                         i32, f32, i32, p, p, p, sz, p]
        L.dspark_accept_workspace_size.restype = sz
        L.dspark_accept_workspace_size.argtypes = [i32, i32, i32]
        L.dspark_accept.restype = i32
        L.dspark_accept.argtypes = [p, p, p, i32, i64, p, p, i32, i32, i32, f32, p, p, p, p, sz, p]
        L.dspark_markov_draft_workspace_size.restype = sz
        L.dspark_markov_draft_workspace_size.argtypes = [i32, i32, i32, i32]
        L.dspark_markov_draft.restype = i32
        L.dspark_markov_draft.argtypes = [p, p, i32, i64, p, p, i32, p, p, i32, p, p, f32, i32, i32,
                                          i32, p, p, p, p, sz, p]
        L.dspark_rnn_draft_workspace_size.restype = sz
        L.dspark_rnn_draft_workspace_size.argtypes = [i32, i32, i32, i32]
        L.dspark_rnn_draft.restype = i32
        L.dspark_rnn_draft.argtypes = [p, p, i32, i64, p, p, p, i32, p, p, i32, p, p, f32, i32, i32,
                                       i32, p, p, p, p, sz, p]
        L.dspark_check_verify_inputs.restype = i32
        L.dspark_check_verify_inputs.argtypes = [p, i32, p, p, i32, i32, i32, i32, p, p]
        L.dspark_check_accept_inputs.restype = i32
        L.dspark_check_accept_inputs.argtypes = [p, p, i32, i32, p, p]
        L.dspark_check_schedule_inputs.restype = i32
        L.dspark_check_schedule_inputs.argtypes = [p, i32, i32, p, p]
        L.dspark_check_draft_inputs.restype = i32
        L.dspark_check_draft_inputs.argtypes = [p, p, i32, i32, p, p]
        _lib = L
    return _lib


def dspark_abi_version() -> int:
    return int(lib().dspark_abi_version())


def dspark_last_error() -> str:
    return lib().dspark_last_error().decode()


def _raise(st: int, what: str) -> None:
    if st != 0:
        raise DSparkError(f"{what}: {STATUS.get(st, st)}: {dspark_last_error()}", st)


def _dev(t: Optional[torch.Tensor], name: str, dtype=None, shape=None, optional=False):
    if t is None:
        if optional:
            return None
        raise DSparkError(f"{name} is required")
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise DSparkError(f"{name} must be a torch tensor on a ROCm device")
    if dtype is not None and t.dtype != dtype:
        raise DSparkError(f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise DSparkError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise DSparkError(f"{name} must be contiguous")
    return t


def _p(t: Optional[torch.Tensor]):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream(stream) -> C.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return C.c_void_p(stream.cuda_stream)


def _workspace(nbytes: int, device, ws: Optional[torch.Tensor]) -> Tuple[Optional[torch.Tensor], int]:
    if nbytes == 0:
        return ws, 0 if ws is None else ws.numel() * ws.element_size()
    if ws is None:
        ws = torch.empty(nbytes, dtype=torch.uint8, device=device)
    return ws, ws.numel() * ws.element_size()


_DT = {torch.float32: DSPARK_F32, torch.bfloat16: DSPARK_BF16}


# ------------------------------------------------------------------ stage 1

def dspark_schedule_workspace_size(R: int, K: int) -> int:
    return int(lib().dspark_schedule_workspace_size(R, K))


# ---------------------------------------------------------------- input checks

CHECK_RULES = {
    "verify": {1: "rows of the request outside the batch (or cu_q decreasing)", 2: "q_len above max_q",
               3: "kv_len outside [q_len, max_pages * page_size]", 4: "block-table entry outside the cache"},
    "accept": {1: "rows of the request outside the batch (or cu_q decreasing)", 2: "len = q_len - 1 outside [0, K]",
               3: "uniform outside [0, 1)"},
    "schedule": {1: "confidence outside [0, 1]"},
    "draft": {1: "temperature not finite and positive", 2: "uniform outside [0, 1)"},
}


def debug_checks() -> bool:
    """DSPARK_DEBUG=1: the stage wrappers check their device-side inputs
    first and raise on the first rule broken (each call then waits for its
    check)."""
    return os.environ.get("DSPARK_DEBUG", "0") not in ("", "0")


def _report(report: torch.Tensor, kind: str, stream) -> Optional[tuple]:
    (torch.cuda.current_stream(report.device) if stream is None else stream).synchronize()
    code, r, i, v = (int(x) for x in report.cpu().tolist())
    return None if code == 0 else (code, r, i, v, CHECK_RULES[kind].get(code, "?"))


def check_verify_inputs(block_table: torch.Tensor, kv_len: torch.Tensor, cu_q: torch.Tensor, max_q: int,
                        page_size: int, num_pages: int, stream=None) -> Optional[tuple]:
    """First broken rule of dspark_verify_attn's device-side inputs as
    (code, request, index, value, rule) or None; waits for the check."""
    _dev(block_table, "block_table", torch.int32)
    R, max_pages = block_table.shape
    _dev(kv_len, "kv_len", torch.int32, (R,))
    _dev(cu_q, "cu_q", torch.int32, (R + 1,))
    report = torch.empty(4, dtype=torch.int32, device=cu_q.device)
    st = lib().dspark_check_verify_inputs(_p(block_table), max_pages, _p(kv_len), _p(cu_q), R, max_q,
                                          page_size, num_pages, _p(report), _stream(stream))
    _raise(st, "dspark_check_verify_inputs")
    return _report(report, "verify", stream)


def check_accept_inputs(cu_q: torch.Tensor, u: Optional[torch.Tensor], K: int, stream=None) -> Optional[tuple]:
    _dev(cu_q, "cu_q", torch.int32)
    R = cu_q.numel() - 1
    _dev(u, "u", torch.float32, (R, K + 1), optional=True)
    report = torch.empty(4, dtype=torch.int32, device=cu_q.device)
    st = lib().dspark_check_accept_inputs(_p(cu_q), _p(u), R, K, _p(report), _stream(stream))
    _raise(st, "dspark_check_accept_inputs")
    return _report(report, "accept", stream)


def check_schedule_inputs(conf: torch.Tensor, stream=None) -> Optional[tuple]:
    _dev(conf, "conf", torch.float32)
    R, K = conf.shape
    report = torch.empty(4, dtype=torch.int32, device=conf.device)
    st = lib().dspark_check_schedule_inputs(_p(conf), R, K, _p(report), _stream(stream))
    _raise(st, "dspark_check_schedule_inputs")
    return _report(report, "schedule", stream)


def check_draft_inputs(u: torch.Tensor, sts_temp: Optional[torch.Tensor] = None,
                       stream=None) -> Optional[tuple]:
    """First broken rule of a draft block's uniforms [R, K] and per-position
    temperatures [K] (request -1) as (code, request, index, value, rule) or
    None; waits for the check."""
    _dev(u, "u", torch.float32)
    R, K = u.shape
    _dev(sts_temp, "sts_temp", torch.float32, (K,), optional=True)
    report = torch.empty(4, dtype=torch.int32, device=u.device)
    st = lib().dspark_check_draft_inputs(_p(u), _p(sts_temp), R, K, _p(report), _stream(stream))
    _raise(st, "dspark_check_draft_inputs")
    return _report(report, "draft", stream)


def _cache_pages(cache: torch.Tensor, strides: Sequence[int], heads: int, page_size: int, dim: int) -> int:
    """Pages a flat cache holds: page p is readable when its last element,
    p * s0 + (heads - 1) * s1 + (page_size - 1) * s2 + dim - 1, is inside."""
    s0, s1, s2 = (int(x) for x in strides)
    span = (heads - 1) * s1 + (page_size - 1) * s2 + dim
    return max(0, (cache.numel() - span) // s0 + 1) if s0 > 0 else 0


def _debug_raise(found: Optional[tuple], what: str) -> None:
    if found is not None:
        code, r, i, v, rule = found
        raise DSparkError(f"{what}: input check failed: request {r}: {rule} (code {code}, index {i}, "
                          f"value {v})", 1)


def dspark_schedule(conf: torch.Tensor, sps: torch.Tensor, mode: int = 0,
                    len_out: Optional[torch.Tensor] = None, cu_q: Optional[torch.Tensor] = None,
                    tok_req: Optional[torch.Tensor] = None, want_tok_req: bool = False,
                    ws: Optional[torch.Tensor] = None, stream=None):
    """conf fp32 [R, K], sps fp64 [> R*(K+1)] -> (len int32 [R], cu_q int32 [R+1], tok_req|None)."""
    _dev(conf, "conf", torch.float32)
    if conf.dim() != 2:
        raise DSparkError("conf must be [R, K]")
    R, K = conf.shape
    _dev(sps, "sps", torch.float64)
    dev = conf.device
    if len_out is None:
        len_out = torch.empty(R, dtype=torch.int32, device=dev)
    if cu_q is None:
        cu_q = torch.empty(R + 1, dtype=torch.int32, device=dev)
    if tok_req is None and want_tok_req:
        tok_req = torch.empty(R * (K + 1), dtype=torch.int32, device=dev)
    _dev(len_out, "len", torch.int32, (R,))
    _dev(cu_q, "cu_q", torch.int32, (R + 1,))
    _dev(tok_req, "tok_req", torch.int32, (R * (K + 1),), optional=True)
    ws, ws_bytes = _workspace(dspark_schedule_workspace_size(R, K), dev, ws)
    if debug_checks() and K > 0:
        _debug_raise(check_schedule_inputs(conf, stream), "dspark_schedule")
    st = lib().dspark_schedule(_p(conf), R, K, _p(sps), sps.numel(), mode, _p(len_out), _p(cu_q),
                               _p(tok_req), _p(ws), ws_bytes, _stream(stream))
    _raise(st, "dspark_schedule")
    return len_out, cu_q, tok_req


def dspark_schedule_noalloc(conf: torch.Tensor, sps: torch.Tensor, mode: int,
                            len_out: torch.Tensor, cu_q: torch.Tensor,
                            tok_req: Optional[torch.Tensor] = None, stream=None):
    """As dspark_schedule, with the library's fixed scratch array as workspace;
    every output is the caller's (nothing is allocated)."""
    _dev(conf, "conf", torch.float32)
    if conf.dim() != 2:
        raise DSparkError("conf must be [R, K]")
    R, K = conf.shape
    _dev(sps, "sps", torch.float64)
    _dev(len_out, "len", torch.int32, (R,))
    _dev(cu_q, "cu_q", torch.int32, (R + 1,))
    _dev(tok_req, "tok_req", torch.int32, (R * (K + 1),), optional=True)
    st = lib().dspark_schedule_noalloc(_p(conf), R, K, _p(sps), sps.numel(), mode, _p(len_out),
                                       _p(cu_q), _p(tok_req), _stream(stream))
    _raise(st, "dspark_schedule_noalloc")
    return len_out, cu_q, tok_req


def dspark_schedule_capacity(conf_prev: torch.Tensor, sps: torch.Tensor,
                             capacity: Optional[torch.Tensor] = None,
                             ws: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """conf_prev fp32 [R, K], sps fp64 [> R*(K+1)] -> capacity int32 [1] (device)."""
    _dev(conf_prev, "conf_prev", torch.float32)
    if conf_prev.dim() != 2:
        raise DSparkError("conf_prev must be [R, K]")
    R, K = conf_prev.shape
    _dev(sps, "sps", torch.float64)
    dev = conf_prev.device
    if capacity is None:
        capacity = torch.empty(1, dtype=torch.int32, device=dev)
    _dev(capacity, "capacity", torch.int32, (1,))
    ws, ws_bytes = _workspace(dspark_schedule_workspace_size(R, K), dev, ws)
    st = lib().dspark_schedule_capacity(_p(conf_prev), R, K, _p(sps), sps.numel(), _p(capacity),
                                        _p(ws), ws_bytes, _stream(stream))
    _raise(st, "dspark_schedule_capacity")
    return capacity


def dspark_schedule_topk(conf: torch.Tensor, capacity: torch.Tensor,
                         len_out: Optional[torch.Tensor] = None,
                         cu_q: Optional[torch.Tensor] = None,
                         tok_req: Optional[torch.Tensor] = None, want_tok_req: bool = False,
                         ws: Optional[torch.Tensor] = None, stream=None):
    """conf fp32 [R, K], capacity int32 [1] (device) -> (len, cu_q, tok_req|None)."""
    _dev(conf, "conf", torch.float32)
    if conf.dim() != 2:
        raise DSparkError("conf must be [R, K]")
    R, K = conf.shape
    _dev(capacity, "capacity", torch.int32, (1,))
    dev = conf.device
    if len_out is None:
        len_out = torch.empty(R, dtype=torch.int32, device=dev)
    if cu_q is None:
        cu_q = torch.empty(R + 1, dtype=torch.int32, device=dev)
    if tok_req is None and want_tok_req:
        tok_req = torch.empty(R * (K + 1), dtype=torch.int32, device=dev)
    _dev(len_out, "len", torch.int32, (R,))
    _dev(cu_q, "cu_q", torch.int32, (R + 1,))
    _dev(tok_req, "tok_req", torch.int32, (R * (K + 1),), optional=True)
    ws, ws_bytes = _workspace(dspark_schedule_workspace_size(R, K), dev, ws)
    st = lib().dspark_schedule_topk(_p(conf), R, K, _p(capacity), _p(len_out), _p(cu_q),
                                    _p(tok_req), _p(ws), ws_bytes, _stream(stream))
    _raise(st, "dspark_schedule_topk")
    return len_out, cu_q, tok_req


# ------------------------------------------------------------------ stage 2

def dspark_verify_attn_workspace_size(R: int, max_q: int, Hq: int, Hkv: int, Dqk: int, Dv: int,
                                      max_pages: int, page_size: int, dtype: torch.dtype) -> int:
    return int(lib().dspark_verify_attn_workspace_size(R, max_q, Hq, Hkv, Dqk, Dv, max_pages,
                                                       page_size, _DT[dtype]))


def dspark_verify_attn(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor,
                       k_strides: Sequence[int], v_strides: Sequence[int],
                       block_table: torch.Tensor, kv_len: torch.Tensor, cu_q: torch.Tensor,
                       max_q: int, Hkv: int, Dv: int, page_size: int, scale: float,
                       out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
                       want_lse: bool = False, ws: Optional[torch.Tensor] = None, stream=None):
    """q [total_q(or more rows), Hq, Dqk]; caches flat or shaped, addressed by element strides.
    Returns (out [rows of q, Hq, Dv], lse|None)."""
    if q.dtype not in _DT:
        raise DSparkError("q must be float32 or bfloat16")
    _dev(q, "q")
    if q.dim() != 3:
        raise DSparkError("q must be [tokens, Hq, Dqk]")
    rows, Hq, Dqk = q.shape
    _dev(k_cache, "k_cache", q.dtype)
    _dev(v_cache, "v_cache", q.dtype)
    _dev(block_table, "block_table", torch.int32)
    if block_table.dim() != 2:
        raise DSparkError("block_table must be [R, max_pages]")
    R, max_pages = block_table.shape
    _dev(kv_len, "kv_len", torch.int32, (R,))
    _dev(cu_q, "cu_q", torch.int32, (R + 1,))
    if out is None:
        out = torch.empty((rows, Hq, Dv), dtype=q.dtype, device=q.device)
    _dev(out, "out", q.dtype, (rows, Hq, Dv))
    if lse is None and want_lse:
        lse = torch.empty((rows, Hq), dtype=torch.float32, device=q.device)
    _dev(lse, "lse", torch.float32, (rows, Hq), optional=True)
    need = dspark_verify_attn_workspace_size(R, max_q, Hq, Hkv, Dqk, Dv, max_pages, page_size,
                                             q.dtype)
    ws, ws_bytes = _workspace(need, q.device, ws)
    if debug_checks():
        num_pages = min(_cache_pages(k_cache, k_strides, Hkv, page_size, Dqk),
                        _cache_pages(v_cache, v_strides, Hkv, page_size, Dv))
        _debug_raise(check_verify_inputs(block_table, kv_len, cu_q, max_q, page_size, max(num_pages, 1),
                                         stream), "dspark_verify_attn")
    ks = (C.c_int64 * 3)(*[int(x) for x in k_strides])
    vs = (C.c_int64 * 3)(*[int(x) for x in v_strides])
    st = lib().dspark_verify_attn(_p(q), _p(k_cache), _p(v_cache), ks, vs, _p(block_table),
                                  max_pages, _p(kv_len), _p(cu_q), R, max_q, Hq, Hkv, Dqk, Dv,
                                  page_size, float(scale), _DT[q.dtype], _p(out), _p(lse), _p(ws),
                                  ws_bytes, _stream(stream))
    _raise(st, "dspark_verify_attn")
    return out, lse


# ------------------------------------------------------------------ stage 3

def dspark_accept_workspace_size(R: int, K: int, V: int) -> int:
    return int(lib().dspark_accept_workspace_size(R, K, V))


def dspark_accept(draft_tok: torch.Tensor, logits: torch.Tensor, cu_q: torch.Tensor,
                  draft_p: Optional[torch.Tensor] = None, u: Optional[torch.Tensor] = None,
                  inv_temperature: float = 1.0, accepted_len: Optional[torch.Tensor] = None,
                  next_tok: Optional[torch.Tensor] = None, accept_rate: Optional[torch.Tensor] = None,
                  want_rate: bool = False, ws: Optional[torch.Tensor] = None, stream=None):
    """draft_tok int32 [R, K]; logits [rows, V] (fp32/bf16, row stride = stride(0));
    draft_p fp32 [R, K, V] and u fp32 [R, K+1] for stochastic acceptance (both None: greedy).
    Returns (accepted_len int32 [R], next_tok int32 [R], accept_rate|None)."""
    _dev(draft_tok, "draft_tok", torch.int32)
    if draft_tok.dim() != 2:
        raise DSparkError("draft_tok must be [R, K]")
    R, K = draft_tok.shape
    if logits.dtype not in _DT or logits.dim() != 2 or logits.device.type != "cuda":
        raise DSparkError("logits must be a 2-D float32/bfloat16 ROCm tensor")
    if logits.stride(1) != 1:
        raise DSparkError("logits rows must be contiguous")
    V = logits.shape[1]
    ld = logits.stride(0)
    _dev(cu_q, "cu_q", torch.int32, (R + 1,))
    _dev(draft_p, "draft_p", torch.float32, (R, K, V), optional=True)
    _dev(u, "u", torch.float32, (R, K + 1), optional=True)
    dev = draft_tok.device
    if accepted_len is None:
        accepted_len = torch.empty(R, dtype=torch.int32, device=dev)
    if next_tok is None:
        next_tok = torch.empty(R, dtype=torch.int32, device=dev)
    if accept_rate is None and want_rate:
        accept_rate = torch.empty(R * (K + 1), dtype=torch.float32, device=dev)
    _dev(accepted_len, "accepted_len", torch.int32, (R,))
    _dev(next_tok, "next_tok", torch.int32, (R,))
    _dev(accept_rate, "accept_rate", torch.float32, optional=True)
    need = dspark_accept_workspace_size(R, K, V)
    ws, ws_bytes = _workspace(need, dev, ws)
    if debug_checks():
        _debug_raise(check_accept_inputs(cu_q, u, K, stream), "dspark_accept")
    st = lib().dspark_accept(_p(draft_tok), _p(draft_p), C.c_void_p(logits.data_ptr()),
                             _DT[logits.dtype], ld, _p(u), _p(cu_q), R, K, V,
                             float(inv_temperature), _p(accepted_len), _p(next_tok),
                             _p(accept_rate), _p(ws), ws_bytes, _stream(stream))
    _raise(st, "dspark_accept")
    return accepted_len, next_tok, accept_rate


def dspark_markov_draft_workspace_size(R: int, K: int, V: int, rank: int) -> int:
    return int(lib().dspark_markov_draft_workspace_size(R, K, V, rank))


def dspark_markov_draft(anchor: torch.Tensor, base_logits: torch.Tensor, W1: torch.Tensor,
                        W2t: torch.Tensor, w_conf: torch.Tensor, u: torch.Tensor, K: int,
                        hidden: Optional[torch.Tensor] = None,
                        sts_temp: Optional[torch.Tensor] = None, inv_temperature: float = 1.0,
                        draft_tok: Optional[torch.Tensor] = None,
                        draft_p: Optional[torch.Tensor] = None, conf: Optional[torch.Tensor] = None,
                        ws: Optional[torch.Tensor] = None, stream=None):
    """anchor int32 [R]; base_logits [R*K, V] (fp32/bf16, row stride = stride(0));
    W1, W2t bf16 [V, rank]; w_conf fp32 [d + rank]; u fp32 [R, K]; hidden bf16
    [R, K, d] or None; sts_temp fp32 [K] or None.
    Returns (draft_tok int32 [R, K], draft_p fp32 [R, K, V], conf fp32 [R, K])."""
    _dev(anchor, "anchor", torch.int32)
    R = anchor.shape[0]
    if base_logits.dtype not in _DT or base_logits.dim() != 2 or base_logits.device.type != "cuda":
        raise DSparkError("base_logits must be a 2-D float32/bfloat16 ROCm tensor")
    if base_logits.stride(1) != 1 or base_logits.shape[0] != R * K:
        raise DSparkError("base_logits must be [R*K, V] with contiguous rows")
    V = base_logits.shape[1]
    ld = base_logits.stride(0)
    _dev(W1, "W1", torch.bfloat16)
    rank = W1.shape[1]
    _dev(W2t, "W2t", torch.bfloat16, (V, rank))
    if W1.shape != (V, rank):
        raise DSparkError("W1 must be [V, rank]")
    d = 0 if hidden is None else hidden.shape[-1]
    _dev(hidden, "hidden", torch.bfloat16, (R, K, d), optional=True)
    _dev(w_conf, "w_conf", torch.float32, (d + rank,))
    _dev(sts_temp, "sts_temp", torch.float32, (K,), optional=True)
    _dev(u, "u", torch.float32, (R, K))
    dev = anchor.device
    if draft_tok is None:
        draft_tok = torch.empty((R, K), dtype=torch.int32, device=dev)
    if draft_p is None:
        draft_p = torch.empty((R, K, V), dtype=torch.float32, device=dev)
    if conf is None:
        conf = torch.empty((R, K), dtype=torch.float32, device=dev)
    _dev(draft_tok, "draft_tok", torch.int32, (R, K))
    _dev(draft_p, "draft_p", torch.float32, (R, K, V))
    _dev(conf, "conf", torch.float32, (R, K))
    need = dspark_markov_draft_workspace_size(R, K, V, rank)
    if need == 0:
        raise DSparkError(f"unsupported shape: R={R} V={V} rank={rank}")
    ws, ws_bytes = _workspace(need, dev, ws)
    if debug_checks():
        _debug_raise(check_draft_inputs(u, sts_temp, stream), "dspark_markov_draft")
    st = lib().dspark_markov_draft(_p(anchor), C.c_void_p(base_logits.data_ptr()),
                                   _DT[base_logits.dtype], ld, _p(W1), _p(W2t), rank, _p(hidden),
                                   _p(w_conf), d, _p(sts_temp), _p(u), float(inv_temperature), R,
                                   K, V, _p(draft_tok), _p(draft_p), _p(conf), _p(ws), ws_bytes,
                                   _stream(stream))
    _raise(st, "dspark_markov_draft")
    return draft_tok, draft_p, conf


def dspark_rnn_draft_workspace_size(R: int, K: int, V: int, rank: int) -> int:
    return int(lib().dspark_rnn_draft_workspace_size(R, K, V, rank))


def dspark_rnn_draft(anchor: torch.Tensor, base_logits: torch.Tensor, W1: torch.Tensor,
                     W2t: torch.Tensor, Wrnn: torch.Tensor, w_conf: torch.Tensor, u: torch.Tensor,
                     K: int, hidden: Optional[torch.Tensor] = None,
                     sts_temp: Optional[torch.Tensor] = None, inv_temperature: float = 1.0,
                     draft_tok: Optional[torch.Tensor] = None,
                     draft_p: Optional[torch.Tensor] = None, conf: Optional[torch.Tensor] = None,
                     ws: Optional[torch.Tensor] = None, stream=None):
    """As dspark_markov_draft, plus Wrnn bf16 [3 rank, 2 rank + d] (gate,
    candidate and output rows; columns [s; e; h]).
    Returns (draft_tok int32 [R, K], draft_p fp32 [R, K, V], conf fp32 [R, K])."""
    _dev(anchor, "anchor", torch.int32)
    R = anchor.shape[0]
    if base_logits.dtype not in _DT or base_logits.dim() != 2 or base_logits.device.type != "cuda":
        raise DSparkError("base_logits must be a 2-D float32/bfloat16 ROCm tensor")
    if base_logits.stride(1) != 1 or base_logits.shape[0] != R * K:
        raise DSparkError("base_logits must be [R*K, V] with contiguous rows")
    V = base_logits.shape[1]
    ld = base_logits.stride(0)
    _dev(W1, "W1", torch.bfloat16)
    rank = W1.shape[1]
    _dev(W2t, "W2t", torch.bfloat16, (V, rank))
    if W1.shape != (V, rank):
        raise DSparkError("W1 must be [V, rank]")
    d = 0 if hidden is None else hidden.shape[-1]
    _dev(hidden, "hidden", torch.bfloat16, (R, K, d), optional=True)
    _dev(Wrnn, "Wrnn", torch.bfloat16, (3 * rank, 2 * rank + d))
    _dev(w_conf, "w_conf", torch.float32, (d + rank,))
    _dev(sts_temp, "sts_temp", torch.float32, (K,), optional=True)
    _dev(u, "u", torch.float32, (R, K))
    dev = anchor.device
    if draft_tok is None:
        draft_tok = torch.empty((R, K), dtype=torch.int32, device=dev)
    if draft_p is None:
        draft_p = torch.empty((R, K, V), dtype=torch.float32, device=dev)
    if conf is None:
        conf = torch.empty((R, K), dtype=torch.float32, device=dev)
    _dev(draft_tok, "draft_tok", torch.int32, (R, K))
    _dev(draft_p, "draft_p", torch.float32, (R, K, V))
    _dev(conf, "conf", torch.float32, (R, K))
    need = dspark_rnn_draft_workspace_size(R, K, V, rank)
    if need == 0:
        raise DSparkError(f"unsupported shape: R={R} V={V} rank={rank}")
    ws, ws_bytes = _workspace(need, dev, ws)
    if debug_checks():
        _debug_raise(check_draft_inputs(u, sts_temp, stream), "dspark_rnn_draft")
    st = lib().dspark_rnn_draft(_p(anchor), C.c_void_p(base_logits.data_ptr()),
                                _DT[base_logits.dtype], ld, _p(W1), _p(W2t), _p(Wrnn), rank,
                                _p(hidden), _p(w_conf), d, _p(sts_temp), _p(u),
                                float(inv_temperature), R, K, V, _p(draft_tok), _p(draft_p),
                                _p(conf), _p(ws), ws_bytes, _stream(stream))
    _raise(st, "dspark_rnn_draft")
    return draft_tok, draft_p, conf
