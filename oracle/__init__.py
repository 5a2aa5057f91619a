"""CPU oracle for the SparseSpec-L decode hot path (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import
this package.  It wraps ``oracle.c`` (plain C, fp64) through ctypes; it shares
no code with the HIP library and never imports it.

Functions take the bf16 bit-pattern arrays produced by the workload generator
and return float64 numpy arrays.  See ``oracle.c`` for the definitions and the
paper passages they follow.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = False, out: Optional[str] = None, extra_flags: Sequence[str] = ()) -> str:
    """Compile oracle.c with gcc (OpenMP) into a shared library; returns its path."""
    out = out or _LIB_PATH
    if force or not os.path.exists(out) or os.path.getmtime(out) < os.path.getmtime(_SRC):
        tmp = out + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall",
               *extra_flags, _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, out)
    return out


_i32p = ctypes.POINTER(ctypes.c_int32)
_u16p = ctypes.POINTER(ctypes.c_uint16)
_f64p = ctypes.POINTER(ctypes.c_double)


def _bind(lib):
    lib.oracle_verify.argtypes = [ctypes.c_int] * 6 + [_i32p, _i32p, _u16p, _u16p, _u16p,
                                                       ctypes.c_double, ctypes.c_int,
                                                       _i32p, ctypes.c_int, _f64p, _f64p]
    lib.oracle_verify.restype = ctypes.c_int
    lib.oracle_select.argtypes = [ctypes.c_int] * 3 + [_i32p, _f64p, ctypes.c_int, ctypes.c_int,
                                                       ctypes.c_int, _i32p, _i32p]
    lib.oracle_select.restype = ctypes.c_int
    lib.oracle_draft.argtypes = [ctypes.c_int] * 6 + [_i32p, _u16p, _u16p, _u16p, _i32p,
                                                      ctypes.c_double, _f64p]
    lib.oracle_draft.restype = ctypes.c_int
    lib.oracle_draft_step.argtypes = [ctypes.c_int] * 8 + [_i32p, _i32p, _u16p, _u16p, _u16p,
                                                           _i32p, ctypes.c_double, _f64p]
    lib.oracle_draft_step.restype = ctypes.c_int
    lib.oracle_draft_step_heads.argtypes = lib.oracle_draft_step.argtypes
    lib.oracle_draft_step_heads.restype = ctypes.c_int
    _f32p = ctypes.POINTER(ctypes.c_float)
    lib.oracle_row_stats.argtypes = [ctypes.c_int] * 3 + [_u16p, _f32p, _f64p, _i32p]
    lib.oracle_row_stats.restype = ctypes.c_int
    lib.oracle_greedy_accept.argtypes = [ctypes.c_int] * 4 + [_i32p, _u16p, _f32p, _i32p, _i32p,
                                                              _i32p]
    lib.oracle_greedy_accept.restype = ctypes.c_int
    lib.oracle_spec_accept.argtypes = [ctypes.c_int] * 4 + [_i32p, _f32p, _f32p, ctypes.c_double,
                                                            _i32p, _f64p, _f64p, _i32p, _i32p]
    lib.oracle_spec_accept.restype = ctypes.c_int
    lib.oracle_head_scores.argtypes = [ctypes.c_int] * 6 + [_i32p, _i32p, _u16p, _u16p,
                                                            ctypes.c_double, ctypes.c_int, _f64p]
    lib.oracle_head_scores.restype = ctypes.c_int
    lib.oracle_draft_heads.argtypes = [ctypes.c_int] * 6 + [_i32p, _u16p, _u16p, _u16p, _i32p,
                                                            ctypes.c_double, _f64p]
    lib.oracle_draft_heads.restype = ctypes.c_int
    lib.oracle_index_count.argtypes = [ctypes.c_int] * 4
    lib.oracle_index_count.restype = ctypes.c_int
    lib.oracle_ema.argtypes = [ctypes.c_double] * 3
    lib.oracle_ema.restype = ctypes.c_double
    lib.oracle_ctrl_observe.argtypes = [_f64p, _f64p, ctypes.c_int, ctypes.c_int, ctypes.c_double]
    lib.oracle_ctrl_observe.restype = ctypes.c_int
    lib.oracle_accept_prob.argtypes = [ctypes.c_double] * 3
    lib.oracle_accept_prob.restype = ctypes.c_double
    lib.oracle_expected_accepted.argtypes = [_f64p, ctypes.c_int]
    lib.oracle_expected_accepted.restype = ctypes.c_double
    lib.oracle_step_efficiency.argtypes = [_f64p, ctypes.c_int, ctypes.c_double, ctypes.c_double]
    lib.oracle_step_efficiency.restype = ctypes.c_double
    lib.oracle_choose_k.argtypes = [_f64p, ctypes.c_int, _i32p, ctypes.c_int,
                                    ctypes.c_double, ctypes.c_double]
    lib.oracle_choose_k.restype = ctypes.c_int
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = ctypes.c_int
    lib.oracle_set_num_threads.argtypes = [ctypes.c_int]
    lib.oracle_set_num_threads.restype = None
    return lib


def load(path: Optional[str] = None):
    """Load (building if needed) the oracle library.  ``path`` loads a variant."""
    global _lib
    if path is not None:
        return _bind(ctypes.CDLL(path))
    if _lib is None:
        _lib = _bind(ctypes.CDLL(build()))
    return _lib


def _p(a: np.ndarray, ty):
    return a.ctypes.data_as(ty)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def verify(w, units: Optional[Sequence[int]] = None, *, q=None, k=None, v=None,
           ctx_len=None, q_len=None, lib=None):
    """Dense verify attention + Eq. 3 scores.

    Returns ``(out, scores)``: ``out`` float64 ``[batch][max_q][Hq][d]`` and
    ``scores`` float64 ``[batch][Hkv][max_ctx]``; rows/units not computed are 0
    and entries past each context length are 0.
    """
    lib = lib or load()
    q = _c(w.q if q is None else q, np.uint16)
    k = _c(w.k if k is None else k, np.uint16)
    v = _c(w.v if v is None else v, np.uint16)
    ctx = _c(w.ctx_len if ctx_len is None else ctx_len, np.int32)
    ql = _c(w.q_len if q_len is None else q_len, np.int32)
    out = np.zeros((w.batch, w.max_q, w.n_q_heads, w.head_dim), dtype=np.float64)
    sc = np.zeros((w.batch, w.n_kv_heads, w.max_ctx), dtype=np.float64)
    if units is None:
        up, nu = None, 0
    else:
        ua = _c(list(units), np.int32)
        up, nu = _p(ua, _i32p), len(ua)
    rc = lib.oracle_verify(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.max_ctx, w.max_q,
                           _p(ctx, _i32p), _p(ql, _i32p), _p(q, _u16p), _p(k, _u16p),
                           _p(v, _u16p), float(w.sm_scale), int(w.window), up, nu,
                           _p(out, _f64p), _p(sc, _f64p))
    if rc != 0:
        raise ValueError("oracle_verify rejected its arguments")
    return out, sc


def select(w, scores: np.ndarray, *, ctx_len=None, k_sink=None, k_recent=None, budget=None,
           lib=None):
    """Eq. 4 index sets.  Returns ``(idx, n_idx)``; idx int32 ``[batch][Hkv][budget]``
    with unused slots set to -1."""
    lib = lib or load()
    ctx = _c(w.ctx_len if ctx_len is None else ctx_len, np.int32)
    ks = w.k_sink if k_sink is None else k_sink
    kr = w.k_recent if k_recent is None else k_recent
    B = w.budget if budget is None else budget
    sc = _c(scores, np.float64)
    max_ctx = sc.shape[-1]
    idx = np.full((w.batch, w.n_kv_heads, B), -1, dtype=np.int32)
    n_idx = np.zeros(w.batch, dtype=np.int32)
    rc = lib.oracle_select(w.batch, w.n_kv_heads, max_ctx, _p(ctx, _i32p), _p(sc, _f64p),
                           int(ks), int(kr), int(B), _p(idx, _i32p), _p(n_idx, _i32p))
    if rc != 0:
        raise ValueError("oracle_select rejected its arguments")
    return idx, n_idx


def index_count(T: int, k_sink: int, k_recent: int, budget: int, lib=None) -> int:
    lib = lib or load()
    return int(lib.oracle_index_count(T, k_sink, k_recent, budget))


def draft(w, idx: np.ndarray, n_idx: np.ndarray, *, q_draft=None, k=None, v=None, lib=None):
    """Eq. 5 draft attention over gathered rows; float64 ``[batch][Hq][d]``."""
    lib = lib or load()
    qd = _c(w.q_draft if q_draft is None else q_draft, np.uint16)
    k = _c(w.k if k is None else k, np.uint16)
    v = _c(w.v if v is None else v, np.uint16)
    idx = _c(idx, np.int32)
    n = _c(n_idx, np.int32)
    B = idx.shape[-1]
    out = np.zeros((w.batch, w.n_q_heads, w.head_dim), dtype=np.float64)
    rc = lib.oracle_draft(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.max_ctx, B,
                          _p(n, _i32p), _p(qd, _u16p), _p(k, _u16p), _p(v, _u16p),
                          _p(idx, _i32p), float(w.sm_scale), _p(out, _f64p))
    if rc != 0:
        raise ValueError("oracle_draft rejected its arguments")
    return out


def draft_step(w, idx: np.ndarray, base_len, cur_len, *, q_draft=None, k=None, v=None,
               k_sink=None, k_recent=None, per_head=False, lib=None):
    """One draft-round step: attention over the fixed sink/TopK part of the
    index set built at ``base_len`` plus the recent window slid to end at
    ``cur_len``; float64 ``[batch][Hq][d]``.  The budget is ``idx.shape[-1]``.
    ``per_head``: idx holds one set per query head ``[batch][Hq][budget]``."""
    lib = lib or load()
    qd = _c(w.q_draft if q_draft is None else q_draft, np.uint16)
    k = _c(w.k if k is None else k, np.uint16)
    v = _c(w.v if v is None else v, np.uint16)
    idx = _c(idx, np.int32)
    base = _c(base_len, np.int32)
    cur = _c(cur_len, np.int32)
    ks = int(w.k_sink if k_sink is None else k_sink)
    kr = int(w.k_recent if k_recent is None else k_recent)
    B = idx.shape[-1]
    out = np.zeros((w.batch, w.n_q_heads, w.head_dim), dtype=np.float64)
    fn = lib.oracle_draft_step_heads if per_head else lib.oracle_draft_step
    rc = fn(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.max_ctx, B,
            ks, kr, _p(base, _i32p), _p(cur, _i32p), _p(qd, _u16p),
            _p(k, _u16p), _p(v, _u16p), _p(idx, _i32p), float(w.sm_scale),
            _p(out, _f64p))
    if rc != 0:
        raise ValueError("oracle_draft_step rejected its arguments")
    return out


def _logit_ptrs(logits: np.ndarray):
    """(bf16 bits pointer, fp32 pointer, keep-alive array) for uint16 or float32 logits."""
    if logits.dtype == np.uint16:
        a = _c(logits, np.uint16)
        return _p(a, _u16p), None, a
    if logits.dtype == np.float32:
        a = _c(logits, np.float32)
        return None, a.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), a
    raise TypeError("logits must be uint16 (bf16 bits) or float32")


def row_stats(logits: np.ndarray, vocab: Optional[int] = None, lib=None):
    """Per-row entropy (nats, float64) and argmax (lowest index) of
    ``logits`` [n_rows][row_stride] (bf16 bits as uint16, or float32)."""
    lib = lib or load()
    n_rows, stride = logits.shape
    V = stride if vocab is None else vocab
    pb, pf, keep = _logit_ptrs(logits)
    H = np.zeros(n_rows, dtype=np.float64)
    a = np.zeros(n_rows, dtype=np.int32)
    if lib.oracle_row_stats(n_rows, V, stride, pb, pf, _p(H, _f64p), _p(a, _i32p)) != 0:
        raise ValueError("oracle_row_stats rejected its arguments")
    return H, a


def greedy_accept(logits: np.ndarray, draft: np.ndarray, k_len, vocab: Optional[int] = None,
                  lib=None):
    """Greedy verification: ``logits`` [batch][max_k + 1][row_stride], ``draft``
    [batch][max_k] int32, ``k_len`` per sequence; returns (n_accepted, next_token)."""
    lib = lib or load()
    batch, rows, stride = logits.shape
    max_k = rows - 1
    V = stride if vocab is None else vocab
    pb, pf, keep = _logit_ptrs(logits)
    d = _c(draft, np.int32).reshape(batch, max_k)
    kl = _c(k_len, np.int32)
    m = np.zeros(batch, dtype=np.int32)
    t = np.zeros(batch, dtype=np.int32)
    if lib.oracle_greedy_accept(batch, max_k, V, stride, _p(kl, _i32p), pb, pf, _p(d, _i32p),
                                _p(m, _i32p), _p(t, _i32p)) != 0:
        raise ValueError("oracle_greedy_accept rejected its arguments")
    return m, t


def spec_accept(tlogits: np.ndarray, dlogits: np.ndarray, draft: np.ndarray, k_len, tau: float,
                u_acc: np.ndarray, u_smp: np.ndarray, vocab: Optional[int] = None, lib=None):
    """Speculative sampling (see ``oracle_spec_accept``): ``tlogits``
    [batch][max_k + 1][row_stride] and ``dlogits`` [batch][max_k][row_stride]
    float32 logits, ``draft`` [batch][max_k] int32, ``u_acc`` [batch][max_k]
    and ``u_smp`` [batch] uniforms in [0, 1); returns (n_accepted, next_token)."""
    lib = lib or load()
    batch, rows, stride = tlogits.shape
    max_k = rows - 1
    V = stride if vocab is None else vocab
    t = _c(tlogits, np.float32).reshape(batch, max_k + 1, stride)
    d = _c(dlogits, np.float32).reshape(batch, max_k, stride) if max_k > 0 else \
        np.zeros((batch, 1, stride), np.float32)
    dr = _c(draft, np.int32).reshape(batch, max(max_k, 1)) if max_k > 0 else \
        np.zeros((batch, 1), np.int32)
    ua = _c(u_acc, np.float64).reshape(batch, max(max_k, 1)) if max_k > 0 else \
        np.zeros((batch, 1), np.float64)
    us = _c(u_smp, np.float64).reshape(batch)
    kl = _c(k_len, np.int32)
    m = np.zeros(batch, dtype=np.int32)
    nt = np.zeros(batch, dtype=np.int32)
    f32p = ctypes.POINTER(ctypes.c_float)
    if lib.oracle_spec_accept(batch, max_k, V, stride, _p(kl, _i32p), _p(t, f32p), _p(d, f32p),
                              float(tau), _p(dr, _i32p), _p(ua, _f64p), _p(us, _f64p),
                              _p(m, _i32p), _p(nt, _i32p)) != 0:
        raise ValueError("oracle_spec_accept rejected its arguments")
    return m, nt


def head_scores(w, *, q=None, k=None, ctx_len=None, q_len=None, lib=None):
    """Eq. 3 per query head: float64 ``[batch][Hq][max_ctx]``."""
    lib = lib or load()
    q = _c(w.q if q is None else q, np.uint16)
    k = _c(w.k if k is None else k, np.uint16)
    ctx = _c(w.ctx_len if ctx_len is None else ctx_len, np.int32)
    ql = _c(w.q_len if q_len is None else q_len, np.int32)
    sc = np.zeros((w.batch, w.n_q_heads, w.max_ctx), dtype=np.float64)
    rc = lib.oracle_head_scores(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.max_ctx, w.max_q,
                                _p(ctx, _i32p), _p(ql, _i32p), _p(q, _u16p), _p(k, _u16p),
                                float(w.sm_scale), int(w.window), _p(sc, _f64p))
    if rc != 0:
        raise ValueError("oracle_head_scores rejected its arguments")
    return sc


def draft_heads(w, idx: np.ndarray, n_idx: np.ndarray, *, q_draft=None, k=None, v=None, lib=None):
    """Eq. 5 with one index set per query head (idx ``[batch][Hq][budget]``);
    float64 ``[batch][Hq][d]``."""
    lib = lib or load()
    qd = _c(w.q_draft if q_draft is None else q_draft, np.uint16)
    k = _c(w.k if k is None else k, np.uint16)
    v = _c(w.v if v is None else v, np.uint16)
    idx = _c(idx, np.int32)
    n = _c(n_idx, np.int32)
    out = np.zeros((w.batch, w.n_q_heads, w.head_dim), dtype=np.float64)
    rc = lib.oracle_draft_heads(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.max_ctx,
                                idx.shape[-1], _p(n, _i32p), _p(qd, _u16p), _p(k, _u16p),
                                _p(v, _u16p), _p(idx, _i32p), float(w.sm_scale), _p(out, _f64p))
    if rc != 0:
        raise ValueError("oracle_draft_heads rejected its arguments")
    return out


def ema(prev: float, observed: float, beta: float, lib=None) -> float:
    return float((lib or load()).oracle_ema(prev, observed, beta))


def ctrl_observe(state: Sequence[float], H: Sequence[float], n_accepted: int, beta: float,
                 lib=None) -> list:
    """Eq. 6 after one verification: returns the new state
    ``[h_acc, h_rej, seen_acc, seen_rej]`` (see ``oracle_ctrl_observe``)."""
    st = _c(list(state), np.float64)
    ha = _c(list(H) if len(H) else [0.0], np.float64)
    if (lib or load()).oracle_ctrl_observe(_p(st, _f64p), _p(ha, _f64p), len(H), int(n_accepted),
                                           float(beta)) != 0:
        raise ValueError("oracle_ctrl_observe rejected its arguments")
    return [float(x) for x in st]


def accept_prob(H: float, h_acc: float, h_rej: float, lib=None) -> float:
    return float((lib or load()).oracle_accept_prob(H, h_acc, h_rej))


def expected_accepted(p: Sequence[float], k: int, lib=None) -> float:
    pa = _c(list(p) if len(p) else [0.0], np.float64)
    return float((lib or load()).oracle_expected_accepted(_p(pa, _f64p), k))


def step_efficiency(p: Sequence[float], k: int, c_draft: float, c_verify: float,
                    lib=None) -> float:
    pa = _c(list(p) if len(p) else [0.0], np.float64)
    return float((lib or load()).oracle_step_efficiency(_p(pa, _f64p), k, c_draft, c_verify))


def choose_k(p: Sequence[float], cands: Sequence[int], c_draft: float, c_verify: float,
             lib=None) -> int:
    pa = _c(list(p) if len(p) else [0.0], np.float64)
    ca = _c(list(cands), np.int32)
    return int((lib or load()).oracle_choose_k(_p(pa, _f64p), len(p), _p(ca, _i32p), len(ca),
                                                c_draft, c_verify))


def num_threads(lib=None) -> int:
    return int((lib or load()).oracle_num_threads())


def set_num_threads(n: int, lib=None) -> None:
    (lib or load()).oracle_set_num_threads(int(n))
