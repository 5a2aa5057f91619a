"""Python binding of the C-ABI library (argument marshalling only).

Each function takes torch tensors, checks their dtype/device/shape against
the layout the C ABI documents, and passes raw device pointers and the current
HIP stream through ctypes.  Every step of the computation runs in the HIP
kernels of ``libsparsespec_l.so``; there is no fallback: if the library is
missing, or a tensor is not on a GPU, the call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence, Tuple

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsparsespec_l.so")

SSL_OK = 0
SSL_ERR_NULL = -1
SSL_ERR_SHAPE = -2
SSL_ERR_UNSUPPORTED = -3
SSL_ERR_BUDGET = -4
SSL_ERR_ALIGN = -5
SSL_ERR_WORKSPACE = -6
SSL_ERR_HIP = -7

VERIFY_AUTO = 0
VERIFY_TWO_SWEEP = 1
VERIFY_ONE_SWEEP = 2
VERIFY_ONE_SWEEP_PERSISTENT = 3   # a schedule verify_plan reports, not a request

EXPORTED = [
    "ssl_status_string", "ssl_build_id", "ssl_exchange_status", "ssl_last_hip_error",
    "ssl_set_cu_budget",
    "ssl_test_exchange_faults", "ssl_index_count",
    "ssl_verify_workspace", "ssl_verify_plan", "ssl_verify_attn", "ssl_verify_attn_static",
    "ssl_select_workspace", "ssl_select_plan", "ssl_select_topb", "ssl_select_draft_workspace",
    "ssl_select_draft", "ssl_decode_step_workspace", "ssl_decode_step_plan", "ssl_decode_step",
    "ssl_draft_workspace", "ssl_draft_attn",
    "ssl_verify_attn_paged", "ssl_draft_attn_paged",
    "ssl_draft_materialize", "ssl_draft_step_workspace", "ssl_draft_step",
    "ssl_draft_materialize_paged", "ssl_draft_step_paged",
    "ssl_logit_stats_workspace", "ssl_logit_stats", "ssl_greedy_accept_workspace",
    "ssl_greedy_accept", "ssl_spec_accept_workspace", "ssl_spec_accept",
    "ssl_ctrl_create", "ssl_ctrl_destroy", "ssl_ctrl_observe", "ssl_ctrl_accept_prob",
    "ssl_ctrl_choose_k", "ssl_ctrl_get_state", "ssl_ctrl_set_state",
]


class Shape(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("max_ctx", ctypes.c_int32), ("max_q", ctypes.c_int32)]


class Params(ctypes.Structure):
    _fields_ = [("sm_scale", ctypes.c_float), ("window", ctypes.c_int32),
                ("k_sink", ctypes.c_int32), ("k_recent", ctypes.c_int32),
                ("budget", ctypes.c_int32), ("out_fp32", ctypes.c_int32),
                ("verify_mode", ctypes.c_int32), ("per_head", ctypes.c_int32)]


class SSLError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        msg = f"{where}: {status_string(status)} (status {status})"
        if status == SSL_ERR_HIP and _lib is not None:
            msg += f": {_lib.ssl_last_hip_error().decode()}"
        super().__init__(msg)


_lib = None
_i32p = ctypes.POINTER(ctypes.c_int32)
_f64p = ctypes.POINTER(ctypes.c_double)
_vp = ctypes.c_void_p
_sz = ctypes.c_size_t
_szp = ctypes.POINTER(ctypes.c_size_t)


def load(path: Optional[str] = None):
    """Load the HIP library.  Raises if it has not been built, or if it was
    built from sources other than the ones in this tree."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"{p} not found: build it with `python -m paper_2607_27735_amd.build`")
    lib = ctypes.CDLL(p)
    lib.ssl_build_id.argtypes = []
    lib.ssl_build_id.restype = ctypes.c_char_p
    if path is None:
        from .build import source_id
        built, tree = lib.ssl_build_id().decode(), source_id()
        if built != tree:
            raise RuntimeError(f"{p} was built from other sources (build id {built}, tree {tree}): "
                               "rebuild it with `python -m paper_2607_27735_amd.build`")
    sp, pp = ctypes.POINTER(Shape), ctypes.POINTER(Params)
    lib.ssl_status_string.argtypes = [ctypes.c_int]
    lib.ssl_status_string.restype = ctypes.c_char_p
    lib.ssl_last_hip_error.argtypes = []
    lib.ssl_last_hip_error.restype = ctypes.c_char_p
    lib.ssl_exchange_status.argtypes = [_vp, ctypes.POINTER(ctypes.c_uint32)]
    lib.ssl_exchange_status.restype = ctypes.c_int
    lib.ssl_set_cu_budget.argtypes = [ctypes.c_int32]
    lib.ssl_set_cu_budget.restype = ctypes.c_int
    lib.ssl_test_exchange_faults.argtypes = [ctypes.c_int32, ctypes.c_int32]
    lib.ssl_test_exchange_faults.restype = ctypes.c_int
    lib.ssl_index_count.argtypes = [ctypes.c_int32] * 4
    lib.ssl_index_count.restype = ctypes.c_int32
    lib.ssl_verify_workspace.argtypes = [sp, pp, _i32p, _i32p, _szp]
    lib.ssl_verify_attn.argtypes = [sp, pp, _i32p, _i32p, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]
    lib.ssl_verify_plan.argtypes = [sp, pp, _i32p, _i32p, _i32p, _i32p, _i32p]
    lib.ssl_verify_attn_static.argtypes = [sp, pp, _i32p, _i32p, _vp, _vp, _vp, _vp, _vp, _vp]
    lib.ssl_select_workspace.argtypes = [sp, pp, _i32p, _szp]
    lib.ssl_select_plan.argtypes = [sp, pp, _i32p, _i32p, _i32p, _i32p]
    lib.ssl_select_draft_workspace.argtypes = [sp, pp, _i32p, _szp]
    lib.ssl_select_draft.argtypes = [sp, pp, _i32p, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]
    lib.ssl_select_topb.argtypes = [sp, pp, _i32p, _vp, _vp, _vp, _vp, _sz, _vp]
    lib.ssl_decode_step_workspace.argtypes = [sp, pp, _i32p, _i32p, _szp]
    lib.ssl_decode_step_plan.argtypes = [sp, pp, _i32p, _i32p, _i32p]
    lib.ssl_decode_step.argtypes = [sp, pp, _i32p, _i32p] + [_vp] * 10 + [_sz, _vp]
    lib.ssl_draft_workspace.argtypes = [sp, pp, _i32p, _szp]
    lib.ssl_draft_attn.argtypes = [sp, pp, _i32p, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]
    lib.ssl_draft_materialize.argtypes = [sp, pp, _i32p, _vp, _vp, _vp, _vp, _vp, _vp]
    lib.ssl_draft_step_workspace.argtypes = [sp, pp, _i32p, _i32p, _szp]
    lib.ssl_draft_step.argtypes = [sp, pp, _i32p, _i32p, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                   _sz, _vp]
    _i32 = ctypes.c_int32
    lib.ssl_verify_attn_paged.argtypes = [sp, pp, _i32p, _i32p, _vp, _vp, _vp, _vp, _i32, _i32,
                                          _vp, _vp, _vp, _sz, _vp]
    lib.ssl_draft_attn_paged.argtypes = [sp, pp, _i32p, _vp, _vp, _vp, _vp, _i32, _i32, _vp, _vp,
                                         _vp, _sz, _vp]
    lib.ssl_draft_materialize_paged.argtypes = [sp, pp, _i32p, _vp, _vp, _vp, _i32, _i32, _vp,
                                                _vp, _vp, _vp]
    lib.ssl_draft_step_paged.argtypes = [sp, pp, _i32p, _i32p, _vp, _vp, _vp, _vp, _i32, _i32,
                                         _vp, _vp, _vp, _vp, _vp, _sz, _vp]
    lib.ssl_logit_stats_workspace.argtypes = [_i32, _i32, _szp]
    lib.ssl_logit_stats.argtypes = [_vp, _i32, _i32, _i32, _i32, _vp, _vp, _vp, _sz, _vp]
    lib.ssl_greedy_accept_workspace.argtypes = [_i32, _i32, _i32, _szp]
    lib.ssl_greedy_accept.argtypes = [_vp, _i32, _i32, _i32, _i32p, _i32, _i32, _vp, _vp, _vp,
                                      _vp, _sz, _vp]
    lib.ssl_spec_accept_workspace.argtypes = [_i32, _i32, _i32, _szp]
    lib.ssl_spec_accept.argtypes = [_vp, _vp, _i32, _i32, _i32, _i32p, _i32, _i32, _vp,
                                    ctypes.c_float, _vp, _vp, _vp, _vp, _vp, _sz, _vp]
    for f in ("ssl_verify_workspace", "ssl_verify_plan", "ssl_verify_attn",
              "ssl_verify_attn_static", "ssl_select_workspace",
              "ssl_select_topb", "ssl_select_plan", "ssl_select_draft_workspace",
              "ssl_select_draft", "ssl_draft_workspace", "ssl_draft_attn", "ssl_draft_materialize",
              "ssl_draft_step_workspace", "ssl_draft_step", "ssl_verify_attn_paged",
              "ssl_draft_attn_paged", "ssl_draft_materialize_paged", "ssl_draft_step_paged",
              "ssl_logit_stats_workspace",
              "ssl_logit_stats", "ssl_greedy_accept_workspace", "ssl_greedy_accept",
              "ssl_spec_accept_workspace", "ssl_spec_accept"):
        getattr(lib, f).restype = ctypes.c_int
    lib.ssl_ctrl_create.argtypes = [ctypes.c_double, _i32p, ctypes.c_int32, ctypes.c_int32]
    lib.ssl_ctrl_create.restype = _vp
    lib.ssl_ctrl_destroy.argtypes = [_vp]
    lib.ssl_ctrl_destroy.restype = None
    lib.ssl_ctrl_observe.argtypes = [_vp, _f64p, ctypes.c_int32, ctypes.c_int32]
    lib.ssl_ctrl_observe.restype = ctypes.c_int
    lib.ssl_ctrl_accept_prob.argtypes = [_vp, ctypes.c_double]
    lib.ssl_ctrl_accept_prob.restype = ctypes.c_double
    lib.ssl_ctrl_choose_k.argtypes = [_vp, _f64p, ctypes.c_int32, ctypes.c_double, ctypes.c_double]
    lib.ssl_ctrl_choose_k.restype = ctypes.c_int32
    lib.ssl_ctrl_get_state.argtypes = [_vp, _f64p]
    lib.ssl_ctrl_get_state.restype = ctypes.c_int
    lib.ssl_ctrl_set_state.argtypes = [_vp, _f64p]
    lib.ssl_ctrl_set_state.restype = ctypes.c_int
    if path is None:
        _lib = lib
    return lib


def status_string(status: int) -> str:
    return load().ssl_status_string(int(status)).decode()


def build_id() -> str:
    return load().ssl_build_id().decode()


EXCHANGE_VERIFY, EXCHANGE_SELECT, EXCHANGE_DRAFT, EXCHANGE_LOGITS = 1, 2, 4, 8


def exchange_status(stream=None) -> int:
    """Reads and clears the current device's exchange status bits (waits for
    the stream)."""
    flags = ctypes.c_uint32(0)
    _check(load().ssl_exchange_status(_stream(stream), ctypes.byref(flags)), "ssl_exchange_status")
    return int(flags.value)


def set_cu_budget(n_cu: int) -> None:
    """CU count the verify and select plans count on (0: the device's own)."""
    _check(load().ssl_set_cu_budget(int(n_cu)), "ssl_set_cu_budget")


def test_exchange_faults(spin_limit: int = 0, mismatch_tags: bool = False) -> None:
    """Testing only: bound exchange waits to spin_limit polls and make every
    published tag unacceptable (see the header)."""
    _check(load().ssl_test_exchange_faults(int(spin_limit), 1 if mismatch_tags else 0),
           "ssl_test_exchange_faults")


def _check(status: int, where: str) -> None:
    if status != SSL_OK:
        raise SSLError(status, where)


def _host_i32(x) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(x, dtype=np.int32).reshape(-1))


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _need_gpu(*ts: torch.Tensor) -> None:
    for t in ts:
        if not t.is_cuda:
            raise RuntimeError("the HIP path needs GPU tensors; there is no CPU fallback")
        if not t.is_contiguous():
            raise RuntimeError("tensors must be contiguous")


def make_params(sm_scale: float, window: int = 16, k_sink: int = 4, k_recent: int = 32,
                budget: int = 2048, out_fp32: bool = False, verify_mode: int = VERIFY_AUTO,
                per_head: bool = False) -> Params:
    return Params(float(sm_scale), int(window), int(k_sink), int(k_recent), int(budget),
                  1 if out_fp32 else 0, int(verify_mode), 1 if per_head else 0)


def index_count(T: int, k_sink: int, k_recent: int, budget: int) -> int:
    return int(load().ssl_index_count(T, k_sink, k_recent, budget))


# ---------------------------------------------------------------------------
# verify
# ---------------------------------------------------------------------------

def verify_shape(q: torch.Tensor, k: torch.Tensor) -> Shape:
    batch, max_q, hq, d = q.shape
    b2, hkv, max_ctx, d2 = k.shape
    return Shape(batch, hq, hkv, d, max_ctx, max_q)


def verify_workspace_bytes(shape: Shape, params: Params, ctx_len, q_len) -> int:
    ctx, ql = _host_i32(ctx_len), _host_i32(q_len)
    n = ctypes.c_size_t(0)
    _check(load().ssl_verify_workspace(ctypes.byref(shape), ctypes.byref(params),
                                       ctx.ctypes.data_as(_i32p), ql.ctypes.data_as(_i32p),
                                       ctypes.byref(n)), "ssl_verify_workspace")
    return int(n.value)


def verify_plan(shape: Shape, params: Params, ctx_len, q_len) -> Tuple[int, int, int]:
    """(schedule, keys per item, items) that verify_attn would use."""
    ctx, ql = _host_i32(ctx_len), _host_i32(q_len)
    sch, ch, it = ctypes.c_int32(0), ctypes.c_int32(0), ctypes.c_int32(0)
    _check(load().ssl_verify_plan(ctypes.byref(shape), ctypes.byref(params),
                                  ctx.ctypes.data_as(_i32p), ql.ctypes.data_as(_i32p),
                                  ctypes.byref(sch), ctypes.byref(ch), ctypes.byref(it)),
           "ssl_verify_plan")
    return int(sch.value), int(ch.value), int(it.value)


def verify_attn(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, ctx_len, q_len,
                params: Params, out: Optional[torch.Tensor] = None,
                scores: Optional[torch.Tensor] = None,
                workspace: Optional[torch.Tensor] = None, stream=None
                ) -> Tuple[torch.Tensor, torch.Tensor]:
    """Verify attention + Eq. 3 scores.  q [B, max_q, Hq, 128] bf16, k/v
    [B, Hkv, max_ctx, 128] bf16; returns (out, scores)."""
    _need_gpu(q, k, v)
    if q.dtype != torch.bfloat16 or k.dtype != torch.bfloat16 or v.dtype != torch.bfloat16:
        raise TypeError("q, k, v must be bfloat16")
    if k.shape != v.shape or q.shape[0] != k.shape[0] or q.shape[3] != k.shape[3]:
        raise ValueError("q/k/v shapes disagree")
    shape = verify_shape(q, k)
    ctx, ql = _host_i32(ctx_len), _host_i32(q_len)
    if len(ctx) != shape.batch or len(ql) != shape.batch:
        raise ValueError("ctx_len / q_len need one entry per sequence")
    odt = torch.float32 if params.out_fp32 else torch.bfloat16
    if out is None:
        out = torch.zeros(q.shape, dtype=odt, device=q.device)
    heads = shape.n_q_heads if params.per_head else shape.n_kv_heads   # score rows per sequence
    if scores is None:
        scores = torch.zeros((shape.batch, heads, shape.max_ctx), dtype=torch.float32,
                             device=q.device)
    _need_gpu(out, scores)
    if out.dtype != odt or scores.dtype != torch.float32:
        raise TypeError("out dtype must match params.out_fp32; scores must be float32")
    if out.shape != q.shape or scores.shape != (shape.batch, heads, shape.max_ctx):
        raise ValueError("out/scores shape")
    need = verify_workspace_bytes(shape, params, ctx, ql)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=q.device)
    _check(load().ssl_verify_attn(ctypes.byref(shape), ctypes.byref(params),
                                  ctx.ctypes.data_as(_i32p), ql.ctypes.data_as(_i32p),
                                  _ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(scores),
                                  _ptr(workspace), workspace.numel(), _stream(stream)),
           "ssl_verify_attn")
    return out, scores


def verify_attn_static(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, ctx_len, q_len,
                       params: Params, out: torch.Tensor, scores: torch.Tensor,
                       stream=None) -> None:
    """ssl_verify_attn_static: verify attention into caller-given ``out`` and
    ``scores`` with the library's own device scratch as the workspace (no
    allocation anywhere in the call)."""
    _need_gpu(q, k, v, out, scores)
    if q.dtype != torch.bfloat16 or k.dtype != torch.bfloat16 or v.dtype != torch.bfloat16:
        raise TypeError("q, k, v must be bfloat16")
    shape = verify_shape(q, k)
    ctx, ql = _host_i32(ctx_len), _host_i32(q_len)
    _check(load().ssl_verify_attn_static(ctypes.byref(shape), ctypes.byref(params),
                                         ctx.ctypes.data_as(_i32p), ql.ctypes.data_as(_i32p),
                                         _ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(scores),
                                         _stream(stream)),
           "ssl_verify_attn_static")


# ---------------------------------------------------------------------------
# select
# ---------------------------------------------------------------------------

def select_topb(scores: torch.Tensor, ctx_len, params: Params, n_q_heads: Optional[int] = None,
                idx: Optional[torch.Tensor] = None, n_idx: Optional[torch.Tensor] = None,
                stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Eq. 4 index sets from scores [B, Hkv, max_ctx] fp32; returns (idx, n_idx)
    with idx [B, Hkv, budget] int32 (slots past n_idx[b] untouched)."""
    _need_gpu(scores)
    if scores.dtype != torch.float32:
        raise TypeError("scores must be float32")
    batch, hkv, max_ctx = scores.shape
    shape = Shape(batch, n_q_heads or hkv, hkv, 128, max_ctx, 1)
    ctx = _host_i32(ctx_len)
    if idx is None:
        idx = torch.full((batch, hkv, params.budget), -1, dtype=torch.int32, device=scores.device)
    if n_idx is None:
        n_idx = torch.zeros(batch, dtype=torch.int32, device=scores.device)
    _need_gpu(idx, n_idx)
    if idx.shape != (batch, hkv, params.budget) or idx.dtype != torch.int32:
        raise ValueError("idx must be int32 [batch, n_kv_heads, budget]")
    ws = torch.empty(max(select_workspace_bytes(shape, params, ctx), 1), dtype=torch.uint8,
                     device=scores.device)
    _check(load().ssl_select_topb(ctypes.byref(shape), ctypes.byref(params),
                                  ctx.ctypes.data_as(_i32p), _ptr(scores), _ptr(idx),
                                  _ptr(n_idx), _ptr(ws), ws.numel(), _stream(stream)),
           "ssl_select_topb")
    return idx, n_idx


def select_plan(shape: Shape, params: Params, ctx_len) -> Tuple[bool, int, int]:
    """(one kernel?, positions per partition, partitions) that select_topb would use."""
    ctx = _host_i32(ctx_len)
    one, part, parts = ctypes.c_int32(0), ctypes.c_int32(0), ctypes.c_int32(0)
    _check(load().ssl_select_plan(ctypes.byref(shape), ctypes.byref(params),
                                  ctx.ctypes.data_as(_i32p), ctypes.byref(one), ctypes.byref(part),
                                  ctypes.byref(parts)), "ssl_select_plan")
    return bool(one.value), int(part.value), int(parts.value)


def select_workspace_bytes(shape: Shape, params: Params, ctx_len) -> int:
    ctx = _host_i32(ctx_len)
    n = ctypes.c_size_t(0)
    _check(load().ssl_select_workspace(ctypes.byref(shape), ctypes.byref(params),
                                       ctx.ctypes.data_as(_i32p), ctypes.byref(n)),
           "ssl_select_workspace")
    return int(n.value)


def select_draft_workspace_bytes(shape: Shape, params: Params, ctx_len) -> int:
    ctx = _host_i32(ctx_len)
    n = ctypes.c_size_t(0)
    _check(load().ssl_select_draft_workspace(ctypes.byref(shape), ctypes.byref(params),
                                             ctx.ctypes.data_as(_i32p), ctypes.byref(n)),
           "ssl_select_draft_workspace")
    return int(n.value)


def select_draft(scores: torch.Tensor, ctx_len, params: Params, q_draft: torch.Tensor,
                 k: torch.Tensor, v: torch.Tensor, idx: Optional[torch.Tensor] = None,
                 n_idx: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None,
                 workspace: Optional[torch.Tensor] = None, stream=None):
    """Eq. 4 index sets and the first Eq. 5 draft step over them in one call;
    returns (idx, n_idx, out)."""
    _need_gpu(scores, q_draft, k, v)
    if scores.dtype != torch.float32:
        raise TypeError("scores must be float32")
    batch, hq, d = q_draft.shape
    _, hkv, max_ctx, _ = k.shape
    units = hq if params.per_head else hkv
    if tuple(scores.shape) != (batch, units, max_ctx):
        raise ValueError("scores must be [batch, units, max_ctx]")
    shape = Shape(batch, hq, hkv, d, max_ctx, 1)
    ctx = _host_i32(ctx_len)
    if idx is None:
        idx = torch.empty((batch, units, params.budget), dtype=torch.int32, device=scores.device)
    if n_idx is None:
        n_idx = torch.empty(batch, dtype=torch.int32, device=scores.device)
    odt = torch.float32 if params.out_fp32 else torch.bfloat16
    if out is None:
        out = torch.empty(q_draft.shape, dtype=odt, device=q_draft.device)
    _need_gpu(idx, n_idx, out)
    need = select_draft_workspace_bytes(shape, params, ctx)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=scores.device)
    _check(load().ssl_select_draft(ctypes.byref(shape), ctypes.byref(params),
                                   ctx.ctypes.data_as(_i32p), _ptr(scores), _ptr(idx), _ptr(n_idx),
                                   _ptr(q_draft), _ptr(k), _ptr(v), _ptr(out), _ptr(workspace),
                                   workspace.numel(), _stream(stream)),
           "ssl_select_draft")
    return idx, n_idx, out


# ---------------------------------------------------------------------------
# the whole decode step
# ---------------------------------------------------------------------------

def decode_step_workspace_bytes(shape: Shape, params: Params, ctx_len, q_len) -> int:
    ctx, ql = _host_i32(ctx_len), _host_i32(q_len)
    n = ctypes.c_size_t(0)
    _check(load().ssl_decode_step_workspace(ctypes.byref(shape), ctypes.byref(params),
                                            ctx.ctypes.data_as(_i32p), ql.ctypes.data_as(_i32p),
                                            ctypes.byref(n)), "ssl_decode_step_workspace")
    return int(n.value)


def decode_step_plan(shape: Shape, params: Params, ctx_len, q_len) -> bool:
    """Whether decode_step runs as one kernel."""
    ctx, ql = _host_i32(ctx_len), _host_i32(q_len)
    one = ctypes.c_int32(0)
    _check(load().ssl_decode_step_plan(ctypes.byref(shape), ctypes.byref(params),
                                       ctx.ctypes.data_as(_i32p), ql.ctypes.data_as(_i32p),
                                       ctypes.byref(one)), "ssl_decode_step_plan")
    return bool(one.value)


def decode_step(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, q_draft: torch.Tensor, ctx_len,
                q_len, params: Params, out: Optional[torch.Tensor] = None,
                scores: Optional[torch.Tensor] = None, idx: Optional[torch.Tensor] = None,
                n_idx: Optional[torch.Tensor] = None, draft_out: Optional[torch.Tensor] = None,
                workspace: Optional[torch.Tensor] = None, stream=None):
    """Verify (+ Eq. 3 scores), Eq. 4 select and the first Eq. 5 draft step
    in one call; returns (out, scores, idx, n_idx, draft_out)."""
    _need_gpu(q, k, v, q_draft)
    if any(t.dtype != torch.bfloat16 for t in (q, k, v, q_draft)):
        raise TypeError("q, k, v, q_draft must be bfloat16")
    if k.shape != v.shape or q.shape[0] != k.shape[0] or q.shape[3] != k.shape[3]:
        raise ValueError("q/k/v shapes disagree")
    shape = verify_shape(q, k)
    if tuple(q_draft.shape) != (shape.batch, shape.n_q_heads, shape.head_dim):
        raise ValueError("q_draft must be [batch, n_q_heads, 128]")
    ctx, ql = _host_i32(ctx_len), _host_i32(q_len)
    if len(ctx) != shape.batch or len(ql) != shape.batch:
        raise ValueError("ctx_len / q_len need one entry per sequence")
    units = shape.n_q_heads if params.per_head else shape.n_kv_heads   # score rows, index sets
    dev = q.device
    odt = torch.float32 if params.out_fp32 else torch.bfloat16
    if out is None:
        out = torch.zeros(q.shape, dtype=odt, device=dev)
    if scores is None:
        scores = torch.zeros((shape.batch, units, shape.max_ctx), dtype=torch.float32, device=dev)
    if idx is None:
        idx = torch.empty((shape.batch, units, params.budget), dtype=torch.int32, device=dev)
    if n_idx is None:
        n_idx = torch.empty(shape.batch, dtype=torch.int32, device=dev)
    if draft_out is None:
        draft_out = torch.empty(q_draft.shape, dtype=odt, device=dev)
    _need_gpu(out, scores, idx, n_idx, draft_out)
    if out.dtype != odt or draft_out.dtype != odt or scores.dtype != torch.float32:
        raise TypeError("out/draft_out dtype must match params.out_fp32; scores must be float32")
    if idx.dtype != torch.int32 or n_idx.dtype != torch.int32:
        raise TypeError("idx and n_idx must be int32")
    if (out.shape != q.shape or draft_out.shape != q_draft.shape
            or scores.shape != (shape.batch, units, shape.max_ctx)
            or idx.shape != (shape.batch, units, params.budget)
            or n_idx.shape != (shape.batch,)):
        raise ValueError("output shapes")
    need = decode_step_workspace_bytes(shape, params, ctx, ql)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    _check(load().ssl_decode_step(ctypes.byref(shape), ctypes.byref(params),
                                  ctx.ctypes.data_as(_i32p), ql.ctypes.data_as(_i32p), _ptr(q),
                                  _ptr(k), _ptr(v), _ptr(out), _ptr(scores), _ptr(idx),
                                  _ptr(n_idx), _ptr(q_draft), _ptr(draft_out), _ptr(workspace),
                                  workspace.numel(), _stream(stream)),
           "ssl_decode_step")
    return out, scores, idx, n_idx, draft_out


# ---------------------------------------------------------------------------
# draft
# ---------------------------------------------------------------------------

def draft_workspace_bytes(shape: Shape, params: Params, n_idx_host) -> int:
    n_idx = _host_i32(n_idx_host)
    n = ctypes.c_size_t(0)
    _check(load().ssl_draft_workspace(ctypes.byref(shape), ctypes.byref(params),
                                      n_idx.ctypes.data_as(_i32p), ctypes.byref(n)),
           "ssl_draft_workspace")
    return int(n.value)


def draft_attn(q_draft: torch.Tensor, k: torch.Tensor, v: torch.Tensor, idx: torch.Tensor,
               n_idx_host, params: Params, out: Optional[torch.Tensor] = None,
               workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Eq. 5 draft attention.  q_draft [B, Hq, 128] bf16; idx [B, Hkv, budget]
    int32; n_idx_host: per-sequence index counts on the host."""
    _need_gpu(q_draft, k, v, idx)
    if q_draft.dtype != torch.bfloat16 or k.dtype != torch.bfloat16 or v.dtype != torch.bfloat16:
        raise TypeError("q_draft, k, v must be bfloat16")
    if idx.dtype != torch.int32:
        raise TypeError("idx must be int32")
    batch, hq, d = q_draft.shape
    _, hkv, max_ctx, _ = k.shape
    shape = Shape(batch, hq, hkv, d, max_ctx, 1)
    units = hq if params.per_head else hkv
    if idx.shape != (batch, units, params.budget):
        raise ValueError("idx must be [batch, n_kv_heads (n_q_heads if per_head), budget]")
    n_idx = _host_i32(n_idx_host)
    odt = torch.float32 if params.out_fp32 else torch.bfloat16
    if out is None:
        out = torch.zeros(q_draft.shape, dtype=odt, device=q_draft.device)
    _need_gpu(out)
    need = draft_workspace_bytes(shape, params, n_idx)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=q_draft.device)
    _check(load().ssl_draft_attn(ctypes.byref(shape), ctypes.byref(params),
                                 n_idx.ctypes.data_as(_i32p), _ptr(q_draft), _ptr(k), _ptr(v),
                                 _ptr(idx), _ptr(out), _ptr(workspace), workspace.numel(),
                                 _stream(stream)), "ssl_draft_attn")
    return out


# ---------------------------------------------------------------------------
# paged KV cache
# ---------------------------------------------------------------------------

def verify_attn_paged(q: torch.Tensor, k_pages: torch.Tensor, v_pages: torch.Tensor,
                      block_table: torch.Tensor, max_ctx: int, ctx_len, q_len, params: Params,
                      out: Optional[torch.Tensor] = None, scores: Optional[torch.Tensor] = None,
                      workspace: Optional[torch.Tensor] = None, stream=None
                      ) -> Tuple[torch.Tensor, torch.Tensor]:
    """Verify attention + Eq. 3 scores over a paged cache: k_pages / v_pages
    [n_pages, Hkv, page_size, 128] bf16, block_table [B, max_blocks] int32;
    scores are [B, Hkv, max_ctx]."""
    _need_gpu(q, k_pages, v_pages, block_table)
    if q.dtype != torch.bfloat16 or k_pages.dtype != torch.bfloat16 or \
            v_pages.dtype != torch.bfloat16:
        raise TypeError("q, k_pages, v_pages must be bfloat16")
    if block_table.dtype != torch.int32 or block_table.dim() != 2 or \
            block_table.shape[0] != q.shape[0]:
        raise ValueError("block_table must be int32 [batch, max_blocks]")
    _, hkv, page, d = k_pages.shape
    batch, max_q, hq, _ = q.shape
    shape = Shape(batch, hq, hkv, d, max_ctx, max_q)
    ctx, ql = _host_i32(ctx_len), _host_i32(q_len)
    odt = torch.float32 if params.out_fp32 else torch.bfloat16
    if out is None:
        out = torch.zeros(q.shape, dtype=odt, device=q.device)
    if scores is None:
        scores = torch.zeros((batch, hq if params.per_head else hkv, max_ctx), dtype=torch.float32, device=q.device)
    _need_gpu(out, scores)
    need = verify_workspace_bytes(shape, params, ctx, ql)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=q.device)
    _check(load().ssl_verify_attn_paged(ctypes.byref(shape), ctypes.byref(params),
                                        ctx.ctypes.data_as(_i32p), ql.ctypes.data_as(_i32p),
                                        _ptr(q), _ptr(k_pages), _ptr(v_pages), _ptr(block_table),
                                        page, block_table.shape[1], _ptr(out), _ptr(scores),
                                        _ptr(workspace), workspace.numel(), _stream(stream)),
           "ssl_verify_attn_paged")
    return out, scores


def draft_attn_paged(q_draft: torch.Tensor, k_pages: torch.Tensor, v_pages: torch.Tensor,
                     block_table: torch.Tensor, max_ctx: int, idx: torch.Tensor, n_idx_host,
                     params: Params, out: Optional[torch.Tensor] = None,
                     workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Eq. 5 draft attention over a paged cache (layouts as verify_attn_paged)."""
    _need_gpu(q_draft, k_pages, v_pages, block_table, idx)
    batch, hq, d = q_draft.shape
    _, hkv, page, _ = k_pages.shape
    units = hq if params.per_head else hkv
    if idx.dtype != torch.int32 or idx.shape != (batch, units, params.budget):
        raise ValueError("idx must be int32 [batch, n_kv_heads (n_q_heads if per_head), budget]")
    shape = Shape(batch, hq, hkv, d, max_ctx, 1)
    n_idx = _host_i32(n_idx_host)
    odt = torch.float32 if params.out_fp32 else torch.bfloat16
    if out is None:
        out = torch.zeros(q_draft.shape, dtype=odt, device=q_draft.device)
    _need_gpu(out)
    need = draft_workspace_bytes(shape, params, n_idx)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=q_draft.device)
    _check(load().ssl_draft_attn_paged(ctypes.byref(shape), ctypes.byref(params),
                                       n_idx.ctypes.data_as(_i32p), _ptr(q_draft), _ptr(k_pages),
                                       _ptr(v_pages), _ptr(block_table), page,
                                       block_table.shape[1], _ptr(idx), _ptr(out),
                                       _ptr(workspace), workspace.numel(), _stream(stream)),
           "ssl_draft_attn_paged")
    return out


# ---------------------------------------------------------------------------
# draft round
# ---------------------------------------------------------------------------

def draft_materialize(k: torch.Tensor, v: torch.Tensor, idx: torch.Tensor, ctx_len_host,
                      params: Params, k_sel: Optional[torch.Tensor] = None,
                      v_sel: Optional[torch.Tensor] = None, stream=None,
                      n_q_heads: Optional[int] = None):
    """Copy the sink and TopK rows of the index sets built at ``ctx_len_host``
    to ``k_sel`` / ``v_sel`` [B, units, budget, 128] bf16 (allocated if None;
    units = Hkv, or Hq with ``params.per_head``, which needs ``n_q_heads``);
    returns them."""
    _need_gpu(k, v, idx)
    if k.dtype != torch.bfloat16 or v.dtype != torch.bfloat16:
        raise TypeError("k, v must be bfloat16")
    if idx.dtype != torch.int32:
        raise TypeError("idx must be int32")
    batch, hkv, max_ctx, d = k.shape
    hq = hkv if n_q_heads is None else int(n_q_heads)
    units = hq if params.per_head else hkv
    if idx.shape != (batch, units, params.budget):
        raise ValueError("idx must be [batch, units, budget]")
    shape = Shape(batch, hq, hkv, d, max_ctx, 1)
    sel_shape = (batch, units, params.budget, d)
    if k_sel is None:
        k_sel = torch.empty(sel_shape, dtype=torch.bfloat16, device=k.device)
    if v_sel is None:
        v_sel = torch.empty(sel_shape, dtype=torch.bfloat16, device=k.device)
    if tuple(k_sel.shape) != sel_shape or tuple(v_sel.shape) != sel_shape:
        raise ValueError("k_sel / v_sel must be [batch, units, budget, 128]")
    _need_gpu(k_sel, v_sel)
    ctx = _host_i32(ctx_len_host)
    _check(load().ssl_draft_materialize(ctypes.byref(shape), ctypes.byref(params),
                                        ctx.ctypes.data_as(_i32p), _ptr(k), _ptr(v), _ptr(idx),
                                        _ptr(k_sel), _ptr(v_sel), _stream(stream)),
           "ssl_draft_materialize")
    return k_sel, v_sel


def draft_step_workspace_bytes(shape: Shape, params: Params, ctx_len_host, cur_len_host) -> int:
    ctx, cur = _host_i32(ctx_len_host), _host_i32(cur_len_host)
    n = ctypes.c_size_t(0)
    _check(load().ssl_draft_step_workspace(ctypes.byref(shape), ctypes.byref(params),
                                           ctx.ctypes.data_as(_i32p), cur.ctypes.data_as(_i32p),
                                           ctypes.byref(n)), "ssl_draft_step_workspace")
    return int(n.value)


def draft_step(q_draft: torch.Tensor, k: torch.Tensor, v: torch.Tensor, ctx_len_host,
               cur_len_host, params: Params, idx: Optional[torch.Tensor] = None,
               k_sel: Optional[torch.Tensor] = None, v_sel: Optional[torch.Tensor] = None,
               out: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
               stream=None) -> torch.Tensor:
    """One draft-round step at lengths ``cur_len_host`` over the sink and TopK
    rows of the index sets built at ``ctx_len_host`` (through ``idx``, or the
    materialized ``k_sel`` / ``v_sel``) and the slid recent window."""
    _need_gpu(q_draft, k, v)
    if q_draft.dtype != torch.bfloat16 or k.dtype != torch.bfloat16 or v.dtype != torch.bfloat16:
        raise TypeError("q_draft, k, v must be bfloat16")
    batch, hq, d = q_draft.shape
    _, hkv, max_ctx, _ = k.shape
    units = hq if params.per_head else hkv
    if k_sel is not None or v_sel is not None:
        if k_sel is None or v_sel is None:
            raise ValueError("give both k_sel and v_sel, or neither")
        _need_gpu(k_sel, v_sel)
        if tuple(k_sel.shape) != (batch, units, params.budget, d) or k_sel.shape != v_sel.shape:
            raise ValueError("k_sel / v_sel must be [batch, units, budget, 128]")
    else:
        if idx is None:
            raise ValueError("idx is needed when no materialized rows are given")
        _need_gpu(idx)
        if idx.shape != (batch, units, params.budget) or idx.dtype != torch.int32:
            raise ValueError("idx must be int32 [batch, units, budget]")
    shape = Shape(batch, hq, hkv, d, max_ctx, 1)
    ctx, cur = _host_i32(ctx_len_host), _host_i32(cur_len_host)
    odt = torch.float32 if params.out_fp32 else torch.bfloat16
    if out is None:
        out = torch.zeros(q_draft.shape, dtype=odt, device=q_draft.device)
    _need_gpu(out)
    need = draft_step_workspace_bytes(shape, params, ctx, cur)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=q_draft.device)
    _check(load().ssl_draft_step(ctypes.byref(shape), ctypes.byref(params),
                                 ctx.ctypes.data_as(_i32p), cur.ctypes.data_as(_i32p),
                                 _ptr(q_draft), _ptr(k), _ptr(v), _ptr(idx), _ptr(k_sel),
                                 _ptr(v_sel), _ptr(out), _ptr(workspace), workspace.numel(),
                                 _stream(stream)),
           "ssl_draft_step")
    return out


def draft_materialize_paged(k_pages: torch.Tensor, v_pages: torch.Tensor,
                            block_table: torch.Tensor, max_ctx: int, idx: torch.Tensor,
                            ctx_len_host, params: Params, k_sel: Optional[torch.Tensor] = None,
                            v_sel: Optional[torch.Tensor] = None, stream=None,
                            n_q_heads: Optional[int] = None):
    """draft_materialize over a paged cache (k_pages / v_pages [n_pages, Hkv,
    page_size, 128] bf16, block_table [B, max_blocks] int32); k_sel / v_sel
    stay dense [B, units, budget, 128]."""
    _need_gpu(k_pages, v_pages, block_table, idx)
    if k_pages.dtype != torch.bfloat16 or v_pages.dtype != torch.bfloat16:
        raise TypeError("k_pages, v_pages must be bfloat16")
    if block_table.dtype != torch.int32 or block_table.dim() != 2:
        raise ValueError("block_table must be int32 [batch, max_blocks]")
    _, hkv, page, d = k_pages.shape
    batch = block_table.shape[0]
    hq = hkv if n_q_heads is None else int(n_q_heads)
    units = hq if params.per_head else hkv
    if idx.dtype != torch.int32 or idx.shape != (batch, units, params.budget):
        raise ValueError("idx must be int32 [batch, units, budget]")
    shape = Shape(batch, hq, hkv, d, int(max_ctx), 1)
    sel_shape = (batch, units, params.budget, d)
    if k_sel is None:
        k_sel = torch.empty(sel_shape, dtype=torch.bfloat16, device=k_pages.device)
    if v_sel is None:
        v_sel = torch.empty(sel_shape, dtype=torch.bfloat16, device=k_pages.device)
    if tuple(k_sel.shape) != sel_shape or tuple(v_sel.shape) != sel_shape:
        raise ValueError("k_sel / v_sel must be [batch, units, budget, 128]")
    _need_gpu(k_sel, v_sel)
    ctx = _host_i32(ctx_len_host)
    _check(load().ssl_draft_materialize_paged(ctypes.byref(shape), ctypes.byref(params),
                                              ctx.ctypes.data_as(_i32p), _ptr(k_pages),
                                              _ptr(v_pages), _ptr(block_table), int(page),
                                              int(block_table.shape[1]), _ptr(idx), _ptr(k_sel),
                                              _ptr(v_sel), _stream(stream)),
           "ssl_draft_materialize_paged")
    return k_sel, v_sel


def draft_step_paged(q_draft: torch.Tensor, k_pages: torch.Tensor, v_pages: torch.Tensor,
                     block_table: torch.Tensor, max_ctx: int, ctx_len_host, cur_len_host,
                     params: Params, idx: Optional[torch.Tensor] = None,
                     k_sel: Optional[torch.Tensor] = None, v_sel: Optional[torch.Tensor] = None,
                     out: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                     stream=None) -> torch.Tensor:
    """draft_step over a paged cache (layouts as draft_materialize_paged)."""
    _need_gpu(q_draft, k_pages, v_pages, block_table)
    if any(t.dtype != torch.bfloat16 for t in (q_draft, k_pages, v_pages)):
        raise TypeError("q_draft, k_pages, v_pages must be bfloat16")
    if block_table.dtype != torch.int32 or block_table.dim() != 2:
        raise ValueError("block_table must be int32 [batch, max_blocks]")
    batch, hq, d = q_draft.shape
    _, hkv, page, _ = k_pages.shape
    units = hq if params.per_head else hkv
    if (k_sel is None) != (v_sel is None):
        raise ValueError("give both k_sel and v_sel, or neither")
    if k_sel is None and (idx is None or idx.dtype != torch.int32
                          or idx.shape != (batch, units, params.budget)):
        raise ValueError("idx must be int32 [batch, units, budget] when no materialized rows are given")
    shape = Shape(batch, hq, hkv, d, int(max_ctx), 1)
    ctx, cur = _host_i32(ctx_len_host), _host_i32(cur_len_host)
    odt = torch.float32 if params.out_fp32 else torch.bfloat16
    if out is None:
        out = torch.zeros(q_draft.shape, dtype=odt, device=q_draft.device)
    _need_gpu(out)
    need = draft_step_workspace_bytes(shape, params, ctx, cur)
    if workspace is None or workspace.numel() < need:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=q_draft.device)
    _check(load().ssl_draft_step_paged(ctypes.byref(shape), ctypes.byref(params),
                                       ctx.ctypes.data_as(_i32p), cur.ctypes.data_as(_i32p),
                                       _ptr(q_draft), _ptr(k_pages), _ptr(v_pages),
                                       _ptr(block_table), int(page), int(block_table.shape[1]),
                                       _ptr(idx), _ptr(k_sel), _ptr(v_sel), _ptr(out),
                                       _ptr(workspace), workspace.numel(), _stream(stream)),
           "ssl_draft_step_paged")
    return out


# ---------------------------------------------------------------------------
# token statistics of logit rows
# ---------------------------------------------------------------------------

SSL_DT_BF16 = 0
SSL_DT_F32 = 1


def _logit_dtype(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return SSL_DT_BF16
    if t.dtype == torch.float32:
        return SSL_DT_F32
    raise TypeError("logits must be bfloat16 or float32")


def logit_stats(logits: torch.Tensor, vocab: Optional[int] = None, entropy: bool = True,
                argmax: bool = True, stream=None):
    """Per-row entropy (nats, fp32) and argmax (int32, lowest index on ties) of
    logits [n_rows, row_stride] (rows contiguous); returns (entropy, argmax),
    None for an output not asked for."""
    _need_gpu(logits)
    n_rows, stride = logits.shape
    if logits.stride(1) != 1 or logits.stride(0) != stride:
        raise ValueError("logits must be contiguous [n_rows, row_stride]")
    V = stride if vocab is None else vocab
    ent = torch.empty(n_rows, dtype=torch.float32, device=logits.device) if entropy else None
    am = torch.empty(n_rows, dtype=torch.int32, device=logits.device) if argmax else None
    n = ctypes.c_size_t(0)
    _check(load().ssl_logit_stats_workspace(n_rows, V, ctypes.byref(n)), "ssl_logit_stats_workspace")
    ws = torch.empty(max(int(n.value), 1), dtype=torch.uint8, device=logits.device)
    _check(load().ssl_logit_stats(_ptr(logits), _logit_dtype(logits), n_rows, V, stride, _ptr(ent),
                                  _ptr(am), _ptr(ws), ws.numel(), _stream(stream)),
           "ssl_logit_stats")
    return ent, am


def greedy_accept(logits: torch.Tensor, draft_tokens: torch.Tensor, k_len_host,
                  vocab: Optional[int] = None, stream=None):
    """Greedy verification: logits [batch, max_k + 1, row_stride], draft_tokens
    [batch, max_k] int32, k_len_host per sequence; returns (n_accepted,
    next_token) int32 [batch]."""
    _need_gpu(logits, draft_tokens)
    batch, rows, stride = logits.shape
    max_k = rows - 1
    if not logits.is_contiguous():
        raise ValueError("logits must be contiguous [batch, max_k + 1, row_stride]")
    if draft_tokens.dtype != torch.int32 or tuple(draft_tokens.shape) != (batch, max_k):
        raise ValueError("draft_tokens must be int32 [batch, max_k]")
    V = stride if vocab is None else vocab
    kl = _host_i32(k_len_host)
    m = torch.empty(batch, dtype=torch.int32, device=logits.device)
    nxt = torch.empty(batch, dtype=torch.int32, device=logits.device)
    n = ctypes.c_size_t(0)
    _check(load().ssl_greedy_accept_workspace(batch, max_k, V, ctypes.byref(n)),
           "ssl_greedy_accept_workspace")
    ws = torch.empty(max(int(n.value), 1), dtype=torch.uint8, device=logits.device)
    _check(load().ssl_greedy_accept(_ptr(logits), _logit_dtype(logits), batch, max_k,
                                    kl.ctypes.data_as(_i32p), V, stride, _ptr(draft_tokens),
                                    _ptr(m), _ptr(nxt), _ptr(ws), ws.numel(), _stream(stream)),
           "ssl_greedy_accept")
    return m, nxt


def spec_accept(target_logits: torch.Tensor, draft_logits: torch.Tensor,
                draft_tokens: torch.Tensor, k_len_host, temperature: float,
                u_accept: torch.Tensor, u_sample: torch.Tensor, vocab: Optional[int] = None,
                stream=None):
    """Speculative sampling: target_logits [batch, max_k + 1, row_stride],
    draft_logits [batch, max_k, row_stride] (same dtype), draft_tokens
    [batch, max_k] int32, u_accept [batch, max_k] and u_sample [batch] float32
    uniforms in [0, 1); returns (n_accepted, next_token) int32 [batch]."""
    _need_gpu(target_logits, draft_logits, draft_tokens, u_accept, u_sample)
    batch, rows, stride = target_logits.shape
    max_k = rows - 1
    if not target_logits.is_contiguous() or not draft_logits.is_contiguous():
        raise ValueError("logits must be contiguous")
    if draft_logits.dtype != target_logits.dtype or \
            tuple(draft_logits.shape) != (batch, max_k, stride):
        raise ValueError("draft_logits must be [batch, max_k, row_stride] of the target's dtype")
    if draft_tokens.dtype != torch.int32 or tuple(draft_tokens.shape) != (batch, max_k):
        raise ValueError("draft_tokens must be int32 [batch, max_k]")
    if u_accept.dtype != torch.float32 or tuple(u_accept.shape) != (batch, max_k) or \
            u_sample.dtype != torch.float32 or tuple(u_sample.shape) != (batch,):
        raise ValueError("u_accept float32 [batch, max_k], u_sample float32 [batch]")
    V = stride if vocab is None else vocab
    kl = _host_i32(k_len_host)
    m = torch.empty(batch, dtype=torch.int32, device=target_logits.device)
    nxt = torch.empty(batch, dtype=torch.int32, device=target_logits.device)
    n = ctypes.c_size_t(0)
    _check(load().ssl_spec_accept_workspace(batch, max_k, V, ctypes.byref(n)),
           "ssl_spec_accept_workspace")
    ws = torch.empty(max(int(n.value), 1), dtype=torch.uint8, device=target_logits.device)
    _check(load().ssl_spec_accept(_ptr(target_logits), _ptr(draft_logits),
                                  _logit_dtype(target_logits), batch, max_k,
                                  kl.ctypes.data_as(_i32p), V, stride, _ptr(draft_tokens),
                                  float(temperature), _ptr(u_accept), _ptr(u_sample), _ptr(m),
                                  _ptr(nxt), _ptr(ws), ws.numel(), _stream(stream)),
           "ssl_spec_accept")
    return m, nxt


# ---------------------------------------------------------------------------
# controller
# ---------------------------------------------------------------------------

class Controller:
    """Eq. 6-8 speculation-length controller (host C code)."""

    def __init__(self, beta: float = 0.9, candidates: Sequence[int] = tuple(range(1, 21)),
                 k_default: int = 4):
        c = _host_i32(list(candidates))
        self._lib = load()
        self._h = self._lib.ssl_ctrl_create(float(beta), c.ctypes.data_as(_i32p), len(c),
                                            int(k_default))
        if not self._h:
            raise ValueError("invalid controller arguments")

    def __del__(self):
        h = getattr(self, "_h", None)
        if h:
            self._lib.ssl_ctrl_destroy(h)
            self._h = None

    def observe(self, entropies: Sequence[float], n_accepted: int) -> None:
        H = np.ascontiguousarray(np.asarray(entropies, dtype=np.float64).reshape(-1))
        _check(self._lib.ssl_ctrl_observe(self._h, H.ctypes.data_as(_f64p), len(H),
                                          int(n_accepted)), "ssl_ctrl_observe")

    def accept_prob(self, H: float) -> float:
        return float(self._lib.ssl_ctrl_accept_prob(self._h, float(H)))

    def choose_k(self, entropies: Sequence[float], c_draft: float, c_verify: float) -> int:
        H = np.ascontiguousarray(np.asarray(entropies, dtype=np.float64).reshape(-1))
        if len(H) == 0:
            H = np.zeros(1)
            n = 0
        else:
            n = len(H)
        k = int(self._lib.ssl_ctrl_choose_k(self._h, H.ctypes.data_as(_f64p), n, float(c_draft),
                                            float(c_verify)))
        if k < 0:
            raise SSLError(k, "ssl_ctrl_choose_k")
        return k

    def state(self) -> Tuple[float, float, bool, bool]:
        s = np.zeros(4)
        _check(self._lib.ssl_ctrl_get_state(self._h, s.ctypes.data_as(_f64p)), "ssl_ctrl_get_state")
        return float(s[0]), float(s[1]), bool(s[2]), bool(s[3])

    def set_state(self, h_acc: float, h_rej: float, seen_acc: bool, seen_rej: bool) -> None:
        s = np.array([h_acc, h_rej, float(seen_acc), float(seen_rej)], dtype=np.float64)
        _check(self._lib.ssl_ctrl_set_state(self._h, s.ctypes.data_as(_f64p)), "ssl_ctrl_set_state")


# ---------------------------------------------------------------------------
# Prepared step: marshalling done once, each call is a single C-ABI call.
# ---------------------------------------------------------------------------

class PreparedStep:
    """One verify + select + draft step over fixed device buffers.

    All argument structures are built once, so ``step()`` (the whole step,
    ssl_decode_step) and each ``verify()`` / ``select()`` / ``draft()`` /
    ``select_draft()`` is one ctypes call into the library on the stream
    given (default: torch's current stream at construction).
    """

    def __init__(self, q, k, v, q_draft, ctx_len, q_len, params: Params, out, scores, idx, n_idx,
                 draft_out, stream=None, shared_workspace: bool = False):
        self._lib = load()
        _need_gpu(q, k, v, q_draft, out, scores, idx, n_idx, draft_out)
        self.shape = verify_shape(q, k)
        self.params = params
        self.ctx = _host_i32(ctx_len)
        self.ql = _host_i32(q_len)
        self.n_idx_host = np.array([index_count(int(t), params.k_sink, params.k_recent,
                                                params.budget) for t in self.ctx], dtype=np.int32)
        self.dshape = Shape(self.shape.batch, self.shape.n_q_heads, self.shape.n_kv_heads,
                            self.shape.head_dim, self.shape.max_ctx, 1)
        vws = verify_workspace_bytes(self.shape, params, self.ctx, self.ql)
        sws = max(select_workspace_bytes(self.shape, params, self.ctx),
                  select_draft_workspace_bytes(self.dshape, params, self.ctx))
        dws = draft_workspace_bytes(self.dshape, params, self.n_idx_host)
        # the one-call step has a workspace of its own (with shared_workspace
        # the three-call form's buffer, made large enough)
        stws = decode_step_workspace_bytes(self.shape, params, self.ctx, self.ql)
        if shared_workspace:   # one buffer for every call, ordered on one stream
            self.vws = torch.empty(max(vws, sws, dws, stws, 1), dtype=torch.uint8, device=q.device)
            self.sws = self.dws = self.stws = self.vws
        else:
            self.vws = torch.empty(max(vws, 1), dtype=torch.uint8, device=q.device)
            self.sws = torch.empty(max(sws, 1), dtype=torch.uint8, device=q.device)
            self.dws = torch.empty(max(dws, 1), dtype=torch.uint8, device=q.device)
            self.stws = torch.empty(max(stws, 1), dtype=torch.uint8, device=q.device)
        self.one_kernel = decode_step_plan(self.shape, params, self.ctx, self.ql)
        self.tensors = (q, k, v, q_draft, out, scores, idx, n_idx, draft_out)
        self.stream = _stream(stream)
        sp, pp = ctypes.byref(self.shape), ctypes.byref(params)
        cp, qp = self.ctx.ctypes.data_as(_i32p), self.ql.ctypes.data_as(_i32p)
        self._v = (sp, pp, cp, qp, q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                   scores.data_ptr(), self.vws.data_ptr(), self.vws.numel(), self.stream)
        self._s = (sp, pp, cp, scores.data_ptr(), idx.data_ptr(), n_idx.data_ptr(),
                   self.sws.data_ptr(), self.sws.numel(), self.stream)
        self._d = (ctypes.byref(self.dshape), pp, self.n_idx_host.ctypes.data_as(_i32p),
                   q_draft.data_ptr(), k.data_ptr(), v.data_ptr(), idx.data_ptr(),
                   draft_out.data_ptr(), self.dws.data_ptr(), self.dws.numel(), self.stream)
        self._sd = (ctypes.byref(self.dshape), pp, cp, scores.data_ptr(), idx.data_ptr(),
                    n_idx.data_ptr(), q_draft.data_ptr(), k.data_ptr(), v.data_ptr(),
                    draft_out.data_ptr(), self.sws.data_ptr(), self.sws.numel(), self.stream)
        self._st = (sp, pp, cp, qp, q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(),
                    scores.data_ptr(), idx.data_ptr(), n_idx.data_ptr(), q_draft.data_ptr(),
                    draft_out.data_ptr(), self.stws.data_ptr(), self.stws.numel(), self.stream)

    def verify(self) -> None:
        _check(self._lib.ssl_verify_attn(*self._v), "ssl_verify_attn")

    def select(self) -> None:
        _check(self._lib.ssl_select_topb(*self._s), "ssl_select_topb")

    def draft(self) -> None:
        _check(self._lib.ssl_draft_attn(*self._d), "ssl_draft_attn")

    def select_draft(self) -> None:
        """select and the first draft step in one call (ssl_select_draft)."""
        _check(self._lib.ssl_select_draft(*self._sd), "ssl_select_draft")

    def step(self) -> None:
        """The whole step in one call (ssl_decode_step)."""
        _check(self._lib.ssl_decode_step(*self._st), "ssl_decode_step")

    def step_two_calls(self) -> None:
        """The same step as verify, then select_draft."""
        self.verify()
        self.select_draft()

    def step_separate(self) -> None:
        """The same step as three calls (verify, select, draft)."""
        self.verify()
        self.select()
        self.draft()


class PreparedRound:
    """A draft round over fixed device buffers: ``step(i)`` for i = 0 .. k_max
    drafted tokens (lengths base_len + i), its fixed rows through ``idx`` or,
    when ``k_sel`` / ``v_sel`` are given, from the copy ``materialize()`` makes
    once per round.  The argument structures are built once, so each call is
    one ctypes call on the stream given (default: torch's current stream at
    construction)."""

    def __init__(self, q_draft, k, v, idx, base_len, k_max: int, params: Params, out,
                 k_sel=None, v_sel=None, stream=None):
        self._lib = load()
        _need_gpu(q_draft, k, v, idx, out)
        sel = k_sel is not None
        if sel:
            _need_gpu(k_sel, v_sel)
        batch, hq, d = q_draft.shape
        _, hkv, max_ctx, _ = k.shape
        self.shape = Shape(batch, hq, hkv, d, max_ctx, 1)
        self.params = params
        self.base = _host_i32(base_len)
        self.curs = [_host_i32(self.base + i) for i in range(k_max + 1)]
        need = max(draft_step_workspace_bytes(self.shape, params, self.base, c) for c in self.curs)
        self.ws = torch.empty(max(need, 1), dtype=torch.uint8, device=q_draft.device)
        self.tensors = (q_draft, k, v, idx, k_sel, v_sel, out)
        self.stream = _stream(stream)
        sp, pp = ctypes.byref(self.shape), ctypes.byref(params)
        bp = self.base.ctypes.data_as(_i32p)
        ks, vs = (k_sel.data_ptr(), v_sel.data_ptr()) if sel else (None, None)
        self._m = (sp, pp, bp, k.data_ptr(), v.data_ptr(), idx.data_ptr(), ks, vs,
                   self.stream) if sel else None
        self._steps = [(sp, pp, bp, c.ctypes.data_as(_i32p), q_draft.data_ptr(), k.data_ptr(),
                        v.data_ptr(), idx.data_ptr(), ks, vs, out.data_ptr(), self.ws.data_ptr(),
                        self.ws.numel(), self.stream) for c in self.curs]

    def materialize(self) -> None:
        if self._m is None:
            raise ValueError("this round reads its fixed rows through idx")
        _check(self._lib.ssl_draft_materialize(*self._m), "ssl_draft_materialize")

    def step(self, i: int) -> None:
        _check(self._lib.ssl_draft_step(*self._steps[i]), "ssl_draft_step")
