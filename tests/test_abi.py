"""C-ABI contract on the CPU: the library loads, exports what the header
declares, and every host-side validation error is reachable (validation runs
before any HIP call, so no GPU is needed)."""
import ctypes
import math
import os
import re

import numpy as np
import pytest

import oracle
from paper_2607_27735_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sparsespec_l.h")

FAKE = 0x10000          # a 256-byte aligned non-null address; never dereferenced
FAKE_ODD = 0x10002


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(B.LIB_PATH):
        from paper_2607_27735_amd import build
        build.build()
    return B.load()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ssl_[a-z_]+)\s*\(", text)))


def test_header_symbols_exported(lib):
    names = declared_functions()
    assert len(names) >= 15
    for n in names:
        assert hasattr(lib, n), f"{n} declared in the header but not exported"
    assert sorted(B.EXPORTED) == names


def test_every_export_has_argtypes(lib):
    """Without argtypes ctypes passes Python ints as 32-bit C ints, which
    truncates pointers and stream handles: every call that takes arguments
    must declare them."""
    for n in B.EXPORTED:
        f = getattr(lib, n)
        if n in ("ssl_build_id", "ssl_last_hip_error"):
            continue
        assert f.argtypes, f"{n} has no argtypes"


def _shape(**kw):
    d = dict(batch=1, n_q_heads=32, n_kv_heads=8, head_dim=128, max_ctx=4096, max_q=8)
    d.update(kw)
    return B.Shape(**d)


def _params(**kw):
    d = dict(sm_scale=1 / math.sqrt(128), window=16, k_sink=4, k_recent=32, budget=256,
             out_fp32=0, verify_mode=0)
    d.update(kw)
    return B.Params(**d)


def _i32(*v):
    a = np.array(v, dtype=np.int32)
    return a, a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def _verify(lib, shape=None, params=None, ctx=(4096,), ql=(7,), q=FAKE, k=FAKE, v=FAKE, out=FAKE,
            scores=FAKE, ws=FAKE, ws_bytes=1 << 40, null_shape=False, null_params=False,
            null_ctx=False):
    shape = shape or _shape(batch=len(ctx))
    params = params or _params()
    ca, cp = _i32(*ctx)
    qa, qp = _i32(*ql)
    return lib.ssl_verify_attn(None if null_shape else ctypes.byref(shape),
                               None if null_params else ctypes.byref(params),
                               None if null_ctx else cp, qp, q, k, v, out, scores, ws, ws_bytes,
                               None)


def test_verify_validation(lib):
    assert _verify(lib, null_shape=True) == B.SSL_ERR_NULL
    assert _verify(lib, null_params=True) == B.SSL_ERR_NULL
    assert _verify(lib, null_ctx=True) == B.SSL_ERR_NULL
    assert _verify(lib, shape=_shape(head_dim=64)) == B.SSL_ERR_UNSUPPORTED
    assert _verify(lib, shape=_shape(batch=0), ctx=(), ql=()) == B.SSL_ERR_SHAPE
    assert _verify(lib, shape=_shape(batch=65), ctx=(100,) * 65, ql=(1,) * 65) == \
        B.SSL_ERR_UNSUPPORTED
    assert _verify(lib, shape=_shape(n_q_heads=30)) == B.SSL_ERR_SHAPE
    assert _verify(lib, shape=_shape(n_kv_heads=0)) == B.SSL_ERR_SHAPE
    assert _verify(lib, ql=(0,)) == B.SSL_ERR_SHAPE
    assert _verify(lib, ctx=(5,), ql=(6,)) == B.SSL_ERR_SHAPE           # q_len > ctx_len
    assert _verify(lib, ctx=(4097,)) == B.SSL_ERR_SHAPE                 # ctx_len > max_ctx
    assert _verify(lib, ql=(9,)) == B.SSL_ERR_SHAPE                     # q_len > max_q
    assert _verify(lib, shape=_shape(max_q=65)) == B.SSL_ERR_SHAPE
    # more than 64 rows per KV head: row blocks, two sweeps only
    assert _verify(lib, shape=_shape(n_q_heads=64, max_q=16), ql=(9,),
                   params=_params(verify_mode=2)) == B.SSL_ERR_UNSUPPORTED
    assert B.verify_plan(_shape(n_q_heads=64, max_q=16), _params(), [4000], [16])[0] == \
        B.VERIFY_TWO_SWEEP
    assert _verify(lib, shape=_shape(n_q_heads=128, n_kv_heads=1), ql=(1,)) == \
        B.SSL_ERR_UNSUPPORTED                                        # group > 64
    assert _verify(lib, params=_params(window=0)) == B.SSL_ERR_SHAPE
    assert _verify(lib, params=_params(sm_scale=0.0)) == B.SSL_ERR_SHAPE
    assert _verify(lib, params=_params(sm_scale=float("nan"))) == B.SSL_ERR_SHAPE
    assert _verify(lib, params=_params(verify_mode=3)) == B.SSL_ERR_SHAPE
    assert _verify(lib, params=_params(verify_mode=-1)) == B.SSL_ERR_SHAPE
    # one-sweep requests whose (sequence, KV head) would need more than 128
    # resident chunks: 2^20 keys, and 65537 keys at 64 rows (512-key chunks)
    big = _shape(max_ctx=1 << 20)
    assert _verify(lib, shape=big, ctx=(1 << 20,), params=_params(verify_mode=2)) == \
        B.SSL_ERR_UNSUPPORTED
    rows64 = _shape(n_q_heads=64, n_kv_heads=8, max_ctx=1 << 17, max_q=8)
    assert _verify(lib, shape=rows64, ctx=(128 * 512 + 1,), ql=(8,),
                   params=_params(verify_mode=2)) == B.SSL_ERR_UNSUPPORTED
    for name in ("q", "k", "v", "out", "scores"):
        assert _verify(lib, **{name: None}) == B.SSL_ERR_NULL, name
        assert _verify(lib, **{name: FAKE_ODD}) == B.SSL_ERR_ALIGN, name
    assert _verify(lib, ws=None) == B.SSL_ERR_WORKSPACE
    assert _verify(lib, ws_bytes=16) == B.SSL_ERR_WORKSPACE
    assert _verify(lib, ws=FAKE + 8) == B.SSL_ERR_ALIGN


def test_verify_workspace_query(lib):
    n = ctypes.c_size_t(0)
    ca, cp = _i32(32768)
    qa, qp = _i32(7)
    s, p = _shape(max_ctx=32768), _params()
    assert lib.ssl_verify_workspace(ctypes.byref(s), ctypes.byref(p), cp, qp, None) == \
        B.SSL_ERR_NULL
    assert lib.ssl_verify_workspace(ctypes.byref(s), ctypes.byref(p), cp, qp, ctypes.byref(n)) == 0
    small = n.value
    assert small > 0
    # one byte short is rejected before anything else happens
    assert lib.ssl_verify_attn(ctypes.byref(s), ctypes.byref(p), cp, qp, FAKE, FAKE, FAKE, FAKE,
                               FAKE, FAKE, small - 1, None) == B.SSL_ERR_WORKSPACE
    ca2, cp2 = _i32(32768, 1000)
    qa2, qp2 = _i32(7, 3)
    s2 = _shape(batch=2, max_ctx=32768)
    assert lib.ssl_verify_workspace(ctypes.byref(s2), ctypes.byref(p), cp2, qp2,
                                    ctypes.byref(n)) == 0
    assert n.value > 0


def _select(lib, shape=None, params=None, ctx=(4096,), scores=FAKE, idx=FAKE, n_idx=FAKE):
    shape = shape or _shape(batch=len(ctx))
    params = params or _params()
    ca, cp = _i32(*ctx)
    return lib.ssl_select_topb(ctypes.byref(shape), ctypes.byref(params), cp, scores, idx, n_idx,
                               None, 0, None)


def test_select_validation(lib):
    assert _select(lib, params=_params(budget=0)) == B.SSL_ERR_BUDGET
    assert _select(lib, params=_params(k_sink=-1)) == B.SSL_ERR_BUDGET
    assert _select(lib, params=_params(k_recent=-1)) == B.SSL_ERR_BUDGET
    assert _select(lib, params=_params(k_sink=200, k_recent=57)) == B.SSL_ERR_BUDGET
    assert _select(lib, ctx=(0,)) == B.SSL_ERR_SHAPE
    assert _select(lib, ctx=(4097,)) == B.SSL_ERR_SHAPE
    assert _select(lib, shape=_shape(head_dim=96)) == B.SSL_ERR_UNSUPPORTED
    for name in ("scores", "idx", "n_idx"):
        assert _select(lib, **{name: None}) == B.SSL_ERR_NULL
        assert _select(lib, **{name: FAKE_ODD}) == B.SSL_ERR_ALIGN
    n = ctypes.c_size_t(7)
    ca, cp = _i32(4096)
    s, p = _shape(), _params()
    assert lib.ssl_select_workspace(ctypes.byref(s), ctypes.byref(p), cp, ctypes.byref(n)) == 0
    assert n.value > 0
    assert _select(lib) == B.SSL_ERR_WORKSPACE          # a workspace is required
    ca2, cp2 = _i32(1 << 21)
    s2 = _shape(max_ctx=1 << 22)
    assert lib.ssl_select_workspace(ctypes.byref(s2), ctypes.byref(p), cp2, ctypes.byref(n)) == 0
    ca3, cp3 = _i32((1 << 21) + 1)                       # beyond 256 partitions of 8192
    assert lib.ssl_select_workspace(ctypes.byref(s2), ctypes.byref(p), cp3,
                                    ctypes.byref(n)) == B.SSL_ERR_UNSUPPORTED


def _decode(lib, shape=None, params=None, ctx=(4096,), ql=(7,), q=FAKE, k=FAKE, v=FAKE, out=FAKE,
            scores=FAKE, idx=FAKE, n_idx=FAKE, qd=FAKE, dout=FAKE, ws=FAKE, ws_bytes=1 << 40):
    shape = shape or _shape(batch=len(ctx))
    params = params or _params()
    ca, cp = _i32(*ctx)
    qa, qp = _i32(*ql)
    return lib.ssl_decode_step(ctypes.byref(shape), ctypes.byref(params), cp, qp, q, k, v, out,
                               scores, idx, n_idx, qd, dout, ws, ws_bytes, None)


def test_decode_step_validation(lib):
    # the verify checks, then the select and draft checks, before any HIP call
    assert _decode(lib, ql=(0,)) == B.SSL_ERR_SHAPE
    assert _decode(lib, ctx=(4097,)) == B.SSL_ERR_SHAPE
    assert _decode(lib, shape=_shape(head_dim=64)) == B.SSL_ERR_UNSUPPORTED
    assert _decode(lib, params=_params(budget=0)) == B.SSL_ERR_BUDGET
    assert _decode(lib, params=_params(k_sink=200, k_recent=57)) == B.SSL_ERR_BUDGET
    assert _decode(lib, params=_params(sm_scale=0.0)) == B.SSL_ERR_SHAPE
    for name in ("q", "k", "v", "out", "scores", "idx", "n_idx", "qd", "dout"):
        assert _decode(lib, **{name: None}) == B.SSL_ERR_NULL, name
        assert _decode(lib, **{name: FAKE_ODD}) == B.SSL_ERR_ALIGN, name
    assert _decode(lib, ws=None) == B.SSL_ERR_WORKSPACE
    assert _decode(lib, ws_bytes=8) == B.SSL_ERR_WORKSPACE
    n = ctypes.c_size_t(0)
    ca, cp = _i32(4096)
    qa, qp = _i32(7)
    s, p = _shape(), _params()
    assert lib.ssl_decode_step_workspace(ctypes.byref(s), ctypes.byref(p), cp, qp,
                                         ctypes.byref(n)) == 0
    assert n.value > 65536   # the epoch prefix and more
    assert _decode(lib, ws_bytes=n.value - 1) == B.SSL_ERR_WORKSPACE
    one = ctypes.c_int32(-1)
    assert lib.ssl_decode_step_plan(ctypes.byref(s), ctypes.byref(p), cp, qp,
                                    ctypes.byref(one)) == 0
    assert one.value in (0, 1)
    assert lib.ssl_decode_step_plan(ctypes.byref(s), ctypes.byref(p), cp, qp, None) == B.SSL_ERR_NULL
    assert lib.ssl_decode_step_workspace(ctypes.byref(s), ctypes.byref(p), cp, qp,
                                         None) == B.SSL_ERR_NULL


def _draft(lib, shape=None, params=None, nidx=(256,), q=FAKE, k=FAKE, v=FAKE, idx=FAKE, out=FAKE,
           ws=FAKE, ws_bytes=1 << 40):
    shape = shape or _shape(batch=len(nidx))
    params = params or _params()
    na, npp = _i32(*nidx)
    return lib.ssl_draft_attn(ctypes.byref(shape), ctypes.byref(params), npp, q, k, v, idx, out,
                              ws, ws_bytes, None)


def test_draft_validation(lib):
    assert _draft(lib, nidx=(0,)) == B.SSL_ERR_SHAPE
    assert _draft(lib, nidx=(257,)) == B.SSL_ERR_SHAPE
    assert _draft(lib, params=_params(budget=10)) == B.SSL_ERR_BUDGET
    assert _draft(lib, shape=_shape(n_q_heads=34, n_kv_heads=2)) == B.SSL_ERR_UNSUPPORTED
    assert _draft(lib, shape=_shape(n_q_heads=30)) == B.SSL_ERR_SHAPE
    for name in ("q", "k", "v", "idx", "out"):
        assert _draft(lib, **{name: None}) == B.SSL_ERR_NULL
        assert _draft(lib, **{name: FAKE_ODD}) == B.SSL_ERR_ALIGN
    assert _draft(lib, ws=None) == B.SSL_ERR_WORKSPACE
    assert _draft(lib, ws_bytes=8) == B.SSL_ERR_WORKSPACE


def _step(lib, shape=None, params=None, ctx=(4000,), cur=(4003,), q=FAKE, k=FAKE, v=FAKE,
          idx=FAKE, ks=FAKE, vs=FAKE, out=FAKE, ws=FAKE, ws_bytes=1 << 40):
    shape = shape or _shape(batch=len(ctx))
    params = params or _params()
    ca, cp = _i32(*ctx)
    ua, up = _i32(*cur)
    return lib.ssl_draft_step(ctypes.byref(shape), ctypes.byref(params), cp, up, q, k, v, idx, ks,
                              vs, out, ws, ws_bytes, None)


def test_draft_round_validation(lib):
    # the drafted tail must lie in the recent window: T <= cur <= T + k_recent, cur <= max_ctx
    assert _step(lib, cur=(3999,)) == B.SSL_ERR_SHAPE
    assert _step(lib, cur=(4033,)) == B.SSL_ERR_SHAPE
    assert _step(lib, ctx=(4090,), cur=(4097,)) == B.SSL_ERR_SHAPE
    assert _step(lib, ctx=(0,), cur=(0,)) == B.SSL_ERR_SHAPE
    assert _step(lib, params=_params(k_recent=0), cur=(4001,)) == B.SSL_ERR_SHAPE
    assert _step(lib, params=_params(budget=10)) == B.SSL_ERR_BUDGET
    assert _step(lib, shape=_shape(n_q_heads=34, n_kv_heads=2)) == B.SSL_ERR_UNSUPPORTED
    for name in ("q", "k", "v", "ks", "vs", "out"):
        assert _step(lib, **{name: None}) == B.SSL_ERR_NULL
        assert _step(lib, **{name: FAKE_ODD}) == B.SSL_ERR_ALIGN
    # fixed rows through idx: idx required and aligned, k_sel / v_sel both absent
    assert _step(lib, ks=None, vs=None, idx=None) == B.SSL_ERR_NULL
    assert _step(lib, ks=None, vs=None, idx=FAKE + 2) == B.SSL_ERR_ALIGN
    assert _step(lib, ks=None, vs=None, idx=FAKE, ws=None) == B.SSL_ERR_WORKSPACE
    assert _step(lib, ws=None) == B.SSL_ERR_WORKSPACE
    assert _step(lib, ws_bytes=8) == B.SSL_ERR_WORKSPACE
    # the workspace covers the step's entries, the same count as the draft's
    s, p = _shape(), _params()
    n1, n2 = ctypes.c_size_t(0), ctypes.c_size_t(0)
    ca, cp = _i32(4000)
    ua, up = _i32(4020)
    na, npp = _i32(B.index_count(4000, p.k_sink, p.k_recent, p.budget))
    assert lib.ssl_draft_step_workspace(ctypes.byref(s), ctypes.byref(p), cp, up, ctypes.byref(n1)) == 0
    assert lib.ssl_draft_workspace(ctypes.byref(s), ctypes.byref(p), npp, ctypes.byref(n2)) == 0
    assert n1.value == n2.value > 0
    # materialization: the same length checks, and its buffers are required
    assert lib.ssl_draft_materialize(ctypes.byref(s), ctypes.byref(p), cp, FAKE, FAKE, FAKE,
                                     None, FAKE, None) == B.SSL_ERR_NULL
    assert lib.ssl_draft_materialize(ctypes.byref(s), ctypes.byref(p), cp, FAKE, FAKE, FAKE,
                                     FAKE_ODD, FAKE, None) == B.SSL_ERR_ALIGN
    za, zp = _i32(0)
    assert lib.ssl_draft_materialize(ctypes.byref(s), ctypes.byref(p), zp, FAKE, FAKE, FAKE,
                                     FAKE, FAKE, None) == B.SSL_ERR_SHAPE


def test_logit_stats_validation(lib):
    n = ctypes.c_size_t(0)
    assert lib.ssl_logit_stats_workspace(7, 128256, ctypes.byref(n)) == 0 and n.value > 0
    assert lib.ssl_logit_stats_workspace(0, 100, ctypes.byref(n)) == B.SSL_ERR_SHAPE
    assert lib.ssl_logit_stats_workspace(1, 524289, ctypes.byref(n)) == B.SSL_ERR_UNSUPPORTED

    def call(logits=FAKE, dtype=0, rows=7, vocab=128256, stride=128256, ent=FAKE, am=FAKE,
             ws=FAKE, ws_bytes=1 << 40):
        return lib.ssl_logit_stats(logits, dtype, rows, vocab, stride, ent, am, ws, ws_bytes, None)
    assert call(dtype=2) == B.SSL_ERR_SHAPE
    assert call(stride=128000) == B.SSL_ERR_SHAPE
    assert call(logits=None) == B.SSL_ERR_NULL
    assert call(ent=None, am=None) == B.SSL_ERR_NULL
    assert call(logits=FAKE_ODD) == B.SSL_ERR_ALIGN
    assert call(vocab=100, stride=100) == B.SSL_ERR_ALIGN          # 200-byte rows
    # 400-byte fp32 rows are aligned: the call gets as far as the workspace check
    assert call(dtype=1, vocab=100, stride=100, ws=None) == B.SSL_ERR_WORKSPACE
    assert call(ent=FAKE + 2) == B.SSL_ERR_ALIGN
    assert call(ws=None) == B.SSL_ERR_WORKSPACE
    assert call(ws_bytes=8) == B.SSL_ERR_WORKSPACE


def test_greedy_accept_validation(lib):
    n = ctypes.c_size_t(0)
    assert lib.ssl_greedy_accept_workspace(4, 6, 128256, ctypes.byref(n)) == 0 and n.value > 0
    assert lib.ssl_greedy_accept_workspace(65, 6, 100, ctypes.byref(n)) == B.SSL_ERR_UNSUPPORTED
    assert lib.ssl_greedy_accept_workspace(1, 64, 100, ctypes.byref(n)) == B.SSL_ERR_UNSUPPORTED

    def call(k=(6, 2), max_k=6, draft=FAKE, m=FAKE, nxt=FAKE, ws=FAKE, ws_bytes=1 << 40):
        ka, kp = _i32(*k)
        return lib.ssl_greedy_accept(FAKE, 0, len(k), max_k, kp, 128256, 128256, draft, m, nxt,
                                     ws, ws_bytes, None)
    assert call(k=(7, 2)) == B.SSL_ERR_SHAPE
    assert call(k=(-1, 2)) == B.SSL_ERR_SHAPE
    assert call(draft=None) == B.SSL_ERR_NULL
    assert call(m=None) == B.SSL_ERR_NULL
    assert call(nxt=FAKE + 1) == B.SSL_ERR_ALIGN
    assert call(ws=None) == B.SSL_ERR_WORKSPACE


def test_spec_accept_validation(lib):
    n = ctypes.c_size_t(0)
    assert lib.ssl_spec_accept_workspace(4, 6, 128256, ctypes.byref(n)) == 0 and n.value > 65536
    assert lib.ssl_spec_accept_workspace(65, 6, 100, ctypes.byref(n)) == B.SSL_ERR_UNSUPPORTED
    assert lib.ssl_spec_accept_workspace(1, 64, 100, ctypes.byref(n)) == B.SSL_ERR_UNSUPPORTED
    assert lib.ssl_spec_accept_workspace(1, 4, (1 << 19) + 1, ctypes.byref(n)) == B.SSL_ERR_UNSUPPORTED
    assert lib.ssl_spec_accept_workspace(0, 4, 100, ctypes.byref(n)) == B.SSL_ERR_SHAPE

    def call(k=(6, 2), max_k=6, tau=1.0, tl=FAKE, dl=FAKE, dtype=0, stride=128256, draft=FAKE,
             ua=FAKE, us=FAKE, m=FAKE, nxt=FAKE, ws=FAKE, ws_bytes=1 << 40):
        ka, kp = _i32(*k)
        return lib.ssl_spec_accept(tl, dl, dtype, len(k), max_k, kp, 128256, stride, draft, tau,
                                   ua, us, m, nxt, ws, ws_bytes, None)
    for tau in (0.0, -1.0, float("nan"), float("inf"), 1e-39):
        assert call(tau=tau) == B.SSL_ERR_SHAPE, tau
    assert call(k=(7, 2)) == B.SSL_ERR_SHAPE
    assert call(dtype=5) == B.SSL_ERR_SHAPE
    assert call(stride=100) == B.SSL_ERR_SHAPE
    assert call(stride=128257) == B.SSL_ERR_ALIGN        # rows must stay 16-byte aligned
    for name in ("tl", "dl", "draft", "ua", "us", "m", "nxt"):
        assert call(**{name: None}) == B.SSL_ERR_NULL, name
    assert call(m=FAKE + 2) == B.SSL_ERR_ALIGN
    assert call(ws=None) == B.SSL_ERR_WORKSPACE
    # nothing drafted anywhere: the drafter's rows, tokens and pass uniforms are not needed
    assert call(k=(0, 0), max_k=0, dl=None, draft=None, ua=None, ws=None) == B.SSL_ERR_WORKSPACE


def test_paged_validation(lib):
    s, p = _shape(), _params()
    ca, cp = _i32(4000)
    qa, qp = _i32(7)

    def ver(bt=FAKE, page=64, blocks=64, ws=FAKE, ws_bytes=1 << 40):
        return lib.ssl_verify_attn_paged(ctypes.byref(s), ctypes.byref(p), cp, qp, FAKE, FAKE,
                                         FAKE, bt, page, blocks, FAKE, FAKE, ws, ws_bytes, None)
    assert ver(bt=None) == B.SSL_ERR_NULL
    assert ver(bt=FAKE + 2) == B.SSL_ERR_ALIGN
    assert ver(page=48) == B.SSL_ERR_SHAPE            # not a multiple of 32
    assert ver(page=0) == B.SSL_ERR_SHAPE
    assert ver(blocks=62) == B.SSL_ERR_SHAPE          # 62 * 64 < 4000
    assert ver(ws=None) == B.SSL_ERR_WORKSPACE         # valid otherwise: stops at the workspace
    na, npp = _i32(256)

    def dra(bt=FAKE, page=64, blocks=64, ws=FAKE):
        return lib.ssl_draft_attn_paged(ctypes.byref(s), ctypes.byref(p), npp, FAKE, FAKE, FAKE,
                                        bt, page, blocks, FAKE, FAKE, ws, 1 << 40, None)
    assert dra(bt=None) == B.SSL_ERR_NULL
    assert dra(page=16) == B.SSL_ERR_SHAPE
    assert dra(blocks=63) == B.SSL_ERR_SHAPE          # 63 * 64 < max_ctx 4096
    assert dra(ws=None) == B.SSL_ERR_WORKSPACE
    # the draft round over pages: the step's and the materialization's checks
    ua, up = _i32(4003)

    def stp(bt=FAKE, page=64, blocks=64, ws=FAKE, cur=up):
        return lib.ssl_draft_step_paged(ctypes.byref(s), ctypes.byref(p), cp, cur, FAKE, FAKE,
                                        FAKE, bt, page, blocks, FAKE, None, None, FAKE, ws,
                                        1 << 40, None)
    assert stp(bt=None) == B.SSL_ERR_NULL
    assert stp(bt=FAKE + 2) == B.SSL_ERR_ALIGN
    assert stp(page=40) == B.SSL_ERR_SHAPE
    assert stp(blocks=63) == B.SSL_ERR_SHAPE          # the pages must cover max_ctx
    ba, bp = _i32(4097)
    assert stp(cur=bp) == B.SSL_ERR_SHAPE             # cur past max_ctx
    assert stp(ws=None) == B.SSL_ERR_WORKSPACE

    def mat(bt=FAKE, page=64, blocks=64, k_sel=FAKE):
        return lib.ssl_draft_materialize_paged(ctypes.byref(s), ctypes.byref(p), cp, FAKE, FAKE,
                                               bt, page, blocks, FAKE, k_sel, FAKE, None)
    assert mat(bt=None) == B.SSL_ERR_NULL
    assert mat(page=0) == B.SSL_ERR_SHAPE
    assert mat(blocks=1) == B.SSL_ERR_SHAPE
    assert mat(k_sel=None) == B.SSL_ERR_NULL
    assert mat(k_sel=FAKE_ODD) == B.SSL_ERR_ALIGN


def test_status_strings(lib):
    seen = set()
    for code in range(0, -8, -1):
        s = B.status_string(code)
        assert s and s != "unknown status"
        seen.add(s)
    assert len(seen) == 8
    assert B.status_string(-99) == "unknown status"


def test_index_count_matches_oracle(lib):
    rng = np.random.default_rng(5)
    for _ in range(300):
        T = int(rng.integers(1, 5000))
        ks, kr = int(rng.integers(0, 40)), int(rng.integers(0, 80))
        B_ = ks + kr + int(rng.integers(0, 3000))
        if B_ < 1:
            continue
        assert B.index_count(T, ks, kr, B_) == oracle.index_count(T, ks, kr, B_)
    assert B.index_count(0, 4, 32, 256) == B.SSL_ERR_SHAPE
    assert B.index_count(10, 4, 32, 20) == B.SSL_ERR_BUDGET


def test_binding_refuses_cpu_tensors(lib):
    import torch
    q = torch.zeros(1, 2, 8, 128, dtype=torch.bfloat16)
    k = torch.zeros(1, 2, 64, 128, dtype=torch.bfloat16)
    with pytest.raises(RuntimeError, match="no CPU fallback"):
        B.verify_attn(q, k, k, [64], [2], B.make_params(0.1))


def test_verify_plan_schedules(lib):
    """Schedules of the named workloads: one sweep fits wherever a (sequence,
    KV head) needs at most 128 chunks of what the LDS logit stash holds (all
    but the 131K context); AUTO takes it there when a KV head has at most 32
    verify rows (not at 44 or 48); TWO_SWEEP always plans."""
    from paper_2607_27735_amd.workloads import CONFIGS
    fits = {1: True, 2: True, 3: True, 4: False, 5: True}
    auto_one = {1: True, 2: True, 3: False, 4: False, 5: False}
    for n, cfg in CONFIGS.items():
        batch = cfg["batch"]
        ctx = cfg.get("ctx_len") or [cfg["ctx_range"][1]] * batch
        ql = cfg.get("q_len") or [cfg["k_range"][1] + 1] * batch
        shape = B.Shape(batch, cfg["n_q_heads"], cfg["n_kv_heads"], 128,
                        cfg.get("max_ctx") or max(ctx), max(ql))
        sch, chunk, items = B.verify_plan(shape, B.make_params(1 / math.sqrt(128)), ctx, ql)
        assert sch == (B.VERIFY_ONE_SWEEP if auto_one[n] else B.VERIFY_TWO_SWEEP), n
        assert chunk % 128 == 0 and items >= 1
        two = B.make_params(1 / math.sqrt(128), verify_mode=B.VERIFY_TWO_SWEEP)
        sch, chunk, items = B.verify_plan(shape, two, ctx, ql)
        assert sch == B.VERIFY_TWO_SWEEP and chunk >= 128
        one = B.make_params(1 / math.sqrt(128), verify_mode=B.VERIFY_ONE_SWEEP)
        if fits[n]:
            sch, chunk, items = B.verify_plan(shape, one, ctx, ql)
            assert sch == B.VERIFY_ONE_SWEEP and chunk % 128 == 0
            assert all(-(-t // chunk) <= 128 for t in ctx)
            assert items == sum(cfg["n_kv_heads"] * -(-t // chunk) for t in ctx)
        else:
            with pytest.raises(B.SSLError):
                B.verify_plan(shape, one, ctx, ql)


# ---------------------------------------------------------------------------
# build identity, exchange health, co-residency planning
# ---------------------------------------------------------------------------

def test_build_id_matches_tree(lib):
    from paper_2607_27735_amd import build
    assert B.build_id() == build.source_id()


def test_load_refuses_a_stale_library(lib, monkeypatch):
    from paper_2607_27735_amd import build
    monkeypatch.setattr(build, "source_id", lambda: "0" * 16)
    monkeypatch.setattr(B, "_lib", None)
    with pytest.raises(RuntimeError, match="built from other sources"):
        B.load()


def test_exchange_hooks_validate(lib):
    assert lib.ssl_exchange_status(None, None) == B.SSL_ERR_NULL
    assert lib.ssl_set_cu_budget(-1) == B.SSL_ERR_SHAPE
    assert lib.ssl_test_exchange_faults(-1, 0) == B.SSL_ERR_SHAPE
    assert lib.ssl_test_exchange_faults(16, 2) == B.SSL_ERR_SHAPE
    assert lib.ssl_test_exchange_faults(0, 0) == B.SSL_OK


@pytest.fixture
def cu_budget(lib):
    yield lambda n: B.set_cu_budget(n)
    B.set_cu_budget(0)


def _plan_32k(rows_q=7, group=4, T=32768, batch=1, hkv=8):
    s = _shape(batch=batch, n_q_heads=hkv * group, n_kv_heads=hkv, max_ctx=T, max_q=rows_q)
    p = _params(budget=2048)
    return s, p, [T] * batch, [rows_q] * batch


def test_verify_plan_follows_the_cu_budget(lib, cu_budget):
    """The one-workgroup-per-chunk one sweep needs the call's chunks to run in
    one round of workgroups and every chunk of a (sequence, KV head) resident
    at once, within half of what the CUs hold (one workgroup per CU here): the
    32K workload's heads take 32 chunks of 1024 keys (the LDS stash's limit at
    28 rows).  Below 256 CUs the persistent form takes over (a grid of the
    budget, at most one grid of chunks per head, 1024 keys of 16-bit stash),
    and below 32 CUs neither fits: two sweeps."""
    s, p, ctx, ql = _plan_32k()
    cu_budget(256)
    assert B.verify_plan(s, p, ctx, ql) == (B.VERIFY_ONE_SWEEP, 1024, 256)
    for n in (64, 32):
        cu_budget(n)
        assert B.verify_plan(s, p, ctx, ql) == (B.VERIFY_ONE_SWEEP_PERSISTENT, 1024, 256), n
    cu_budget(62)   # 896 keys: 296 chunks in five rounds of 62, against 256 in five
    assert B.verify_plan(s, p, ctx, ql) == (B.VERIFY_ONE_SWEEP_PERSISTENT, 896, 296)
    cu_budget(31)
    assert B.verify_plan(s, p, ctx, ql)[0] == B.VERIFY_TWO_SWEEP
    cu_budget(16)
    assert B.verify_plan(s, p, ctx, ql)[0] == B.VERIFY_TWO_SWEEP
    # a one-sweep request that cannot be resident is refused, not launched
    one = _params(budget=2048, verify_mode=B.VERIFY_ONE_SWEEP)
    n = ctypes.c_size_t(0)
    ctx_a, ctx_p = _i32(*ctx)
    q_a, q_p = _i32(*ql)
    assert lib.ssl_verify_workspace(ctypes.byref(s), ctypes.byref(one), ctx_p, q_p,
                                    ctypes.byref(n)) == B.SSL_ERR_UNSUPPORTED
    # a short context still takes one sweep in a small budget (persistent: its
    # 32 chunks over 16 workgroups)
    s2, p2, ctx2, ql2 = _plan_32k(T=4096)
    assert B.verify_plan(s2, p2, ctx2, ql2)[0] == B.VERIFY_ONE_SWEEP_PERSISTENT


def test_persistent_plan_limits(lib, cu_budget):
    """The persistent form: at most 48 rows per KV head (its kernel is built for
    three row tiles), at most 64 chunks per head, a grid of what the budget
    holds and never more workgroups than chunks; its chunks a multiple of 128
    keys within the two 16-bit stash buffers' limit."""
    cu_budget(64)
    for rows_q, group, ok in ((7, 4, True), (6, 8, True), (16, 4, False)):
        s, p, ctx, ql = _plan_32k(rows_q=rows_q, group=group)
        sch, chunk, items = B.verify_plan(s, p, ctx, ql)
        if ok:
            assert sch == B.VERIFY_ONE_SWEEP_PERSISTENT and chunk % 128 == 0, (rows_q, group)
            assert -(-32768 // chunk) <= 64 and items == 8 * -(-32768 // chunk)
        else:
            assert sch == B.VERIFY_TWO_SWEEP, (rows_q, group)
    # a head of 131K keys needs more than 64 chunks of what 48 rows allow
    s, p, ctx, ql = _plan_32k(rows_q=6, group=8, T=131072)
    assert B.verify_plan(s, p, ctx, ql)[0] == B.VERIFY_TWO_SWEEP


def test_auto_one_sweep_at_three_row_tiles_needs_one_round(lib, cu_budget):
    """33-64 rows per KV head: AUTO takes the one-workgroup-per-chunk one sweep
    when its chunks run in one round of workgroups (44 rows at 16K: 256 chunks
    of 512 keys), the persistent form where that applies, and two sweeps where
    neither does (48 rows over 64K keys per head: 103 chunks of 640 keys)."""
    cu_budget(256)
    s, p, ctx, ql = _plan_32k(rows_q=11, group=4, T=16384)
    assert B.verify_plan(s, p, ctx, ql) == (B.VERIFY_ONE_SWEEP, 512, 256)
    assert B.decode_step_plan(s, p, ctx, ql) is True
    s, p, ctx, ql = _plan_32k(rows_q=6, group=8, T=8192)
    assert B.verify_plan(s, p, ctx, ql)[0] == B.VERIFY_ONE_SWEEP
    s, p, ctx, ql = _plan_32k(rows_q=9, group=4, T=32768)   # 416 chunks of 640: persistent
    assert B.verify_plan(s, p, ctx, ql)[0] == B.VERIFY_ONE_SWEEP_PERSISTENT
    s, p, ctx, ql = _plan_32k(rows_q=6, group=8, T=65536, batch=4)
    assert B.verify_plan(s, p, ctx, ql)[0] == B.VERIFY_TWO_SWEEP
    # 64 rows (four row tiles): one sweep in one round, else two sweeps (the
    # persistent form is built for up to three row tiles)
    s, p, ctx, ql = _plan_32k(rows_q=16, group=4, T=4096)
    assert B.verify_plan(s, p, ctx, ql)[0] == B.VERIFY_ONE_SWEEP
    s, p, ctx, ql = _plan_32k(rows_q=8, group=8, T=32768)
    assert B.verify_plan(s, p, ctx, ql)[0] == B.VERIFY_TWO_SWEEP


def test_select_plan_follows_the_cu_budget(lib, cu_budget):
    s, p, ctx, _ = _plan_32k()
    cu_budget(256)
    assert B.select_plan(s, p, ctx) == (True, 1024, 32)
    cu_budget(32)          # 16 resident partitions < 32 per unit: three kernels
    assert B.select_plan(s, p, ctx) == (False, 1024, 32)
    cu_budget(256)         # more than 256 partitions in the call: three kernels
    s8, p8, ctx8, _ = _plan_32k(batch=2)
    assert B.select_plan(s8, p8, ctx8)[0] is False


def test_every_workspace_starts_with_the_epoch_words(lib):
    """All layouts share a 64 KiB prefix of exchange epochs (8192 words), so calls
    that share a workspace never store other data over each other's epochs."""
    s, p, ctx, ql = _plan_32k()
    assert B.verify_workspace_bytes(s, p, ctx, ql) > 65536
    assert B.select_workspace_bytes(s, p, ctx) > 65536
    assert B.draft_workspace_bytes(s, p, [2048]) > 65536
    assert B.decode_step_workspace_bytes(s, p, ctx, ql) > 65536
    n = ctypes.c_size_t(0)
    assert lib.ssl_logit_stats_workspace(1, 1000, ctypes.byref(n)) == B.SSL_OK and n.value > 65536


def test_static_verify_validates_before_any_hip_call(lib):
    """ssl_verify_attn_static checks its arguments, and that the workspace its
    plan needs fits the library's 128 MiB scratch, before looking the scratch
    up (so these errors need no GPU)."""
    s, p = _shape(), _params()
    ctx, cp = _i32(4000)
    ql, qp = _i32(5)
    f = lib.ssl_verify_attn_static
    assert f(None, ctypes.byref(p), cp, qp, FAKE, FAKE, FAKE, FAKE, FAKE, None) == B.SSL_ERR_NULL
    assert f(ctypes.byref(s), ctypes.byref(p), cp, qp, None, FAKE, FAKE, FAKE, FAKE,
             None) == B.SSL_ERR_NULL
    assert f(ctypes.byref(s), ctypes.byref(p), cp, qp, FAKE_ODD, FAKE, FAKE, FAKE, FAKE,
             None) == B.SSL_ERR_ALIGN
    bad = _shape(head_dim=64)
    assert f(ctypes.byref(bad), ctypes.byref(p), cp, qp, FAKE, FAKE, FAKE, FAKE, FAKE,
             None) == B.SSL_ERR_UNSUPPORTED
    # 16 sequences of 131072 keys: a workspace beyond the scratch
    big = _shape(batch=16, max_ctx=131072)
    ctxb, cbp = _i32(*[131072] * 16)
    qlb, qbp = _i32(*[5] * 16)
    n = ctypes.c_size_t(0)
    assert lib.ssl_verify_workspace(ctypes.byref(big), ctypes.byref(p), cbp, qbp,
                                    ctypes.byref(n)) == B.SSL_OK
    assert n.value > 128 << 20
    assert f(ctypes.byref(big), ctypes.byref(p), cbp, qbp, FAKE, FAKE, FAKE, FAKE, FAKE,
             None) == B.SSL_ERR_WORKSPACE


def test_two_sweep_chunk_minimises_rounds(lib, cu_budget):
    """The two-sweep chunk is the power of two in [128, 65536] that minimises
    (rounds of one item per CU) x (chunk + 256 keys), the smallest on ties:
    checked by brute force over random ragged shapes and CU budgets."""
    import numpy as np
    rng = np.random.default_rng(11)
    for _ in range(60):
        batch = int(rng.integers(1, 9))
        hkv = int(rng.choice([1, 2, 4, 8]))
        ctx = [int(x) for x in rng.integers(1, 200000, size=batch)]
        ql = [1] * batch
        n_cu = int(rng.choice([1, 3, 8, 64, 256]))
        cu_budget(n_cu)
        s = _shape(batch=batch, n_q_heads=hkv * 4, n_kv_heads=hkv, max_ctx=max(ctx), max_q=1)
        p = _params(budget=64, verify_mode=B.VERIFY_TWO_SWEEP)
        sch, chunk, items = B.verify_plan(s, p, ctx, ql)
        best = None
        for c in (128 << j for j in range(10)):
            n = sum(hkv * -(-t // c) for t in ctx)
            cost = -(-n // n_cu) * (c + 256)
            if best is None or cost < best[0]:
                best = (cost, c, n)
        assert (sch, chunk, items) == (B.VERIFY_TWO_SWEEP, best[1], best[2]), (batch, hkv, ctx, n_cu)
