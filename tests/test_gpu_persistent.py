"""GPU parity of the persistent one-sweep verify schedule.

Where one-sweep chunks would take more than one round of workgroups, verify
runs a persistent grid that takes every grid-th chunk and keeps two chunks'
probabilities in 16-bit form (relative error 2^-11).  These cases lower the
CU budget (ssl_set_cu_budget) so that small shapes, which the oracle checks
element by element, take that schedule with several chunks per workgroup,
units that straddle two rounds, ragged contexts and row counts, and 16, 32
and 48 rows per KV head; the paged cache and per-head scores take it too, a
captured graph replays it, and forced exchange faults make it give up
cleanly."""
import numpy as np
import pytest
import torch

import oracle
from gpu_common import Dev, abs_v, check_outputs, check_score_mass, check_scores, dev_bf16, params_of
from paper_2607_27735_amd import binding as B
from paper_2607_27735_amd.workloads import generate

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU visible", allow_module_level=True)

NAN_BF16 = np.uint16(0x7FC0)


def _poison(w):
    for b in range(w.batch):
        w.k[b, :, w.ctx_len[b]:] = NAN_BF16
        w.v[b, :, w.ctx_len[b]:] = NAN_BF16
        w.q[b, w.q_len[b]:] = NAN_BF16
    return w


# name: (workload, CU budget)
CASES = {
    # 28 rows (two row tiles), three sequences, units of 3-5 chunks over 16 workgroups
    "kv8-rows28": (lambda: _poison(generate(
        501, name="kv8-rows28", batch=3, n_q_heads=32, n_kv_heads=8, ctx_len=[3000, 1700, 4097],
        q_len=[7, 3, 5], max_ctx=4100, max_q=7, budget=300, heavy_hitters=4)), 16),
    # 16 rows (one row tile), a short and a long sequence
    "kv2-rows16": (lambda: _poison(generate(
        502, name="kv2-rows16", batch=2, n_q_heads=8, n_kv_heads=2, ctx_len=[9000, 900],
        q_len=[4, 2], max_ctx=9000, max_q=4, budget=400)), 6),
    # 48 rows (three row tiles, the 70B group of 8)
    "kv8-rows48-g8": (lambda: _poison(generate(
        503, name="kv8-rows48-g8", batch=2, n_q_heads=64, n_kv_heads=8, ctx_len=[2600, 1300],
        q_len=[6, 4], max_ctx=2600, max_q=6, budget=200)), 8),
    # sixteen sequences of 1-3000 keys and 1-8 positions: many short units,
    # several per round, some of a single chunk
    "b16-short": (lambda: _poison(generate(
        505, name="b16-short", batch=16, n_q_heads=8, n_kv_heads=2,
        ctx_len=[2433, 2551, 917, 2110, 2226, 53, 935, 2997, 601, 2338, 1248, 1530, 2013, 235, 658, 983],
        q_len=[3, 7, 8, 6, 2, 7, 3, 8, 7, 5, 6, 2, 3, 3, 8, 7], max_ctx=3000, max_q=8, budget=128)), 8),
    # tiny contexts: chunks of a single key, sequences shorter than a tile
    "tiny-T": (lambda: _poison(generate(
        504, name="tiny-T", batch=4, n_q_heads=8, n_kv_heads=2, ctx_len=[1, 5, 130, 700],
        q_len=[1, 5, 3, 2], max_ctx=700, budget=16, k_sink=4, k_recent=8)), 2),
}


@pytest.fixture(autouse=True)
def _reset():
    torch.cuda.synchronize()
    B.exchange_status()
    yield
    B.set_cu_budget(0)
    B.test_exchange_faults(0, False)
    torch.cuda.synchronize()
    B.exchange_status()


def _mask(w):
    return np.arange(w.max_q)[None, :, None] < w.q_len[:, None, None] * np.ones((1, 1, w.n_q_heads), bool)


def _run(d, p, out_fill=-7.0, s_fill=-1.0, out_dtype=torch.float32):
    w = d.w
    out = torch.full(d.q.shape, out_fill, dtype=out_dtype, device="cuda")
    sc = torch.full((w.batch, w.n_kv_heads, w.max_ctx), s_fill, dtype=torch.float32, device="cuda")
    B.verify_attn(d.q, d.k, d.v, w.ctx_len, w.q_len, p, out=out, scores=sc)
    torch.cuda.synchronize()
    return out.float().cpu().numpy().astype(np.float64), sc.cpu().numpy().astype(np.float64)


def _plan(d, p):
    plan = B.verify_plan(B.verify_shape(d.q, d.k), p, d.w.ctx_len, d.w.q_len)
    print(f"  plan {plan}", flush=True)
    return plan


@pytest.mark.parametrize("name", list(CASES))
def test_persistent_verify_matches_oracle(name):
    make, budget = CASES[name]
    w = make()
    print(f"[persistent] {w.describe()}, CU budget {budget}", flush=True)
    d = Dev(w)
    B.set_cu_budget(budget)
    p = params_of(w, out_fp32=True)
    sch, chunk, items = _plan(d, p)
    assert sch == B.VERIFY_ONE_SWEEP_PERSISTENT and items > budget
    out, s = _run(d, p)
    out_ref, s_ref = oracle.verify(w)
    oabs, _ = oracle.verify(w, v=abs_v(w))
    mask = _mask(w)
    err = check_outputs(out, out_ref, oabs, mask)
    worst = check_scores(s, s_ref, w.ctx_len)
    check_score_mass(s, w)
    assert np.all(out[~mask] == -7.0)
    for b in range(w.batch):
        assert np.all(s[b, :, w.ctx_len[b]:] == -1.0)
    assert B.exchange_status() == 0
    # the same call again gives the same bits (fixed summation orders)
    out2, s2 = _run(d, p, out_fill=3.0, s_fill=5.0)
    assert np.array_equal(out2[mask], out[mask])
    for b in range(w.batch):
        assert np.array_equal(s2[b, :, :w.ctx_len[b]], s[b, :, :w.ctx_len[b]])
    print(f"  max|dO|={err:.2e} worst rel dS={worst:.2e}")


def test_persistent_bf16_outputs_and_single_round_agreement():
    """bf16 outputs stay within half a bf16 ulp of the oracle's bar, and the
    persistent scores agree with the one-workgroup-per-chunk schedule's
    (fp32 stash) to the 16-bit code's 2^-11."""
    make, budget = CASES["kv8-rows28"]
    w = make()
    d = Dev(w)
    p16 = params_of(w, out_fp32=False)
    out_ref, s_ref = oracle.verify(w)
    oabs, _ = oracle.verify(w, v=abs_v(w))
    B.set_cu_budget(0)
    assert _plan(d, p16)[0] == B.VERIFY_ONE_SWEEP
    _, s_one = _run(d, p16, out_dtype=torch.bfloat16)
    B.set_cu_budget(budget)
    assert _plan(d, p16)[0] == B.VERIFY_ONE_SWEEP_PERSISTENT
    out, s = _run(d, p16, out_dtype=torch.bfloat16)
    check_outputs(out, out_ref, oabs, _mask(w), out_fp32=False)
    check_scores(s, s_ref, w.ctx_len)
    for b in range(w.batch):
        T = int(w.ctx_len[b])
        rel = np.abs(s[b, :, :T] - s_one[b, :, :T]) / np.maximum(s_one[b, :, :T], 1e-300)
        assert rel.max() <= 2 ** -10, rel.max()


def test_persistent_per_head_scores():
    make, budget = CASES["kv8-rows28"]
    w = make()
    d = Dev(w)
    B.set_cu_budget(budget)
    p = B.make_params(w.sm_scale, window=w.window, k_sink=w.k_sink, k_recent=w.k_recent,
                      budget=w.budget, out_fp32=True, per_head=True)
    assert _plan(d, p)[0] == B.VERIFY_ONE_SWEEP_PERSISTENT
    out = torch.full(d.q.shape, -7.0, dtype=torch.float32, device="cuda")
    sc = torch.full((w.batch, w.n_q_heads, w.max_ctx), -1.0, dtype=torch.float32, device="cuda")
    B.verify_attn(d.q, d.k, d.v, w.ctx_len, w.q_len, p, out=out, scores=sc)
    torch.cuda.synchronize()
    s = sc.cpu().numpy().astype(np.float64)
    s_ref = oracle.head_scores(w)
    check_scores(s, s_ref, w.ctx_len, what="per-head S")
    out_ref, _ = oracle.verify(w)
    oabs, _ = oracle.verify(w, v=abs_v(w))
    check_outputs(out.cpu().numpy().astype(np.float64), out_ref, oabs, _mask(w))


def test_persistent_paged_matches_dense():
    """Over a shuffled page pool the persistent schedule gives the dense call's
    bits."""
    from test_gpu_paged import paged
    make, budget = CASES["kv8-rows28"]
    w = make()
    d = Dev(w)
    B.set_cu_budget(budget)
    p = params_of(w, out_fp32=True)
    assert _plan(d, p)[0] == B.VERIFY_ONE_SWEEP_PERSISTENT
    kp, vp, bt, max_blocks = paged(w, 64, seed=77)
    out, sc = B.verify_attn_paged(d.q, dev_bf16(kp), dev_bf16(vp), torch.from_numpy(bt).cuda(), w.max_ctx,
                                  w.ctx_len, w.q_len, p)
    torch.cuda.synchronize()
    out = out.float().cpu().numpy().astype(np.float64)
    sc = sc.cpu().numpy().astype(np.float64)
    out_d, s_d = _run(d, p)
    mask = _mask(w)
    assert np.array_equal(out[mask], out_d[mask])
    for b in range(w.batch):
        T = int(w.ctx_len[b])
        assert np.array_equal(sc[b, :, :T], s_d[b, :, :T])


def test_persistent_graph_replays():
    """A captured persistent call, replayed over new cache contents, matches
    the eager call on every replay (the exchange epochs)."""
    make, budget = CASES["kv2-rows16"]
    w = make()
    d = Dev(w)
    B.set_cu_budget(budget)
    p = params_of(w, out_fp32=True)
    assert _plan(d, p)[0] == B.VERIFY_ONE_SWEEP_PERSISTENT
    shape = B.verify_shape(d.q, d.k)
    ws = torch.zeros(B.verify_workspace_bytes(shape, p, w.ctx_len, w.q_len), dtype=torch.uint8,
                     device="cuda")
    out = torch.zeros(d.q.shape, dtype=torch.float32, device="cuda")
    sc = torch.zeros((w.batch, w.n_kv_heads, w.max_ctx), dtype=torch.float32, device="cuda")
    k_live, v_live = d.k.clone(), d.v.clone()
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        B.verify_attn(d.q, k_live, v_live, w.ctx_len, w.q_len, p, out=out, scores=sc, workspace=ws,
                      stream=stream)
        stream.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            B.verify_attn(d.q, k_live, v_live, w.ctx_len, w.q_len, p, out=out, scores=sc, workspace=ws,
                          stream=stream)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(9)
    for rep in range(4):
        k_live.copy_(d.k * (1.0 + 0.25 * rep))
        v_live.copy_(torch.randn(d.v.shape, generator=gen, device="cuda").to(torch.bfloat16))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        o_g, s_g = out.clone(), sc.clone()
        o_e, s_e = torch.zeros_like(out), torch.zeros_like(sc)
        B.verify_attn(d.q, k_live, v_live, w.ctx_len, w.q_len, p, out=o_e, scores=s_e)
        torch.cuda.synchronize()
        for b in range(w.batch):
            T, nq = int(w.ctx_len[b]), int(w.q_len[b])
            assert torch.equal(o_g[b, :nq], o_e[b, :nq]), rep
            assert torch.equal(s_g[b, :, :T], s_e[b, :, :T]), rep
    assert B.exchange_status() == 0


def test_persistent_gives_up_cleanly():
    """Every statistics wait forced to give up (a small poll limit and tags no
    wait accepts): the kernel finishes, writes neither scores nor outputs and
    raises the verify bit; normal calls then work again."""
    make, budget = CASES["kv8-rows28"]
    w = make()
    d = Dev(w)
    B.set_cu_budget(budget)
    p = params_of(w, out_fp32=True)
    assert _plan(d, p)[0] == B.VERIFY_ONE_SWEEP_PERSISTENT
    B.test_exchange_faults(64, True)
    out, s = _run(d, p)
    assert B.exchange_status() == B.EXCHANGE_VERIFY
    assert np.all(out == -7.0) and np.all(s == -1.0)
    B.test_exchange_faults(0, False)
    out, s = _run(d, p)
    assert B.exchange_status() == 0
    out_ref, s_ref = oracle.verify(w)
    oabs, _ = oracle.verify(w, v=abs_v(w))
    check_outputs(out, out_ref, oabs, _mask(w))
    check_scores(s, s_ref, w.ctx_len)
