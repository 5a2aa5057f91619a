"""The same calls under different work decompositions (a check for races and
for decomposition-dependent results).

The CU count the plans assume (ssl_set_cu_budget) changes how calls are cut:
select runs as one kernel with its partitions exchanging, or as three
kernels; the draft takes 128, 256 or 512 index entries per workgroup; verify
changes its chunking and schedule.  Index sets are integer results and must
be bit-identical under every decomposition (and equal to the oracle's);
floating-point outputs must each meet the oracle's bar and agree with each
other within twice the per-element bound."""
import numpy as np
import pytest
import torch

import oracle
from gpu_common import Dev, abs_v, check_outputs, gpu_draft, gpu_select, gpu_verify
from paper_2607_27735_amd import binding as B
from paper_2607_27735_amd.workloads import generate

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU visible", allow_module_level=True)

BUDGETS = [0, 64, 16, 4, 1]


@pytest.fixture(autouse=True)
def _reset_budget():
    yield
    B.set_cu_budget(0)


def _workload():
    return generate(701, name="sched", batch=3, n_q_heads=32, n_kv_heads=8,
                    ctx_len=[9000, 2500, 6000], q_len=[5, 2, 7], budget=700, max_ctx=9000,
                    heavy_hitters=4)


@pytest.mark.parametrize("kind", ["random", "ties"])
def test_select_identical_under_every_schedule(kind):
    w = _workload()
    rng = np.random.default_rng(3 if kind == "random" else 4)
    shape = (w.batch, w.n_kv_heads, w.max_ctx)
    s32 = (rng.random(shape) if kind == "random" else rng.integers(0, 6, shape) / 5.0).astype(np.float32)
    idx_ref, n_ref = oracle.select(w, s32.astype(np.float64))
    vshape = B.Shape(w.batch, w.n_q_heads, w.n_kv_heads, 128, w.max_ctx, w.max_q)
    p = B.make_params(w.sm_scale, budget=w.budget, k_sink=w.k_sink, k_recent=w.k_recent)
    first, schedules = None, set()
    for cus in BUDGETS:
        B.set_cu_budget(cus)
        one, part, parts = B.select_plan(vshape, p, w.ctx_len)
        schedules.add(one)
        print(f"[select {kind}] CU budget {cus}: one kernel {one}, {parts} x {part}", flush=True)
        idx, n_idx = gpu_select(w, s32)
        assert np.array_equal(n_idx, n_ref)
        for b in range(w.batch):
            assert np.array_equal(idx[b, :, :n_ref[b]], idx_ref[b, :, :n_ref[b]])
        if first is None:
            first = (idx, n_idx)
        assert np.array_equal(idx, first[0]) and np.array_equal(n_idx, first[1])
    assert schedules == {True, False}   # both schedules were exercised
    assert B.exchange_status() == 0


def test_draft_agrees_across_workgroup_sizes():
    w = _workload()
    _, s_ref = oracle.verify(w)
    idx_ref, n_ref = oracle.select(w, s_ref.astype(np.float32).astype(np.float64))
    idx_dev = np.where(idx_ref < 0, 0, idx_ref).astype(np.int32)
    o_ref = oracle.draft(w, idx_dev, n_ref)
    oabs = oracle.draft(w, idx_dev, n_ref, v=abs_v(w))
    d = Dev(w)
    outs = []
    for cus in BUDGETS:
        B.set_cu_budget(cus)
        o = gpu_draft(d, idx_dev, n_ref)
        check_outputs(o, o_ref, oabs, np.ones(o_ref.shape[:2], dtype=bool), what=f"draft {cus}")
        outs.append(o)
    for o in outs[1:]:
        assert np.all(np.abs(o - outs[0]) <= 2 * (4e-3 * oabs + 1e-6))
    assert B.exchange_status() == 0


def test_verify_agrees_across_chunkings():
    w = _workload()
    out_ref, s_ref = oracle.verify(w)
    oabs, _ = oracle.verify(w, v=abs_v(w))
    mask = np.arange(w.max_q)[None, :, None] < w.q_len[:, None, None] * np.ones((1, 1, w.n_q_heads), bool)
    d = Dev(w)
    outs, plans = [], set()
    for cus in BUDGETS:
        B.set_cu_budget(cus)
        p = B.make_params(w.sm_scale, window=w.window)
        plans.add(B.verify_plan(B.verify_shape(d.q, d.k), p, w.ctx_len, w.q_len))
        o, s = gpu_verify(d)
        check_outputs(o, out_ref, oabs, mask, what=f"verify {cus}")
        for b in range(w.batch):
            T = int(w.ctx_len[b])
            rel = np.abs(s[b, :, :T] - s_ref[b, :, :T]) / np.maximum(s_ref[b, :, :T], 1e-30)
            assert np.all(rel[s_ref[b, :, :T] > 0] <= 1e-3)
        outs.append(o)
    for o in outs[1:]:
        assert np.all(np.abs(o - outs[0])[mask] <= 2 * (4e-3 * oabs[mask] + 1e-6))
    assert len(plans) >= 3   # several chunkings (and both schedules) were exercised
    assert B.exchange_status() == 0


@pytest.mark.parametrize("ctx,cus,chunk", [([16384, 16379], 16, 16384), ([32768, 30000], 8, 32768)])
def test_two_sweep_large_chunks(ctx, cus, chunk):
    """Two sweeps over chunks of 16384 and 32768 keys (the chunk the plan takes
    when a call's units outnumber the CUs: fewer rounds of workgroups), with a
    ragged last chunk and a sequence shorter than one chunk, against the
    oracle."""
    w = generate(702, name="big-chunks", batch=2, n_q_heads=32, n_kv_heads=8, ctx_len=ctx,
                 q_len=[7, 4], budget=512, heavy_hitters=4)
    d = Dev(w)
    B.set_cu_budget(cus)
    p = B.make_params(w.sm_scale, window=w.window, verify_mode=B.VERIFY_TWO_SWEEP)
    assert B.verify_plan(B.verify_shape(d.q, d.k), p, w.ctx_len, w.q_len)[:2] == (B.VERIFY_TWO_SWEEP, chunk)
    o, s = gpu_verify(d, mode=B.VERIFY_TWO_SWEEP)
    out_ref, s_ref = oracle.verify(w)
    oabs, _ = oracle.verify(w, v=abs_v(w))
    mask = np.arange(w.max_q)[None, :, None] < w.q_len[:, None, None] * np.ones((1, 1, w.n_q_heads), bool)
    check_outputs(o, out_ref, oabs, mask, what=f"two sweeps, chunk {chunk}")
    for b in range(w.batch):
        T = int(w.ctx_len[b])
        rel = np.abs(s[b, :, :T] - s_ref[b, :, :T]) / np.maximum(s_ref[b, :, :T], 1e-30)
        assert np.all(rel[s_ref[b, :, :T] > 0] <= 1e-3)
        assert np.all(s[b, :, T:] == -1.0)
    assert B.exchange_status() == 0
