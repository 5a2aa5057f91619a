"""GPU parity of the whole decode step in one call (ssl_decode_step): verify
with its Eq. 3 scores, the Eq. 4 index sets and the first Eq. 5 draft step.

Where verify takes one sweep in one round of chunk workgroups of >= 512 keys
the step is one kernel (each chunk workgroup is also a select partition and
drafts over its own selections); elsewhere (the small cases here) it is verify
followed by select_draft.  Either way: the outputs and scores equal
verify_attn's bit for bit (the same arithmetic) and meet the oracle's bars;
the index sets equal, bit for bit, the oracle's select run on the step's own
fp32 scores; the draft output meets the draft bar against the oracle's draft
over those index sets; slots past n_idx are not written."""
import numpy as np
import pytest
import torch

import oracle
from gpu_common import Dev, abs_v, check_decode_step, gpu_decode_step, params_of
from paper_2607_27735_amd import binding as B
from paper_2607_27735_amd.workloads import generate, make_config
from test_gpu_parity import SMALL, small_case

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU visible", allow_module_level=True)


@pytest.mark.parametrize("name", list(SMALL))
def test_decode_step_matches_oracle(name):
    w, out_ref, s_ref, oabs_ref = small_case(name)
    check_decode_step(w, out_ref, s_ref, oabs_ref)


@pytest.mark.parametrize("name", ["tiny-config", "ragged-b3", "kv8-b3"])
def test_decode_step_bf16_outputs(name):
    w, out_ref, s_ref, oabs_ref = small_case(name)
    check_decode_step(w, out_ref, s_ref, oabs_ref, out_fp32=False)


# Shapes whose step runs as one kernel on the full device (every chunk
# workgroup resident at once, chunks of >= 512 keys): ragged contexts with
# ragged last chunks, ragged verify lengths, groups of 4, 8 and 16, two to
# four row tiles.
ONE_KERNEL = {
    "b2-kv8-ragged": lambda: generate(611, name="b2-kv8-ragged", batch=2, n_q_heads=32,
                                      n_kv_heads=8, ctx_len=[8192, 5000], q_len=[5, 3],
                                      budget=512, max_ctx=8200, heavy_hitters=4),
    "b3-kv4-g8": lambda: generate(612, name="b3-kv4-g8", batch=3, n_q_heads=32, n_kv_heads=4,
                                  ctx_len=[20000, 9000, 13001], q_len=[4, 2, 3], budget=1000,
                                  max_ctx=20000),
    "b1-kv2-g16": lambda: generate(613, name="b1-kv2-g16", batch=1, n_q_heads=32, n_kv_heads=2,
                                   ctx_len=[60000], q_len=[2], budget=2048, window=1),
    # 44 rows per KV head: three row tiles, chunks of 512 keys in one round
    "b1-kv8-rows44": lambda: generate(615, name="b1-kv8-rows44", batch=1, n_q_heads=32, n_kv_heads=8,
                                      ctx_len=[16384], q_len=[11], budget=2048, heavy_hitters=4),
    # 64 rows per KV head (group 8): four row tiles, chunks of 512 keys
    "b1-kv8-rows64": lambda: generate(616, name="b1-kv8-rows64", batch=1, n_q_heads=64, n_kv_heads=8,
                                      ctx_len=[16384], q_len=[8], budget=2048),
}


@pytest.mark.parametrize("name", list(ONE_KERNEL))
def test_decode_step_one_kernel(name):
    w = ONE_KERNEL[name]()
    out_ref, s_ref = oracle.verify(w)
    oabs_ref, _ = oracle.verify(w, v=abs_v(w))
    check_decode_step(w, out_ref, s_ref, oabs_ref, expect_one_kernel=True)
    check_decode_step(w, out_ref, s_ref, oabs_ref, out_fp32=False, expect_one_kernel=True)


def test_decode_step_select_cases():
    """Budgets that take every middle position, none, only the sink or only
    the recent window (no radix select: ranges), and ordinary ones, over a
    ragged batch in one kernel."""
    w = ONE_KERNEL["b2-kv8-ragged"]()
    out_ref, s_ref = oracle.verify(w)
    oabs_ref, _ = oracle.verify(w, v=abs_v(w))
    for budget, ks, kr in [(300, 4, 32), (8192, 4, 32), (64, 64, 0), (10, 0, 10), (36, 4, 32),
                           (1, 0, 0), (5000, 0, 0), (4999, 0, 0)]:
        print(f"[decode step] budget {budget} sink {ks} recent {kr}", flush=True)
        check_decode_step(w, out_ref, s_ref, oabs_ref, budget=budget, k_sink=ks, k_recent=kr,
                          expect_one_kernel=True)


def test_decode_step_small_cu_budget():
    """Planned for 16 CUs, a 4K two-head case runs as one kernel of 16
    workgroups (512-key chunks); the results stay right."""
    w = generate(614, name="cu16", batch=1, n_q_heads=8, n_kv_heads=2, ctx_len=[4000],
                 q_len=[5], budget=256)
    out_ref, s_ref = oracle.verify(w)
    oabs_ref, _ = oracle.verify(w, v=abs_v(w))
    B.set_cu_budget(16)
    try:
        check_decode_step(w, out_ref, s_ref, oabs_ref, expect_one_kernel=True)
    finally:
        B.set_cu_budget(0)


def test_decode_step_plan_follows_verify():
    """One kernel only where verify takes one sweep and per_head is off."""
    w = make_config(2)
    d = Dev(w)
    shape = B.verify_shape(d.q, d.k)
    p = params_of(w)
    assert B.decode_step_plan(shape, p, w.ctx_len, w.q_len)
    p2 = params_of(w, mode=B.VERIFY_TWO_SWEEP)
    assert not B.decode_step_plan(shape, p2, w.ctx_len, w.q_len)
    p3 = params_of(w)
    p3.per_head = 1
    assert not B.decode_step_plan(shape, p3, w.ctx_len, w.q_len)


def test_decode_step_deterministic():
    w = ONE_KERNEL["b2-kv8-ragged"]()
    d = Dev(w)
    a = gpu_decode_step(d)
    b = gpu_decode_step(d)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
