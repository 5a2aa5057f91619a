"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Small cases are compared element by element (several tiles and work items,
ragged tails, edge cases); the five named workloads run at full size, in the
benchmark's launch configuration, and are compared element by element on
every (sequence, KV head) unit, plus properties that hold at any size.  Oracle inputs never come
from the GPU: index sets fed to both draft paths are the oracle's own.
"""
import functools

import numpy as np
import pytest
import torch

import oracle
from gpu_common import (Dev, abs_v, check_band, check_decode_step, check_index_structure,
                        check_outputs, check_score_mass, check_scores, gpu_draft, gpu_select,
                        gpu_select_draft, gpu_verify, params_of)
from paper_2607_27735_amd import binding as B
from paper_2607_27735_amd.workloads import f32_to_bf16_bits, generate, make_config

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU visible", allow_module_level=True)

NAN_BF16 = np.uint16(0x7FC0)


def _poison_padding(w):
    """Padding rows (beyond ctx_len / q_len) hold NaN: they must never be read."""
    for b in range(w.batch):
        w.k[b, :, w.ctx_len[b]:] = NAN_BF16
        w.v[b, :, w.ctx_len[b]:] = NAN_BF16
        w.q[b, w.q_len[b]:] = NAN_BF16
    return w


SMALL = {
    "tiny-config": lambda: make_config(1),
    "ragged-b3": lambda: _poison_padding(generate(
        101, name="ragged-b3", batch=3, n_q_heads=8, n_kv_heads=2, ctx_len=[1000, 333, 2049],
        q_len=[3, 1, 7], max_ctx=2100, max_q=8, budget=256)),
    "rows64-g8": lambda: generate(102, name="rows64-g8", batch=1, n_q_heads=16, n_kv_heads=2,
                                  ctx_len=[700], q_len=[8], budget=128),
    "g16": lambda: _poison_padding(generate(
        103, name="g16", batch=2, n_q_heads=32, n_kv_heads=2, ctx_len=[513, 129], q_len=[4, 2],
        budget=200, max_ctx=600)),
    "mha-g1": lambda: generate(104, name="mha-g1", batch=1, n_q_heads=4, n_kv_heads=4,
                               ctx_len=[300], q_len=[5], budget=64),
    "tiny-T": lambda: _poison_padding(generate(
        105, name="tiny-T", batch=4, n_q_heads=8, n_kv_heads=2, ctx_len=[1, 5, 17, 33],
        q_len=[1, 5, 3, 2], budget=16, k_sink=4, k_recent=8, max_ctx=40)),
    "window2": lambda: generate(106, name="window2", batch=1, n_q_heads=8, n_kv_heads=2,
                                ctx_len=[900], q_len=[6], window=2, budget=100),
    "chunk-ragged": lambda: generate(107, name="chunk-ragged", batch=1, n_q_heads=8,
                                     n_kv_heads=2, ctx_len=[4097], q_len=[3], budget=300),
    # eight KV heads, several rows per finishing workgroup, one-chunk heads
    "kv8-b3": lambda: _poison_padding(generate(
        108, name="kv8-b3", batch=3, n_q_heads=32, n_kv_heads=8, ctx_len=[1000, 333, 2049],
        q_len=[3, 1, 7], max_ctx=2100, max_q=8, budget=256)),
    "kv8-g16": lambda: _poison_padding(generate(
        109, name="kv8-g16", batch=3, n_q_heads=128, n_kv_heads=8, ctx_len=[1, 130, 700],
        q_len=[1, 4, 4], max_ctx=720, max_q=4, budget=64)),
    # the first index of a sequence, seeded by its prompt: the last W = 16 prompt
    # positions as the query block (64 rows per KV head at group 4)
    "prefill-seed-g4": lambda: _poison_padding(generate(
        110, name="prefill-seed-g4", batch=2, n_q_heads=32, n_kv_heads=8, ctx_len=[4096, 1500],
        q_len=[16, 16], max_ctx=4100, budget=256, heavy_hitters=4)),
    # the same at the 70B shape (group 8): 128 rows per KV head, two row blocks
    "prefill-seed-g8": lambda: _poison_padding(generate(
        111, name="prefill-seed-g8", batch=2, n_q_heads=64, n_kv_heads=8, ctx_len=[4096, 1500],
        q_len=[16, 16], max_ctx=4100, budget=256, heavy_hitters=4)),
    # row blocks over a ragged batch (blocks of 8 positions: the second block
    # has no rows of the second sequence) with the window ending inside a block
    "rowblocks-ragged": lambda: _poison_padding(generate(
        112, name="rowblocks-ragged", batch=3, n_q_heads=16, n_kv_heads=2, ctx_len=[3000, 700, 2049],
        q_len=[20, 3, 11], max_ctx=3010, max_q=20, window=12, budget=200)),
}


def _row_blocks(w):
    """Whether a KV head has more verify rows than one launch holds (64)."""
    return int(max(w.q_len)) * (w.n_q_heads // w.n_kv_heads) > 64


@functools.lru_cache(maxsize=None)
def small_case(name):
    w = SMALL[name]()
    out_ref, s_ref = oracle.verify(w)
    oabs_ref, _ = oracle.verify(w, v=abs_v(w))
    return w, out_ref, s_ref, oabs_ref


def _row_mask(w):
    return np.arange(w.max_q)[None, :, None] < w.q_len[:, None, None] * np.ones(
        (1, 1, w.n_q_heads), dtype=bool)


MODES = {"two-sweep": B.VERIFY_TWO_SWEEP, "one-sweep": B.VERIFY_ONE_SWEEP}


@pytest.mark.parametrize("mode", list(MODES))
@pytest.mark.parametrize("name", list(SMALL))
def test_verify_matches_oracle(name, mode):
    w, out_ref, s_ref, oabs_ref = small_case(name)
    print(f"[verify {mode}] {w.describe()}", flush=True)
    d = Dev(w)
    if _row_blocks(w) and mode == "one-sweep":
        with pytest.raises(B.SSLError) as e:      # row blocks take two sweeps
            gpu_verify(d, out_fp32=True, mode=MODES[mode])
        assert e.value.status == B.SSL_ERR_UNSUPPORTED
        return
    out, s = gpu_verify(d, out_fp32=True, mode=MODES[mode])
    mask = _row_mask(w)
    err = check_outputs(out, out_ref, oabs_ref, mask)
    worst = check_scores(s, s_ref, w.ctx_len)
    check_score_mass(s, w)
    # rows past q_len and scores past ctx_len are not written
    assert np.all(out[~mask] == -7.0)
    for b in range(w.batch):
        assert np.all(s[b, :, w.ctx_len[b]:] == -1.0)
    print(f"  max|dO|={err:.2e} worst rel dS={worst:.2e}")


@pytest.mark.parametrize("mode", list(MODES))
@pytest.mark.parametrize("name", ["tiny-config", "ragged-b3", "g16"])
def test_verify_bf16_outputs(name, mode):
    w, out_ref, s_ref, oabs_ref = small_case(name)
    out, s = gpu_verify(Dev(w), out_fp32=False, mode=MODES[mode])
    check_outputs(out, out_ref, oabs_ref, _row_mask(w), out_fp32=False)
    check_scores(s, s_ref, w.ctx_len)


@pytest.mark.parametrize("name", list(SMALL))
def test_select_bitexact_on_shared_scores(name):
    """GPU select and oracle select on the same fp32 scores (the oracle's verify
    scores rounded to fp32) give identical index sets."""
    w, out_ref, s_ref, oabs_ref = small_case(name)
    s32 = s_ref.astype(np.float32)
    idx_ref, n_ref = oracle.select(w, s32.astype(np.float64))
    idx, n_idx = gpu_select(w, s32)
    assert np.array_equal(n_idx, n_ref)
    for b in range(w.batch):
        assert np.array_equal(idx[b, :, :n_ref[b]], idx_ref[b, :, :n_ref[b]])
    check_index_structure(idx, n_idx, w.ctx_len, w.k_sink, w.k_recent, w.budget)


@pytest.mark.parametrize("name", list(SMALL))
def test_select_band_end_to_end(name):
    """GPU verify -> GPU select, judged by the band rule against fp64 scores."""
    w, out_ref, s_ref, oabs_ref = small_case(name)
    d = Dev(w)
    _, s = gpu_verify(d)
    s32 = np.where(s < 0, 0.0, s).astype(np.float32)
    idx, n_idx = gpu_select(w, s32)
    check_index_structure(idx, n_idx, w.ctx_len, w.k_sink, w.k_recent, w.budget)
    check_band(idx, n_idx, s_ref, w.ctx_len, w.k_sink, w.k_recent, w.budget)


@pytest.mark.parametrize("name", list(SMALL))
def test_draft_matches_oracle(name):
    w, out_ref, s_ref, oabs_ref = small_case(name)
    idx_ref, n_ref = oracle.select(w, s_ref.astype(np.float32).astype(np.float64))
    idx_dev = np.where(idx_ref < 0, 0, idx_ref).astype(np.int32)
    o_ref = oracle.draft(w, idx_dev, n_ref)
    oabs = oracle.draft(w, idx_dev, n_ref, v=abs_v(w))
    o = gpu_draft(Dev(w), idx_dev, n_ref)
    check_outputs(o, o_ref, oabs, np.ones(o_ref.shape[:2], dtype=bool), what="draft")
    ob = gpu_draft(Dev(w), idx_dev, n_ref, out_fp32=False)
    check_outputs(ob, o_ref, oabs, np.ones(o_ref.shape[:2], dtype=bool), out_fp32=False,
                  what="draft-bf16")


@pytest.mark.parametrize("cus", [1, 4])
@pytest.mark.parametrize("name", ["ragged-b3", "g16", "kv8-b3", "chunk-ragged"])
def test_draft_wide_workgroups(name, cus):
    """Planned for 1 or 4 CUs, the draft takes 512 or 256 entries per workgroup
    (4 or 2 tiles per wave, ragged last tiles and units); same bars."""
    w, out_ref, s_ref, oabs_ref = small_case(name)
    idx_ref, n_ref = oracle.select(w, s_ref.astype(np.float32).astype(np.float64))
    idx_dev = np.where(idx_ref < 0, 0, idx_ref).astype(np.int32)
    o_ref = oracle.draft(w, idx_dev, n_ref)
    oabs = oracle.draft(w, idx_dev, n_ref, v=abs_v(w))
    B.set_cu_budget(cus)
    try:
        o = gpu_draft(Dev(w), idx_dev, n_ref)
    finally:
        B.set_cu_budget(0)
    check_outputs(o, o_ref, oabs, np.ones(o_ref.shape[:2], dtype=bool), what="draft")


def _check_select_draft(w, s32, budget=None, k_sink=None, k_recent=None, out_fp32=True):
    """ssl_select_draft against the oracle: index sets bit-exact with the
    oracle's select on the same fp32 scores, the draft over them at the draft
    bar, slots past n_idx untouched."""
    budget = w.budget if budget is None else budget
    ks = w.k_sink if k_sink is None else k_sink
    kr = w.k_recent if k_recent is None else k_recent
    idx_ref, n_ref = oracle.select(w, s32.astype(np.float64), budget=budget, k_sink=ks,
                                   k_recent=kr)
    idx, n_idx, o = gpu_select_draft(Dev(w), s32, out_fp32=out_fp32, budget=budget, k_sink=ks,
                                     k_recent=kr)
    assert np.array_equal(n_idx, n_ref)
    for b in range(w.batch):
        assert np.array_equal(idx[b, :, :n_ref[b]], idx_ref[b, :, :n_ref[b]])
    check_index_structure(idx, n_idx, w.ctx_len, ks, kr, budget)
    idx_dev = np.where(idx_ref < 0, 0, idx_ref).astype(np.int32)
    o_ref = oracle.draft(w, idx_dev, n_ref)
    oabs = oracle.draft(w, idx_dev, n_ref, v=abs_v(w))
    check_outputs(o, o_ref, oabs, np.ones(o_ref.shape[:2], dtype=bool), out_fp32=out_fp32,
                  what="select+draft")


@pytest.mark.parametrize("name", list(SMALL))
def test_select_draft_matches_oracle(name):
    w, out_ref, s_ref, oabs_ref = small_case(name)
    _check_select_draft(w, s_ref.astype(np.float32))


def test_select_draft_special_cases():
    """Units that need no radix select (every middle position taken, or none)
    run the draft over ranges; ties, zeros and one huge score."""
    w = generate(205, name="seldraft", batch=2, n_q_heads=8, n_kv_heads=2, ctx_len=[3000, 2500],
                 q_len=[1, 1], budget=300)
    rng = np.random.default_rng(9)
    shape = (w.batch, w.n_kv_heads, w.max_ctx)
    for label, s32 in {"random": rng.random(shape).astype(np.float32),
                       "quantized-ties": (rng.integers(0, 5, shape) / 4.0).astype(np.float32),
                       "all-zero": np.zeros(shape, np.float32),
                       "one-huge": np.where(rng.random(shape) < 0.001, 1e30, 1e-3).astype(np.float32)
                       }.items():
        for budget, ks, kr in [(300, 4, 32), (3000, 4, 32), (64, 64, 0), (10, 0, 10), (36, 4, 32)]:
            print(f"[select+draft] {label} budget {budget} sink {ks} recent {kr}", flush=True)
            _check_select_draft(w, s32, budget=budget, k_sink=ks, k_recent=kr)


def test_select_special_cases():
    w = generate(201, name="sel", batch=2, n_q_heads=4, n_kv_heads=2, ctx_len=[3000, 2500],
                 q_len=[1, 1], budget=300, head_dim=128)
    rng = np.random.default_rng(7)
    shape = (w.batch, w.n_kv_heads, w.max_ctx)
    cases = {
        "random": rng.random(shape).astype(np.float32),
        "quantized-ties": (rng.integers(0, 5, shape) / 4.0).astype(np.float32),
        "all-zero": np.zeros(shape, np.float32),
        "all-equal": np.full(shape, 0.37, np.float32),
        "tiny-values": (rng.random(shape) * 1e-30).astype(np.float32),
        "one-huge": np.where(rng.random(shape) < 0.001, 1e30, 1e-3).astype(np.float32),
        # -0 and +0 are equal scores: ties broken by position like any others
        "signed-zeros": np.where(rng.random(shape) < 0.2, rng.random(shape),
                                 np.where(rng.random(shape) < 0.5, -0.0, 0.0)).astype(np.float32),
    }
    for label, s32 in cases.items():
        for budget, ks, kr in [(300, 4, 32), (36, 4, 32), (3000, 4, 32), (301, 0, 0),
                               (64, 64, 0), (10, 0, 10), (1, 0, 0)]:
            idx_ref, n_ref = oracle.select(w, s32.astype(np.float64), budget=budget, k_sink=ks,
                                           k_recent=kr)
            idx, n_idx = gpu_select(w, s32, budget=budget, k_sink=ks, k_recent=kr)
            assert np.array_equal(n_idx, n_ref), (label, budget)
            for b in range(w.batch):
                assert np.array_equal(idx[b, :, :n_ref[b]], idx_ref[b, :, :n_ref[b]]), \
                    (label, budget, ks, kr, b)
            check_index_structure(idx, n_idx, w.ctx_len, ks, kr, budget)
    # committed length shorter than the cache, and shorter than the sink
    s32 = cases["random"]
    for ctx in ([17, 3], [2999, 1]):
        idx_ref, n_ref = oracle.select(w, s32.astype(np.float64), ctx_len=np.array(ctx))
        idx, n_idx = gpu_select(w, s32, ctx_len=ctx)
        assert np.array_equal(n_idx, n_ref)
        for b in range(w.batch):
            assert np.array_equal(idx[b, :, :n_ref[b]], idx_ref[b, :, :n_ref[b]])


def test_select_long_contexts():
    """Contexts long enough that one (sequence, KV head) spans many partitions,
    several rounds per partition and more than one emission chunk; with
    quantised or equal scores the threshold bin holds far more candidates than
    the finishing workgroup caches.  Bit-exact against the oracle."""
    from types import SimpleNamespace
    rng = np.random.default_rng(11)
    # the first three calls have at most 256 partitions in all and finish inside the
    # mark kernel; the last (16 x 8 units of 20 partitions) uses the finish kernel
    for batch, hkv, ctx in ((2, 2, [140001, 65537]), (2, 2, [262144, 3]), (2, 2, [40000, 33000]),
                            (16, 8, [20000 - 37 * i for i in range(16)])):
        w = SimpleNamespace(batch=batch, n_q_heads=hkv * 2, n_kv_heads=hkv, max_ctx=max(ctx),
                            ctx_len=np.array(ctx, dtype=np.int32), sm_scale=1.0, window=16,
                            k_sink=4, k_recent=32, budget=4096)
        shape = (w.batch, w.n_kv_heads, w.max_ctx)
        cases = {
            "lognormal": np.exp(rng.normal(-8.0, 1.0, shape)).astype(np.float32),
            "quantized-ties": (rng.integers(0, 3, shape) / 2.0).astype(np.float32),
            "all-equal": np.full(shape, 0.25, np.float32),
        }
        for label, s32 in cases.items():
            for budget in (4096, 20000):
                print(f"select long ctx={ctx} {label} budget={budget}", flush=True)
                idx_ref, n_ref = oracle.select(w, s32.astype(np.float64), budget=budget)
                idx, n_idx = gpu_select(w, s32, budget=budget)
                assert np.array_equal(n_idx, n_ref), (ctx, label, budget)
                for b in range(w.batch):
                    assert np.array_equal(idx[b, :, :n_ref[b]], idx_ref[b, :, :n_ref[b]]), \
                        (ctx, label, budget, b)


def test_draft_full_budget_equals_dense():
    """Sparse attention with every position selected is dense attention: the
    draft kernel over idx = [0, T) equals the verify kernel with one row."""
    w = generate(301, name="dense", batch=2, n_q_heads=8, n_kv_heads=2, ctx_len=[1500, 777],
                 q_len=[1, 1], budget=1500)
    w.q[:, 0] = w.q_draft
    d = Dev(w)
    out_v, _ = gpu_verify(d)
    idx = np.zeros((2, 2, 1500), dtype=np.int32)
    for b in range(2):
        idx[b, :, :w.ctx_len[b]] = np.arange(w.ctx_len[b])
    o = gpu_draft(d, idx, w.ctx_len.copy())
    assert np.abs(o - out_v[:, 0]).max() < 2e-3 * np.abs(out_v[:, 0]).max() + 1e-5
    ref, _ = oracle.verify(w)
    oabs, _ = oracle.verify(w, v=abs_v(w))
    check_outputs(o, ref[:, 0], oabs[:, 0], np.ones((2, 8), dtype=bool), what="draft-dense")


def test_draft_permutation_invariant():
    w = generate(302, name="perm", batch=1, n_q_heads=8, n_kv_heads=2, ctx_len=[2000], q_len=[1],
                 budget=200)
    rng = np.random.default_rng(3)
    idx = np.stack([rng.choice(2000, 200, replace=False) for _ in range(2)])[None].astype(np.int32)
    d = Dev(w)
    o1 = gpu_draft(d, idx, np.array([200]))
    o2 = gpu_draft(d, idx[:, :, ::-1].copy(), np.array([200]))
    # Each order rounds its probabilities to bf16 against its own running
    # maximum, so the two may differ by twice the per-output bound.
    oabs = oracle.draft(w, idx, np.array([200]), v=abs_v(w))
    assert np.all(np.abs(o1 - o2) <= 2 * (4e-3 * oabs + 1e-6))
    ref = oracle.draft(w, idx, np.array([200]))
    check_outputs(o2, ref, oabs, np.ones(ref.shape[:2], dtype=bool), what="draft-reversed")


def test_value_one_gives_one():
    w = generate(303, name="v1", batch=2, n_q_heads=8, n_kv_heads=2, ctx_len=[3000, 100],
                 q_len=[5, 2], budget=256)
    w.v[:] = f32_to_bf16_bits(np.float32(1.0))
    out, s = gpu_verify(Dev(w))
    for b in range(2):
        assert np.abs(out[b, :w.q_len[b]] - 1.0).max() < 2.0 ** -8


@pytest.mark.parametrize("mode", list(MODES))
def test_deterministic_and_stream(mode):
    w, out_ref, s_ref, oabs_ref = small_case("ragged-b3")
    d = Dev(w)
    o1, s1 = gpu_verify(d, mode=MODES[mode])
    o2, s2 = gpu_verify(d, mode=MODES[mode])
    assert np.array_equal(o1, o2) and np.array_equal(s1, s2)
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        o3, s3 = gpu_verify(d, mode=MODES[mode])
    assert np.array_equal(o1, o3) and np.array_equal(s1, s3)


def test_schedules_agree():
    """Both schedules compute the same thing: outputs agree within the bf16
    rounding of P (each rounds against its own running maximum) and scores
    within fp32 rounding."""
    w, out_ref, s_ref, oabs_ref = small_case("tiny-config")
    d = Dev(w)
    o1, s1 = gpu_verify(d, mode=B.VERIFY_TWO_SWEEP)
    o2, s2 = gpu_verify(d, mode=B.VERIFY_ONE_SWEEP)
    mask = _row_mask(w)
    assert np.all(np.abs(o1 - o2)[mask] <= 2 * (4e-3 * oabs_ref[mask] + 1e-6))
    T = int(w.ctx_len[0])
    assert np.abs(s1[..., :T] - s2[..., :T]).max() <= 1e-5 * s_ref[..., :T].max()


# ---------------------------------------------------------------------------
# The five named workloads at full size.
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("n", [1, 2, 3, 4, 5])
def test_workload_full_size(n):
    """Every (sequence, KV head) unit of the workload against the oracle: verify
    outputs and scores element by element, select bit-exact on shared fp32
    scores and by the band rule on the GPU's own scores, draft on all heads."""
    w = make_config(n)
    print(f"[workload {n}] {w.describe()}", flush=True)
    d = Dev(w)
    # bf16 outputs: the benchmark's launch configuration; fp32 outputs: the
    # same kernels without the output's own rounding, at the plain 1e-2 bar
    out, s = gpu_verify(d, out_fp32=False)
    out32, s2 = gpu_verify(d, out_fp32=True)
    print("  gpu verify done; oracle on all units", flush=True)
    out_ref, s_ref = oracle.verify(w)
    oabs_ref, _ = oracle.verify(w, v=abs_v(w))
    err = check_outputs(out, out_ref, oabs_ref, _row_mask(w), out_fp32=False)
    err32 = check_outputs(out32, out_ref, oabs_ref, _row_mask(w), out_fp32=True)
    worst = check_scores(s, s_ref, w.ctx_len)
    check_score_mass(s, w)
    assert np.array_equal(s, s2)
    print(f"  max|dO| bf16 out {err:.2e}, fp32 out {err32:.2e}; worst rel dS={worst:.2e}",
          flush=True)

    # select: bit-exact on shared fp32 scores (the oracle's, rounded to fp32)
    s32 = s_ref.astype(np.float32)
    idx_ref, n_ref = oracle.select(w, s32.astype(np.float64))
    idx, n_idx = gpu_select(w, s32)
    assert np.array_equal(n_idx, n_ref)
    for b in range(w.batch):
        assert np.array_equal(idx[b, :, :n_ref[b]], idx_ref[b, :, :n_ref[b]])
    # select end to end on the GPU's own scores: structure and the band rule
    idx_e, n_e = gpu_select(w, np.where(s < 0, 0.0, s).astype(np.float32))
    check_index_structure(idx_e, n_e, w.ctx_len, w.k_sink, w.k_recent, w.budget)
    check_band(idx_e, n_e, s_ref, w.ctx_len, w.k_sink, w.k_recent, w.budget)
    if "heavy_positions" in w.structure:
        hp = w.structure["heavy_positions"]
        got = sum(int(p) in set(idx_e[b, c, :n_e[b]].tolist())
                  for b in range(w.batch) for c in range(w.n_kv_heads) for p in hp[b, c])
        print(f"  planted heavy hitters selected: {got}/{hp.size}")

    # select and the first draft step in one call
    _check_select_draft(w, s32, out_fp32=False)
    # the whole step in one call (the benchmark's step): one kernel where
    # verify takes one sweep in one round of workgroups of >= 512-key chunks
    # (32K)
    one = check_decode_step(w, out_ref, s_ref, oabs_ref, out_fp32=False)
    assert one == (n == 2)

    # draft on the oracle's index sets, all heads
    idx_dev = np.where(idx_ref < 0, 0, idx_ref).astype(np.int32)
    o_ref = oracle.draft(w, idx_dev, n_ref)
    oabs = oracle.draft(w, idx_dev, n_ref, v=abs_v(w))
    o = gpu_draft(d, idx_dev, n_ref, out_fp32=False)
    check_outputs(o, o_ref, oabs, np.ones(o_ref.shape[:2], dtype=bool), out_fp32=False,
                  what="draft")
