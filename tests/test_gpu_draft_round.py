"""GPU parity of the draft round against the oracle: the sink and TopK rows of
the oracle's index sets are materialized once, then each step attends over them
and the recent window slid to end at the newest drafted token.  The drafted
tokens' K/V rows are cache rows past the base length (the generator fills them
like every other row); the padding past the last step's length holds NaN and
must never be read.  Every step's query is a new seeded draw."""
import numpy as np
import pytest
import torch

import oracle
from gpu_common import abs_v, check_outputs, dev_bf16, params_of
from paper_2607_27735_amd import binding as B
from paper_2607_27735_amd.workloads import f32_to_bf16_bits, generate, make_config

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU visible", allow_module_level=True)

NAN_BF16 = np.uint16(0x7FC0)


def _case(name):
    """(workload, base lengths, drafted steps)."""
    if name == "headline-8b-T32K":
        # the 32K workload; its last six positions play the drafted tokens
        w = make_config(2)
        return w, w.ctx_len - 6, 6
    spec = {
        "small-b2": dict(seed=201, batch=2, n_q_heads=8, n_kv_heads=2, base=[3000, 700], steps=6,
                         budget=300, k_sink=4, k_recent=32),
        "tiny-T": dict(seed=202, batch=4, n_q_heads=8, n_kv_heads=2, base=[1, 5, 17, 33],
                       steps=8, budget=16, k_sink=4, k_recent=8),
        "g16": dict(seed=203, batch=2, n_q_heads=32, n_kv_heads=2, base=[513, 129], steps=5,
                    budget=200, k_sink=4, k_recent=32),
        "window-only": dict(seed=204, batch=1, n_q_heads=8, n_kv_heads=2, base=[100], steps=16,
                            budget=16, k_sink=0, k_recent=16),
        "kv8-ragged": dict(seed=205, batch=3, n_q_heads=32, n_kv_heads=8, base=[2049, 333, 1000],
                           steps=7, budget=256, k_sink=4, k_recent=32),
    }[name]
    base = np.array(spec["base"], dtype=np.int32)
    steps = spec["steps"]
    w = generate(spec["seed"], name=name, batch=spec["batch"], n_q_heads=spec["n_q_heads"],
                 n_kv_heads=spec["n_kv_heads"], ctx_len=list(base + steps),
                 q_len=[1] * spec["batch"], max_ctx=int(base.max()) + steps + 4,
                 budget=spec["budget"], k_sink=spec["k_sink"], k_recent=spec["k_recent"])
    for b in range(w.batch):
        w.k[b, :, base[b] + steps:] = NAN_BF16
        w.v[b, :, base[b] + steps:] = NAN_BF16
    return w, base, steps


NAMES = ["small-b2", "tiny-T", "g16", "window-only", "kv8-ragged", "headline-8b-T32K"]


@pytest.mark.parametrize("name", NAMES)
def test_draft_round_matches_oracle(name):
    _check_round(name)


@pytest.mark.parametrize("cus", [1, 4])
@pytest.mark.parametrize("name", ["small-b2", "kv8-ragged"])
def test_draft_round_wide_workgroups(name, cus):
    """Planned for 1 or 4 CUs, the draft kernels take 512 or 256 entries per
    workgroup (4 or 2 tiles per wave, ragged last tiles) on these small
    rounds: the same bars against the oracle."""
    B.set_cu_budget(cus)
    try:
        _check_round(name)
    finally:
        B.set_cu_budget(0)


def _check_round(name):
    w, base, steps = _case(name)
    print(f"[draft round] {name}: batch {w.batch}, {w.n_q_heads}/{w.n_kv_heads} heads, "
          f"base {list(base)}, {steps} steps, budget {w.budget}", flush=True)
    rng = np.random.default_rng(int(base.sum()) + steps)
    scores = rng.random((w.batch, w.n_kv_heads, w.max_ctx))
    idx, n_idx = oracle.select(w, scores, ctx_len=base)
    p = params_of(w)
    k, v = dev_bf16(w.k), dev_bf16(w.v)
    idx_d = torch.from_numpy(np.ascontiguousarray(idx)).cuda()
    k_sel, v_sel = B.draft_materialize(k, v, idx_d, base, p)
    torch.cuda.synchronize()
    # the materialized rows are the cache rows of the sink and TopK entries, bit for bit
    ks, vs = k_sel.view(torch.int16).cpu().numpy(), v_sel.view(torch.int16).cpu().numpy()
    kc, vc = w.k.view(np.int16), w.v.view(np.int16)
    for b in range(w.batch):
        T = int(base[b])
        r_T = max(T - w.k_recent, min(w.k_sink, T))
        nf = int(n_idx[b]) - (T - r_T)
        for c in range(w.n_kv_heads):
            rows = idx[b, c, :nf]
            assert np.all(rows < r_T)
            assert np.array_equal(ks[b, c, :nf], kc[b, c, rows])
            assert np.array_equal(vs[b, c, :nf], vc[b, c, rows])
    worst = 0.0
    for i in range(steps + 1):
        qb = f32_to_bf16_bits(rng.standard_normal(w.q_draft.shape).astype(np.float32))
        cur = base + i
        o_ref = oracle.draft_step(w, idx, base, cur, q_draft=qb)
        oabs = oracle.draft_step(w, idx, base, cur, q_draft=qb, v=abs_v(w))
        o = B.draft_step(dev_bf16(qb), k, v, base, cur, p, k_sel=k_sel, v_sel=v_sel)
        o_idx = B.draft_step(dev_bf16(qb), k, v, base, cur, p, idx=idx_d)
        torch.cuda.synchronize()
        o = o.float().cpu().numpy().astype(np.float64)
        worst = max(worst, check_outputs(o, o_ref, oabs, np.ones(o_ref.shape[:2], dtype=bool),
                                         what=f"draft step {i}"))
        # the fixed rows through idx: the same rows in the same order, the same result
        assert np.array_equal(o_idx.float().cpu().numpy(), o.astype(np.float32))
        if i == 0:   # before any drafted token the step is the plain draft over idx
            o0 = B.draft_attn(dev_bf16(qb), k, v, idx_d, n_idx, p)
            torch.cuda.synchronize()
            assert np.array_equal(o0.float().cpu().numpy(), o.astype(np.float32))
    print(f"  worst max|dO| over the round = {worst:.2e}")


def test_draft_round_bf16_outputs():
    w, base, steps = _case("small-b2")
    rng = np.random.default_rng(7)
    scores = rng.random((w.batch, w.n_kv_heads, w.max_ctx))
    idx, _ = oracle.select(w, scores, ctx_len=base)
    p = params_of(w, out_fp32=False)
    k, v = dev_bf16(w.k), dev_bf16(w.v)
    k_sel, v_sel = B.draft_materialize(k, v, torch.from_numpy(idx).cuda(), base, p)
    for i in (0, 3, steps):
        o_ref = oracle.draft_step(w, idx, base, base + i)
        oabs = oracle.draft_step(w, idx, base, base + i, v=abs_v(w))
        o = B.draft_step(dev_bf16(w.q_draft), k, v, base, base + i, p, k_sel=k_sel, v_sel=v_sel)
        torch.cuda.synchronize()
        check_outputs(o.float().cpu().numpy().astype(np.float64), o_ref, oabs,
                      np.ones(o_ref.shape[:2], dtype=bool), out_fp32=False, what=f"bf16 step {i}")


def test_draft_round_rejects_long_tail():
    w, base, steps = _case("small-b2")
    p = params_of(w)
    k, v = dev_bf16(w.k), dev_bf16(w.v)
    sel = torch.zeros((w.batch, w.n_kv_heads, w.budget, 128), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(B.SSLError):
        B.draft_step(dev_bf16(w.q_draft), k, v, base, base + w.k_recent + 1, p, k_sel=sel,
                     v_sel=sel)
    with pytest.raises(B.SSLError):
        B.draft_step(dev_bf16(w.q_draft), k, v, base, base - 1, p, k_sel=sel, v_sel=sel)


@pytest.mark.parametrize("page", [32, 128])
@pytest.mark.parametrize("name", ["small-b2", "tiny-T", "kv8-ragged", "headline-8b-T32K"])
def test_paged_draft_round(name, page):
    """The round over a paged cache (shuffled block table, NaN in every pool
    row no table entry names below the round's last length): the materialized
    rows equal the dense ones, and every step, through the index list and from
    the materialized rows, equals the dense round bit for bit and meets the
    oracle's bar."""
    from test_gpu_paged import paged
    w, base, steps = _case(name)
    print(f"[paged draft round] {name}, page {page}", flush=True)
    rng = np.random.default_rng(int(base.sum()) + page)
    scores = rng.random((w.batch, w.n_kv_heads, w.max_ctx))
    idx, n_idx = oracle.select(w, scores, ctx_len=base)
    p = params_of(w)
    k, v = dev_bf16(w.k), dev_bf16(w.v)
    kp, vp, bt, max_blocks = paged(w, page, seed=page + 11)   # the pages hold rows < ctx_len
    kpd, vpd, btd = dev_bf16(kp), dev_bf16(vp), torch.from_numpy(bt).cuda()
    idx_d = torch.from_numpy(np.ascontiguousarray(idx)).cuda()
    k_sel, v_sel = B.draft_materialize(k, v, idx_d, base, p)
    pk_sel, pv_sel = B.draft_materialize_paged(kpd, vpd, btd, w.max_ctx, idx_d, base, p)
    torch.cuda.synchronize()
    for b in range(w.batch):
        T = int(base[b])
        nf = int(n_idx[b]) - (T - max(T - w.k_recent, min(w.k_sink, T)))
        assert torch.equal(pk_sel[b, :, :nf], k_sel[b, :, :nf])
        assert torch.equal(pv_sel[b, :, :nf], v_sel[b, :, :nf])
    for i in range(steps + 1):
        qb = f32_to_bf16_bits(rng.standard_normal(w.q_draft.shape).astype(np.float32))
        qd = dev_bf16(qb)
        cur = base + i
        o_dense = B.draft_step(qd, k, v, base, cur, p, idx=idx_d)
        o_pi = B.draft_step_paged(qd, kpd, vpd, btd, w.max_ctx, base, cur, p, idx=idx_d)
        o_ps = B.draft_step_paged(qd, kpd, vpd, btd, w.max_ctx, base, cur, p, k_sel=pk_sel,
                                  v_sel=pv_sel)
        torch.cuda.synchronize()
        assert torch.equal(o_pi, o_dense), f"step {i}: paged (index list) differs from dense"
        assert torch.equal(o_ps, o_dense), f"step {i}: paged (materialized) differs from dense"
        o_ref = oracle.draft_step(w, idx, base, cur, q_draft=qb)
        oabs = oracle.draft_step(w, idx, base, cur, q_draft=qb, v=abs_v(w))
        check_outputs(o_ps.float().cpu().numpy().astype(np.float64), o_ref, oabs,
                      np.ones(o_ref.shape[:2], dtype=bool), what=f"paged draft step {i}")
