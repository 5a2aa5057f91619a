"""GPU parity of the paged KV cache: the dense workload's K/V rows are placed
in a page pool under a shuffled block table; verify (both schedules) and draft
over the pages must match the oracle on the dense layout at the usual bars,
and the dense GPU path bit for bit (same arithmetic in the same order).  Pool
pages no block table names, table entries past a sequence's pages, and rows
past a sequence's length in its last page hold NaN: none may be used."""
import numpy as np
import pytest
import torch

import oracle
from gpu_common import (Dev, abs_v, check_outputs, check_scores, dev_bf16, gpu_draft, gpu_verify,
                        params_of)
from paper_2607_27735_amd import binding as B
from paper_2607_27735_amd.workloads import generate, make_config

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU visible", allow_module_level=True)

NAN_BF16 = np.uint16(0x7FC0)


def paged(w, page, seed, spare=5):
    """(k_pages, v_pages, block_table, max_blocks): pages [n, Hkv, page, 128]."""
    rng = np.random.default_rng(seed)
    max_blocks = (w.max_ctx + page - 1) // page
    need = [(int(t) + page - 1) // page for t in w.ctx_len]
    n_pages = sum(need) + spare + 1
    perm = rng.permutation(n_pages - 1)      # the last page is the NaN page
    nan_page = n_pages - 1
    kp = np.full((n_pages, w.n_kv_heads, page, w.head_dim), NAN_BF16, dtype=np.uint16)
    vp = kp.copy()
    bt = np.full((w.batch, max_blocks), nan_page, dtype=np.int32)
    nxt = 0
    for b in range(w.batch):
        T = int(w.ctx_len[b])
        for j in range(need[b]):
            pg = int(perm[nxt]); nxt += 1
            bt[b, j] = pg
            lo, hi = j * page, min((j + 1) * page, T)
            kp[pg, :, :hi - lo] = w.k[b, :, lo:hi]
            vp[pg, :, :hi - lo] = w.v[b, :, lo:hi]
    return kp, vp, bt, max_blocks


def _cases():
    return {
        "ragged-b3-p64": (lambda: generate(401, name="ragged-b3", batch=3, n_q_heads=8,
                                           n_kv_heads=2, ctx_len=[1000, 333, 2049],
                                           q_len=[3, 1, 7], max_ctx=2100, max_q=8, budget=256), 64),
        "tiny-T-p32": (lambda: generate(402, name="tiny-T", batch=4, n_q_heads=8, n_kv_heads=2,
                                        ctx_len=[1, 5, 17, 33], q_len=[1, 5, 3, 2], budget=16,
                                        k_sink=4, k_recent=8, max_ctx=40), 32),
        "rows48-g8-p256": (lambda: generate(403, name="rows48", batch=2, n_q_heads=16,
                                            n_kv_heads=2, ctx_len=[3000, 700], q_len=[6, 6],
                                            budget=200), 256),
        "llama8b-T32K-p128": (lambda: make_config(2), 128),
    }


CASES = _cases()
MODES = {"two-sweep": B.VERIFY_TWO_SWEEP, "one-sweep": B.VERIFY_ONE_SWEEP}


@pytest.mark.parametrize("mode", list(MODES))
@pytest.mark.parametrize("name", list(CASES))
def test_paged_verify_and_draft(name, mode):
    make, page = CASES[name]
    w = make()
    print(f"[paged] {name}, page {page}, {mode}", flush=True)
    kp, vp, bt, max_blocks = paged(w, page, seed=len(name) * 7 + page)
    out_ref, s_ref = oracle.verify(w)
    oabs, _ = oracle.verify(w, v=abs_v(w))
    p = params_of(w, mode=MODES[mode])
    d = Dev(w)
    kpd, vpd = dev_bf16(kp), dev_bf16(vp)
    btd = torch.from_numpy(bt).cuda()
    out, sc = B.verify_attn_paged(d.q, kpd, vpd, btd, w.max_ctx, w.ctx_len, w.q_len, p)
    torch.cuda.synchronize()
    out = out.float().cpu().numpy().astype(np.float64)
    sc = sc.cpu().numpy().astype(np.float64)
    mask = np.arange(w.max_q)[None, :, None] < w.q_len[:, None, None] * np.ones((1, 1, w.n_q_heads), bool)
    check_outputs(out, out_ref, oabs, mask, what="paged verify O")
    check_scores(sc, s_ref, w.ctx_len, what="paged verify S")
    # the dense path, bit for bit
    out_d, sc_d = gpu_verify(d, mode=MODES[mode])
    assert np.array_equal(out[mask], out_d[mask])
    for b in range(w.batch):
        assert np.array_equal(sc[b, :, :w.ctx_len[b]], sc_d[b, :, :w.ctx_len[b]])
    if mode != "two-sweep":
        return
    # draft over the pages: the oracle's index sets on the fp32 scores
    idx_ref, n_ref = oracle.select(w, s_ref.astype(np.float32).astype(np.float64))
    idx_dev = np.where(idx_ref < 0, 0, idx_ref).astype(np.int32)
    o_ref = oracle.draft(w, idx_dev, n_ref)
    oa = oracle.draft(w, idx_dev, n_ref, v=abs_v(w))
    o = B.draft_attn_paged(d.qd, kpd, vpd, btd, w.max_ctx, torch.from_numpy(idx_dev).cuda(),
                           n_ref, p)
    torch.cuda.synchronize()
    o = o.float().cpu().numpy().astype(np.float64)
    od = gpu_draft(d, idx_dev, n_ref)
    check_outputs(o, o_ref, oa, np.ones(o_ref.shape[:2], dtype=bool), what="paged draft")
    assert np.array_equal(o, od)
    # planned for one CU: 512 entries per workgroup (4 tiles per wave)
    B.set_cu_budget(1)
    try:
        o4 = B.draft_attn_paged(d.qd, kpd, vpd, btd, w.max_ctx, torch.from_numpy(idx_dev).cuda(),
                                n_ref, p)
        torch.cuda.synchronize()
        od4 = gpu_draft(d, idx_dev, n_ref)
    finally:
        B.set_cu_budget(0)
    o4 = o4.float().cpu().numpy().astype(np.float64)
    check_outputs(o4, o_ref, oa, np.ones(o_ref.shape[:2], dtype=bool), what="paged draft, wide")
    assert np.array_equal(o4, od4)
