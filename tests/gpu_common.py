"""Helpers for the GPU parity tests: device upload of generated inputs, calls
through the C-ABI binding, and the tolerance checks.

Tolerances (bf16 inputs, fp32 accumulation):

* outputs: the stated bar is max |O - O_ref| <= 1e-2 for fp32 outputs, plus
  half a bf16 ulp of the output for bf16 outputs.  A tighter per-element
  bound follows from the arithmetic: the only rounding larger than fp32's is
  that of the probabilities to bf16 before the P.V product (8 significant
  bits, round to nearest: relative error at most 2^-8), so
  |O - O_ref| <= 2^-8 * sum_i P_i |v_i| plus fp32 terms; the tests allow
  4e-3 * sum_i P_i |v_i| + 1e-6, with sum_i P_i |v_i| from the oracle run on
  |V| (plus 2^-8 |O_ref| when outputs are bf16);
* scores: |S - S_ref| <= 1e-3 * S_ref for every key with S_ref > 0;
* index sets: bit-exact against the oracle's select run on the same fp32
  scores; against the oracle's fp64 scores, the band rule: every middle
  position with S_ref > tau (1 + 1e-3) is selected, none with
  S_ref < tau (1 - 1e-3) is, the middle count is exact, and sink and recent
  are exact (tau = the K_mid-th largest reference middle score).
"""
from __future__ import annotations

import numpy as np
import torch

import oracle
from paper_2607_27735_amd import binding as B


def dev_bf16(bits: np.ndarray) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16).copy())
    return t.view(torch.bfloat16).cuda()


def params_of(w, out_fp32=True, budget=None, k_sink=None, k_recent=None, window=None,
              mode=B.VERIFY_AUTO):
    return B.make_params(w.sm_scale, window=w.window if window is None else window,
                         k_sink=w.k_sink if k_sink is None else k_sink,
                         k_recent=w.k_recent if k_recent is None else k_recent,
                         budget=w.budget if budget is None else budget, out_fp32=out_fp32,
                         verify_mode=mode)


class Dev:
    """A workload's tensors on the GPU."""

    def __init__(self, w):
        self.w = w
        self.q = dev_bf16(w.q)
        self.k = dev_bf16(w.k)
        self.v = dev_bf16(w.v)
        self.qd = dev_bf16(w.q_draft)


def gpu_verify(d: Dev, out_fp32=True, scores_fill=-1.0, out_fill=-7.0, window=None,
               mode=B.VERIFY_AUTO):
    w = d.w
    p = params_of(w, out_fp32=out_fp32, window=window, mode=mode)
    odt = torch.float32 if out_fp32 else torch.bfloat16
    out = torch.full(d.q.shape, out_fill, dtype=odt, device="cuda")
    sc = torch.full((w.batch, w.n_kv_heads, w.max_ctx), scores_fill, dtype=torch.float32,
                    device="cuda")
    B.verify_attn(d.q, d.k, d.v, w.ctx_len, w.q_len, p, out=out, scores=sc)
    torch.cuda.synchronize()
    return out.float().cpu().numpy().astype(np.float64), sc.cpu().numpy().astype(np.float64)


def gpu_select(w, scores32: np.ndarray, ctx_len=None, budget=None, k_sink=None, k_recent=None,
               idx_fill=-7):
    p = params_of(w, budget=budget, k_sink=k_sink, k_recent=k_recent)
    s = torch.from_numpy(np.ascontiguousarray(scores32, dtype=np.float32)).cuda()
    idx = torch.full((w.batch, w.n_kv_heads, p.budget), idx_fill, dtype=torch.int32,
                     device="cuda")
    n_idx = torch.full((w.batch,), -1, dtype=torch.int32, device="cuda")
    B.select_topb(s, w.ctx_len if ctx_len is None else ctx_len, p, n_q_heads=w.n_q_heads,
                  idx=idx, n_idx=n_idx)
    torch.cuda.synchronize()
    return idx.cpu().numpy(), n_idx.cpu().numpy()


def gpu_draft(d: Dev, idx: np.ndarray, n_idx: np.ndarray, out_fp32=True, budget=None):
    w = d.w
    p = params_of(w, out_fp32=out_fp32, budget=budget)
    it = torch.from_numpy(np.ascontiguousarray(idx, dtype=np.int32)).cuda()
    out = B.draft_attn(d.qd, d.k, d.v, it, n_idx, p)
    torch.cuda.synchronize()
    return out.float().cpu().numpy().astype(np.float64)


def abs_v(w) -> np.ndarray:
    """|V| as bf16 bits (clearing the sign bit is exact)."""
    return (w.v & np.uint16(0x7FFF)).astype(np.uint16)


def half_ulp_bf16(x: np.ndarray) -> np.ndarray:
    """Half the spacing of bf16 numbers (8 significant bits) at |x|."""
    ax = np.abs(np.asarray(x, dtype=np.float64))
    e = np.floor(np.log2(np.where(ax > 0, ax, 1.0)))
    return np.where(ax > 0, np.exp2(e - 8), 0.0)


def check_outputs(o_gpu, o_ref, oabs_ref, rows_mask, out_fp32=True, what="O"):
    """rows_mask: boolean array broadcastable to o_ref[..., 0] selecting checked rows.

    fp32 outputs: max |dO| <= 1e-2.  bf16 outputs add the rounding of the
    output itself, half a bf16 ulp, taken at the larger of |O| and |O_ref|
    (a rounded value is never in a lower binade than the value rounded)."""
    sel = np.broadcast_to(rows_mask[..., None], o_ref.shape)
    diff = np.abs(o_gpu - o_ref)[sel]
    assert np.all(np.isfinite(o_gpu[sel])), f"{what}: non-finite outputs"
    maxabs = float(diff.max()) if diff.size else 0.0
    if out_fp32:
        assert maxabs <= 1e-2, f"{what}: max |dO| = {maxabs:.3e} > 1e-2"
    else:
        bar = 1e-2 + half_ulp_bf16(np.maximum(np.abs(o_gpu), np.abs(o_ref)))[sel]
        worst = float((diff - bar).max()) if diff.size else -1.0
        assert worst <= 0, (f"{what}: max |dO| = {maxabs:.3e}; exceeds 1e-2 + half a bf16 ulp by "
                            f"{worst:.3e}")
    bound = 4e-3 * oabs_ref + 1e-6
    if not out_fp32:
        bound = bound + 2.0 ** -8 * np.abs(o_ref)
    bad = (np.abs(o_gpu - o_ref) > bound) & sel
    assert not bad.any(), (f"{what}: {int(bad.sum())} elements beyond the derived bound; worst "
                           f"excess {float((np.abs(o_gpu - o_ref) - bound)[bad].max()):.3e}")
    return maxabs


def check_scores(s_gpu, s_ref, ctx_len, units=None, what="S"):
    batch, hkv, _ = s_ref.shape
    worst = 0.0
    for b in range(batch):
        T = int(ctx_len[b])
        for c in range(hkv):
            if units is not None and b * hkv + c not in units:
                continue
            g, r = s_gpu[b, c, :T], s_ref[b, c, :T]
            pos = r > 0
            rel = np.abs(g - r)[pos] / r[pos]
            if rel.size:
                worst = max(worst, float(rel.max()))
            assert np.all(g[~pos] == 0.0), f"{what}: nonzero score where the reference is 0"
    assert worst <= 1e-3, f"{what}: worst relative score error {worst:.3e} > 1e-3"
    return worst


def check_score_mass(s_gpu, w, units=None):
    for b in range(w.batch):
        T, nq = int(w.ctx_len[b]), int(w.q_len[b])
        want = min(w.window, nq) * w.group
        for c in range(w.n_kv_heads):
            if units is not None and b * w.n_kv_heads + c not in units:
                continue
            tot = float(np.sum(s_gpu[b, c, :T], dtype=np.float64))
            assert abs(tot - want) <= 2e-5 * want, f"score mass {tot} != {want} (b={b}, c={c})"


def spans(T, ks, kr):
    s_end = min(ks, T)
    r_start = max(T - kr, s_end)
    return s_end, r_start


def check_index_structure(idx, n_idx, ctx_len, ks, kr, budget, idx_fill=-7):
    batch, hkv, _ = idx.shape
    for b in range(batch):
        T = int(ctx_len[b])
        n = oracle.index_count(T, ks, kr, budget)
        assert n_idx[b] == n, f"n_idx[{b}] = {n_idx[b]} != {n}"
        s_end, r_start = spans(T, ks, kr)
        for c in range(hkv):
            row = idx[b, c, :n]
            assert np.all(np.diff(row) > 0) and row[0] >= 0 and row[-1] < T
            assert np.array_equal(row[:s_end], np.arange(s_end))
            assert np.array_equal(row[n - (T - r_start):], np.arange(r_start, T))
            assert np.all(idx[b, c, n:] == idx_fill), "wrote past n_idx"


def check_band(idx, n_idx, s_ref, ctx_len, ks, kr, budget, eps=1e-3, units=None):
    batch, hkv, _ = idx.shape
    k_mid = budget - ks - kr
    for b in range(batch):
        T = int(ctx_len[b])
        s_end, r_start = spans(T, ks, kr)
        take = min(k_mid, r_start - s_end)
        for c in range(hkv):
            if units is not None and b * hkv + c not in units:
                continue
            n = int(n_idx[b])
            chosen = np.zeros(T, dtype=bool)
            chosen[idx[b, c, :n]] = True
            m = chosen[s_end:r_start]
            assert int(m.sum()) == take, "middle count"
            if take == r_start - s_end:
                continue
            mid = s_ref[b, c, s_end:r_start]
            tau = float(np.partition(mid, len(mid) - take)[len(mid) - take])
            assert np.all(m[mid > tau * (1 + eps)]), "clearly-above position missing"
            assert not np.any(m[mid < tau * (1 - eps)]), "clearly-below position selected"


def gpu_select_draft(d: Dev, scores32: np.ndarray, out_fp32=True, budget=None, k_sink=None,
                     k_recent=None, ctx_len=None):
    """ssl_select_draft on the given fp32 scores: (idx, n_idx, draft out)."""
    w = d.w
    p = params_of(w, out_fp32=out_fp32, budget=budget, k_sink=k_sink, k_recent=k_recent)
    s = torch.from_numpy(np.ascontiguousarray(scores32, dtype=np.float32)).cuda()
    idx = torch.full((w.batch, w.n_kv_heads, p.budget), -7, dtype=torch.int32, device="cuda")
    n_idx = torch.full((w.batch,), -1, dtype=torch.int32, device="cuda")
    odt = torch.float32 if out_fp32 else torch.bfloat16
    out = torch.full(d.qd.shape, -7.0, dtype=odt, device="cuda")
    B.select_draft(s, w.ctx_len if ctx_len is None else ctx_len, p, d.qd, d.k, d.v, idx=idx,
                   n_idx=n_idx, out=out)
    torch.cuda.synchronize()
    return idx.cpu().numpy(), n_idx.cpu().numpy(), out.float().cpu().numpy().astype(np.float64)


def gpu_decode_step(d: Dev, out_fp32=True, budget=None, k_sink=None, k_recent=None, mode=B.VERIFY_AUTO):
    """ssl_decode_step into sentinel-filled outputs: (out, scores, idx, n_idx,
    draft out) on the host, outputs as float64."""
    w = d.w
    p = params_of(w, out_fp32=out_fp32, budget=budget, k_sink=k_sink, k_recent=k_recent, mode=mode)
    odt = torch.float32 if out_fp32 else torch.bfloat16
    out = torch.full(d.q.shape, -7.0, dtype=odt, device="cuda")
    sc = torch.full((w.batch, w.n_kv_heads, w.max_ctx), -1.0, dtype=torch.float32, device="cuda")
    idx = torch.full((w.batch, w.n_kv_heads, p.budget), -7, dtype=torch.int32, device="cuda")
    n_idx = torch.full((w.batch,), -1, dtype=torch.int32, device="cuda")
    dout = torch.full(d.qd.shape, -7.0, dtype=odt, device="cuda")
    B.decode_step(d.q, d.k, d.v, d.qd, w.ctx_len, w.q_len, p, out=out, scores=sc, idx=idx,
                  n_idx=n_idx, draft_out=dout)
    torch.cuda.synchronize()
    f64 = lambda t: t.float().cpu().numpy().astype(np.float64)
    return f64(out), sc.cpu().numpy(), idx.cpu().numpy(), n_idx.cpu().numpy(), f64(dout)


def check_decode_step(w, out_ref, s_ref, oabs_ref, out_fp32=True, budget=None, k_sink=None,
                      k_recent=None, expect_one_kernel=None):
    """ssl_decode_step against verify_attn (bit for bit) and the oracle (see
    test_gpu_decode_step); returns whether the step ran as one kernel."""
    d = Dev(w)
    p = params_of(w, out_fp32=out_fp32, budget=budget, k_sink=k_sink, k_recent=k_recent)
    one = B.decode_step_plan(B.verify_shape(d.q, d.k), p, w.ctx_len, w.q_len)
    print(f"[decode step] {w.describe()} one kernel: {one}", flush=True)
    if expect_one_kernel is not None:
        assert one == expect_one_kernel
    out, s, idx, n_idx, dout = gpu_decode_step(d, out_fp32=out_fp32, budget=budget, k_sink=k_sink,
                                               k_recent=k_recent)
    # verify: the same arithmetic as verify_attn, and the oracle's bars
    out_v, s_v = gpu_verify(d, out_fp32=out_fp32)
    mask = np.arange(w.max_q)[None, :, None] < w.q_len[:, None, None] * np.ones(
        (1, 1, w.n_q_heads), dtype=bool)
    assert np.array_equal(out[mask], out_v[mask]), "outputs differ from verify_attn"
    for b in range(w.batch):
        T = int(w.ctx_len[b])
        assert np.array_equal(s[b, :, :T], s_v[b, :, :T]), "scores differ from verify_attn"
        assert np.all(s[b, :, T:] == -1.0)
    assert np.all(out[~mask] == -7.0)
    check_outputs(out, out_ref, oabs_ref, mask, out_fp32=out_fp32)
    check_scores(s, s_ref, w.ctx_len)
    check_score_mass(s, w)
    # select: bit-exact against the oracle's select on the step's own scores
    ks = w.k_sink if k_sink is None else k_sink
    kr = w.k_recent if k_recent is None else k_recent
    bud = w.budget if budget is None else budget
    idx_ref, n_ref = oracle.select(w, s.astype(np.float64), budget=bud, k_sink=ks, k_recent=kr)
    assert np.array_equal(n_idx, n_ref)
    for b in range(w.batch):
        assert np.array_equal(idx[b, :, :n_ref[b]], idx_ref[b, :, :n_ref[b]])
    check_index_structure(idx, n_idx, w.ctx_len, ks, kr, bud)
    # draft over those index sets
    idx_dev = np.where(idx_ref < 0, 0, idx_ref).astype(np.int32)
    o_ref = oracle.draft(w, idx_dev, n_ref)
    oabs = oracle.draft(w, idx_dev, n_ref, v=abs_v(w))
    check_outputs(dout, o_ref, oabs, np.ones(o_ref.shape[:2], dtype=bool), out_fp32=out_fp32,
                  what="decode-step draft")
    return one
