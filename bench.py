#!/usr/bin/env python3
"""Benchmark of one SparseSpec-L decode-step hot path (one layer) on one GPU.

A step is verify attention with score emission, top-B selection and one draft
attention step (at this workload one call of the C ABI, ssl_decode_step, which
runs them in one kernel), over the Llama-3-8B-shaped 32K-context workload (batch 1, 32 query / 8 KV heads, head_dim 128, k = 6,
B = 2048, four planted heavy-hitter keys per KV head).  Inputs are seeded and
synthetic and already resident in HBM when timing starts.

Every step reads a different copy of the KV cache (enough copies that each
step's cache was last touched more than 512 MiB earlier, and that the rows a
draft gathers from a copy were last gathered more than 512 MiB of such rows
earlier, up to 256 copies), so the 256 MB Infinity Cache cannot serve it and
the numbers are HBM numbers.

Prints one JSON line: µs per step (lower is better), per-call times from HIP
events on the launch stream, the verify call against the HBM roofline, and the
CPU oracle timed on the host's cores on the same workload.
"""
from __future__ import annotations

import argparse
import gc
import json
import math
import os
import statistics
import sys
import time

METRIC = "µs per verify+select+draft step and HBM GB/s (% of peak) at 32K ctx, 1 GPU"
HBM_PEAK_GBPS = 8000.0


def algorithmic_bytes(w, out_bytes: int):
    """Bytes each call must move at least once (see the design notes)."""
    hkv, hq, d = w.n_kv_heads, w.n_q_heads, w.head_dim
    T = [int(t) for t in w.ctx_len]
    q = [int(x) for x in w.q_len]
    from paper_2607_27735_amd.binding import index_count
    n = [index_count(t, w.k_sink, w.k_recent, w.budget) for t in T]
    verify = sum(hkv * t * d * 2 * 2 + hkv * t * 4 for t in T) + \
        sum(qb * hq * d * 2 + qb * hq * d * out_bytes for qb in q)
    select = sum(hkv * t * 4 + hkv * nb * 4 for t, nb in zip(T, n)) + 4 * w.batch
    draft = sum(hkv * nb * (d * 2 * 2 + 4) for nb in n) + w.batch * hq * d * (2 + out_bytes)
    return {"verify": verify, "select": select, "draft": draft}, n


def kv_copies(w, kv_bytes: int) -> int:
    """KV copies to rotate: each call's cache bytes, and each draft's gathered
    rows, last touched more than 512 MiB (twice the Infinity Cache) earlier;
    at least 2, at most 256."""
    draft = algorithmic_bytes(w, out_bytes=2)[0]["draft"]
    need = max(math.ceil((512 << 20) / kv_bytes), math.ceil((512 << 20) / max(draft, 1))) + 1
    return int(min(256, max(2, need)))


REPO = os.path.dirname(os.path.abspath(__file__))
TRAFFIC_FILE = os.path.join(REPO, "profiles", "verify_traffic_llama8b_T32K.txt")
OUR_KERNELS = ("verify_fused_kernel", "verify_pipe_kernel", "verify_stats_kernel", "verify_main_kernel",
               "verify_combine_kernel", "select_hist_kernel", "select_mark_kernel",
               "select_finish_kernel", "select_fused_kernel", "draft_materialize_kernel",
               "draft_kernel", "logit_stats_kernel", "greedy_accept_kernel", "spec_stats_kernel",
               "spec_rows_kernel", "spec_decide_kernel", "spec_mass_kernel", "spec_sample_kernel")
VERIFY_KERNELS = ("verify_fused_kernel", "verify_pipe_kernel", "verify_stats_kernel", "verify_main_kernel",
                  "verify_combine_kernel")


def sources_sha256() -> str:
    """Hash of the HIP/C++ sources and the ABI header, in a fixed order."""
    import hashlib
    h = hashlib.sha256()
    dirs = [os.path.join(REPO, "paper_2607_27735_amd", "csrc"), os.path.join(REPO, "include")]
    for d in dirs:
        for name in sorted(os.listdir(d)):
            if name.endswith((".hip", ".h", ".cpp")):
                h.update(name.encode())
                with open(os.path.join(d, name), "rb") as f:
                    h.update(f.read())
    return h.hexdigest()


def kernel_short(name: str) -> str:
    for k in OUR_KERNELS:
        if k in name:
            return k + ("<" + name.split("<", 1)[1].split(">", 1)[0] + ">" if "<" in name else "")
    return name


def is_paged(short: str) -> bool:
    """Whether a kernel (short name with template arguments) is the paged-cache
    instance: the last template flag of the verify kernels, mode 3 of the draft."""
    if "<" not in short:
        return False
    args = [x.strip() for x in short.split("<", 1)[1].rstrip(">").split(",")]
    k = short.split("<")[0]
    if k == "verify_fused_kernel":   # <row tiles, stream, paged, whole step>
        return len(args) >= 3 and args[2] == "true"
    if k in ("verify_stats_kernel", "verify_main_kernel", "verify_pipe_kernel"):
        return len(args) == 2 and args[1] == "true"
    return k == "draft_kernel" and args[0] == "3"


def is_step_kernel(short: str) -> bool:
    """Whether a kernel (short name with template arguments) is the one-kernel
    decode step: the verify kernel's fourth template flag."""
    if not short.startswith("verify_fused_kernel<"):
        return False
    args = [x.strip() for x in short.split("<", 1)[1].rstrip(">").split(",")]
    return len(args) == 4 and args[3] == "true"


def summarize_trace(d: str, command: str, title: str = "") -> str:
    """Markdown table of a rocprofv3 --kernel-trace --stats run."""
    import csv
    import glob
    f = glob.glob(os.path.join(d, "**", "*kernel_stats.csv"), recursive=True)[0]
    rows = [r for r in csv.DictReader(open(f)) if any(k in r["Name"] for k in OUR_KERNELS)]
    out = ([f"# Kernel trace: {title}", ""] if title else []) + [f"command: `{command}`", "",
           "| kernel | calls | avg us | min us | max us |", "|---|---:|---:|---:|---:|"]
    for r in sorted(rows, key=lambda r: -float(r["AverageNs"])):
        out.append(f"| {kernel_short(r['Name'])} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} "
                   f"| {float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} |")
    per_call = {}
    for r in rows:
        short = kernel_short(r["Name"])
        k = short.split("<")[0]
        mode = short.split("<", 1)[1].split(",")[0].strip(" >") if "<" in short else ""
        sel_draft = k == "select_fused_kernel" and short.rstrip(">").endswith("true")
        call = ("decode step (one kernel)" if is_step_kernel(short)
                else "select + first draft step (one kernel)" if sel_draft
                else "verify (paged)" if k.startswith("verify") and is_paged(short)
                else "draft (paged)" if is_paged(short)
                else "verify" if k.startswith("verify") else "select" if k.startswith("select")
                else "draft round materialize" if "materialize" in k
                else "draft round step (index list)" if k == "draft_kernel" and mode == "1"
                else "draft round step (materialized rows)" if k == "draft_kernel" and mode == "2"
                else "logit statistics" if k.startswith("logit")
                else "greedy acceptance" if k.startswith("greedy")
                else "speculative sampling" if k.startswith("spec_") else "draft")
        per_call[call] = per_call.get(call, 0.0) + float(r["AverageNs"]) / 1e3
    out += ["", "sum of kernel averages per call: " +
            ", ".join(f"{c} {v:.2f} us" for c, v in per_call.items())]
    return "\n".join(out) + "\n"


def back_to_back_us(fn, reps: int, stream, torch) -> float:
    """Average duration of the calls fn(0), ..., fn(reps - 1) issued back to
    back, between two HIP events on ``stream``.  One untimed call, fn(-1)
    (the input copy that precedes the first in rotation order), goes first, so
    that the region starts with the stream busy: it then holds the calls
    alone, not the host's latency to its first launch."""
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    fn(-1)
    e0.record(stream)
    for r in range(reps):
        fn(r)
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e3 / reps


def graph_step_bench(B, kvs, q, qd, w, params, out, scores, idx, n_idx, dout, stream, reps, torch):
    """The same step captured in a HIP graph, one graph per KV copy: K replays
    back to back, wall clock between two synchronizations."""
    cap = torch.cuda.Stream()
    cap.wait_stream(stream)
    graphs = []
    for (k, v) in kvs:
        with torch.cuda.stream(cap):
            st = B.PreparedStep(q, k, v, qd, w.ctx_len, w.q_len, params, out, scores, idx, n_idx,
                                dout, stream=cap)
            st.step()   # eager warm-up on the capture stream
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=cap):
            st.step()
        graphs.append((g, st))
    stream.wait_stream(cap)
    torch.cuda.synchronize()
    for g, _ in graphs:
        g.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(reps):
        graphs[i % len(graphs)][0].replay()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    return {"step_us": round((t1 - t0) * 1e6 / reps, 3),
            "timing": f"{reps} replays back to back of one captured step graph per KV copy "
                      f"({len(graphs)} copies), wall clock between two synchronizations"}


def draft_round_bench(B, w, kvs, qd, params, scores, stream, reps, torch, np):
    """A draft round on the workload (next to the headline, not part of it):
    the index sets are built at T - k (k = max q_len - 1, at most K_recent),
    so that the last k cached positions play the drafted tokens; then one
    materialization and the steps at lengths T - k + i, each timed as
    ``reps`` back-to-back calls (rotating the KV copies and their own
    materialized rows) between two HIP events, beside the plain draft call
    over the same index lists."""
    k = max(1, min(int(max(w.q_len)) - 1, w.k_recent))
    base = np.maximum(w.ctx_len - k, 1).astype(np.int32)
    dev = qd.device
    idx = torch.zeros((w.batch, w.n_kv_heads, w.budget), dtype=torch.int32, device=dev)
    n_idx = torch.zeros(w.batch, dtype=torch.int32, device=dev)
    B.select_topb(scores, base, params, n_q_heads=w.n_q_heads, idx=idx, n_idx=n_idx,
                  stream=stream)
    n_host = [B.index_count(int(t), w.k_sink, w.k_recent, w.budget) for t in base]
    out = torch.empty(qd.shape, dtype=torch.bfloat16, device=dev)
    sel_shape = (w.batch, w.n_kv_heads, w.budget, w.head_dim)
    rounds = [B.PreparedRound(qd, kk, vv, idx, base, k, params, out, stream=stream)
              for (kk, vv) in kvs]
    mats = [B.PreparedRound(qd, kk, vv, idx, base, k, params, out,
                            k_sel=torch.empty(sel_shape, dtype=torch.bfloat16, device=dev),
                            v_sel=torch.empty(sel_shape, dtype=torch.bfloat16, device=dev),
                            stream=stream) for (kk, vv) in kvs]
    n = len(rounds)
    dshape = B.Shape(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.max_ctx, 1)
    dws = torch.empty(max(B.draft_workspace_bytes(dshape, params, n_host), 1), dtype=torch.uint8,
                      device=dev)

    def timed(fn):
        for r in range(n):
            fn(r)
        return back_to_back_us(fn, reps, stream, torch)

    step_us = [timed(lambda r, i=i: rounds[r % n].step(i)) for i in range(k)]
    mat_us = timed(lambda r: mats[r % n].materialize())
    mstep_us = [timed(lambda r, i=i: mats[r % n].step(i)) for i in range(k)]
    # the plain draft call, prepared like the round's calls (one ctypes call each)
    import ctypes
    lib = B.load()
    n_arr = np.array(n_host, dtype=np.int32)
    dargs = [(ctypes.byref(dshape), ctypes.byref(params), n_arr.ctypes.data_as(B._i32p),
              qd.data_ptr(), kk.data_ptr(), vv.data_ptr(), idx.data_ptr(), out.data_ptr(),
              dws.data_ptr(), dws.numel(), B._stream(stream)) for (kk, vv) in kvs]
    for a in dargs:
        B._check(lib.ssl_draft_attn(*a), "ssl_draft_attn")
    draft_us = timed(lambda r: lib.ssl_draft_attn(*dargs[r % n]))
    entries = sum(n_host) * w.n_kv_heads
    step_bytes = entries * (w.head_dim * 2 * 2) + w.batch * w.n_q_heads * w.head_dim * 4
    mean_step = statistics.fmean(step_us)
    return {"k": k, "base_len": list(map(int, base)),
            "step_us": [round(x, 3) for x in step_us], "step_us_mean": round(mean_step, 3),
            "round_us": round(sum(step_us), 3),
            "plain_draft_us": round(draft_us, 3),
            "materialize_us": round(mat_us, 3),
            "materialized_step_us_mean": round(statistics.fmean(mstep_us), 3),
            "materialized_round_us": round(mat_us + sum(mstep_us), 3),
            "step_alg_bytes": step_bytes,
            "step_gbps": round(step_bytes / (mean_step * 1e-6) / 1e9, 1),
            "timing": f"{reps} back-to-back calls per figure between two HIP events "
                      f"(after one untimed call), "
                      f"rotating {n} KV copies"}


def vocab_side_bench(B, w, stream, reps, torch, np, vocab=128256):
    """The token statistics around the path at this workload's step (next to
    the headline, not part of it): draft entropies over k = max q_len - 1 draft
    rows and greedy acceptance over the k + 1 verify rows of every sequence,
    synthetic seeded bf16 logits over a Llama-3-sized vocabulary, each timed
    as ``reps`` back-to-back calls (rotating copies beyond the 256 MB cache)
    between two HIP events."""
    import ctypes
    from paper_2607_27735_amd.workloads import f32_to_bf16_bits
    k = max(1, int(max(w.q_len)) - 1)
    rng = np.random.default_rng(2024)
    dev = torch.device("cuda:0")
    draft_rows = w.batch * k
    verify_rows = w.batch * (k + 1)
    x = f32_to_bf16_bits((rng.standard_normal((verify_rows, vocab)) * 2.0).astype(np.float32))
    logits = torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).to(dev)
    copy_bytes = logits.numel() * 2
    n = max(2, math.ceil((512 << 20) / copy_bytes) + 1)
    copies = [logits] + [logits.clone() for _ in range(n - 1)]
    lib = B.load()
    # draft entropies: the first k rows of each copy stand for the draft logits
    ent = torch.empty(draft_rows, dtype=torch.float32, device=dev)
    nws = ctypes.c_size_t(0)
    B._check(lib.ssl_logit_stats_workspace(draft_rows, vocab, ctypes.byref(nws)), "ws")
    ws1 = torch.empty(max(nws.value, 1), dtype=torch.uint8, device=dev)
    sargs = [(c.data_ptr(), B.SSL_DT_BF16, draft_rows, vocab, vocab, ent.data_ptr(), None,
              ws1.data_ptr(), ws1.numel(), B._stream(stream)) for c in copies]
    # acceptance: drafts agree with the verify argmax for the first half of each sequence
    k_len = np.full(w.batch, k, dtype=np.int32)
    draft = torch.zeros((w.batch, k), dtype=torch.int32, device=dev)
    m = torch.empty(w.batch, dtype=torch.int32, device=dev)
    nxt = torch.empty(w.batch, dtype=torch.int32, device=dev)
    B._check(lib.ssl_greedy_accept_workspace(w.batch, k, vocab, ctypes.byref(nws)), "ws")
    ws2 = torch.empty(max(nws.value, 1), dtype=torch.uint8, device=dev)
    aargs = [(c.data_ptr(), B.SSL_DT_BF16, w.batch, k, k_len.ctypes.data_as(B._i32p), vocab, vocab,
              draft.data_ptr(), m.data_ptr(), nxt.data_ptr(), ws2.data_ptr(), ws2.numel(),
              B._stream(stream)) for c in copies]
    # speculative sampling: the k + 1 verify rows of each sequence as the
    # target, the first k rows of the next copy as the drafter's rows
    u_acc = torch.from_numpy(rng.random((w.batch, k)).astype(np.float32)).to(dev)
    u_smp = torch.from_numpy(rng.random(w.batch).astype(np.float32)).to(dev)
    B._check(lib.ssl_spec_accept_workspace(w.batch, k, vocab, ctypes.byref(nws)), "ws")
    ws3 = torch.empty(max(nws.value, 1), dtype=torch.uint8, device=dev)
    pargs = [(c.data_ptr(), copies[(i + 1) % n].data_ptr(), B.SSL_DT_BF16, w.batch, k,
              k_len.ctypes.data_as(B._i32p), vocab, vocab, draft.data_ptr(), 1.0,
              u_acc.data_ptr(), u_smp.data_ptr(), m.data_ptr(), nxt.data_ptr(), ws3.data_ptr(),
              ws3.numel(), B._stream(stream)) for i, c in enumerate(copies)]
    for a in sargs:
        B._check(lib.ssl_logit_stats(*a), "ssl_logit_stats")
    for a in aargs:
        B._check(lib.ssl_greedy_accept(*a), "ssl_greedy_accept")
    for a in pargs:
        B._check(lib.ssl_spec_accept(*a), "ssl_spec_accept")

    def timed(fn):
        return back_to_back_us(fn, reps, stream, torch)

    ent_us = timed(lambda r: lib.ssl_logit_stats(*sargs[r % n]))
    acc_us = timed(lambda r: lib.ssl_greedy_accept(*aargs[r % n]))
    spec_us = timed(lambda r: lib.ssl_spec_accept(*pargs[r % n]))
    eb, ab = draft_rows * vocab * 2, verify_rows * vocab * 2
    return {"vocab": vocab, "logits": "bf16, N(0, 2^2), seeded",
            "entropy_rows": draft_rows, "entropy_us": round(ent_us, 3),
            "entropy_gbps": round(eb / (ent_us * 1e-6) / 1e9, 1),
            "accept_rows": verify_rows, "accept_us": round(acc_us, 3),
            "accept_gbps": round(ab / (acc_us * 1e-6) / 1e9, 1),
            "spec_accept_rows": verify_rows + draft_rows, "spec_accept_us": round(spec_us, 3),
            "timing": f"{reps} back-to-back calls per figure between two HIP events "
                      f"(after one untimed call), "
                      f"rotating {n} logit copies"}


def paged_bench(B, w, kvs, q, qd, params, stream, reps, torch, np, page=128):
    """Verify and draft over a paged copy of the workload's cache (next to the
    headline, not part of it): each KV copy's rows are placed in a page pool of
    its own under a shuffled block table; each figure is ``reps`` back-to-back
    calls (rotating the pools) between two HIP events, beside the same calls on
    the dense copies."""
    import ctypes
    dev = q.device
    rng = np.random.default_rng(7)
    max_blocks = (w.max_ctx + page - 1) // page
    pools = []
    for (k, v) in kvs:
        n_pages = w.batch * max_blocks
        perm = torch.from_numpy(rng.permutation(n_pages).astype(np.int64)).to(dev)
        # dense [B, Hkv, max_blocks * page, d] -> pages [B * max_blocks, Hkv, page, d]
        def to_pages(x):
            pad = max_blocks * page - w.max_ctx
            if pad:
                x = torch.nn.functional.pad(x, (0, 0, 0, pad))
            x = x.reshape(w.batch, w.n_kv_heads, max_blocks, page, w.head_dim)
            x = x.permute(0, 2, 1, 3, 4).reshape(n_pages, w.n_kv_heads, page, w.head_dim)
            out = torch.empty_like(x)
            out[perm] = x
            return out
        bt = perm.reshape(w.batch, max_blocks).to(torch.int32)
        pools.append((to_pages(k), to_pages(v), bt.contiguous()))
    lib = B.load()
    vshape = B.Shape(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.max_ctx, w.max_q)
    ctx, ql = B._host_i32(w.ctx_len), B._host_i32(w.q_len)
    out = torch.empty(q.shape, dtype=torch.bfloat16, device=dev)
    sc = torch.empty((w.batch, w.n_kv_heads, w.max_ctx), dtype=torch.float32, device=dev)
    vws = torch.empty(max(B.verify_workspace_bytes(vshape, params, ctx, ql), 1), dtype=torch.uint8,
                      device=dev)
    n_idx = np.array([B.index_count(int(t), w.k_sink, w.k_recent, w.budget) for t in w.ctx_len],
                     dtype=np.int32)
    dshape = B.Shape(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.max_ctx, 1)
    dws = torch.empty(max(B.draft_workspace_bytes(dshape, params, n_idx), 1), dtype=torch.uint8,
                      device=dev)
    idx = torch.zeros((w.batch, w.n_kv_heads, w.budget), dtype=torch.int32, device=dev)
    B.verify_attn(q, kvs[0][0], kvs[0][1], w.ctx_len, w.q_len, params, out=out, scores=sc,
                  stream=stream)
    B.select_topb(sc, w.ctx_len, params, n_q_heads=w.n_q_heads, idx=idx, stream=stream)
    dout = torch.empty(qd.shape, dtype=torch.bfloat16, device=dev)
    sp, pp = ctypes.byref(vshape), ctypes.byref(params)
    cp, qp = ctx.ctypes.data_as(B._i32p), ql.ctypes.data_as(B._i32p)
    dsp, np_ = ctypes.byref(dshape), n_idx.ctypes.data_as(B._i32p)
    st = B._stream(stream)
    pv = [(sp, pp, cp, qp, q.data_ptr(), kp.data_ptr(), vp.data_ptr(), bt.data_ptr(), page,
           max_blocks, out.data_ptr(), sc.data_ptr(), vws.data_ptr(), vws.numel(), st)
          for (kp, vp, bt) in pools]
    dv = [(sp, pp, cp, qp, q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), sc.data_ptr(),
           vws.data_ptr(), vws.numel(), st) for (k, v) in kvs]
    pd = [(dsp, pp, np_, qd.data_ptr(), kp.data_ptr(), vp.data_ptr(), bt.data_ptr(), page,
           max_blocks, idx.data_ptr(), dout.data_ptr(), dws.data_ptr(), dws.numel(), st)
          for (kp, vp, bt) in pools]
    dd = [(dsp, pp, np_, qd.data_ptr(), k.data_ptr(), v.data_ptr(), idx.data_ptr(),
           dout.data_ptr(), dws.data_ptr(), dws.numel(), st) for (k, v) in kvs]
    n = len(pools)

    def timed(fn, args):
        for a in args:
            B._check(fn(*a), "paged bench")
        return back_to_back_us(lambda r: fn(*args[r % n]), reps, stream, torch)

    res = {"page_size": page, "max_blocks": max_blocks,
           "verify_paged_us": round(timed(lib.ssl_verify_attn_paged, pv), 3),
           "verify_dense_us": round(timed(lib.ssl_verify_attn, dv), 3),
           "draft_paged_us": round(timed(lib.ssl_draft_attn_paged, pd), 3),
           "draft_dense_us": round(timed(lib.ssl_draft_attn, dd), 3),
           "timing": f"{reps} back-to-back calls per figure between two HIP events "
                      f"(after one untimed call), "
                     f"rotating {n} pools / dense copies; block tables shuffled"}
    del pools
    return res


def summarize_traffic(fetch_dir: str, write_dir: str, copy_mib: int, command: str,
                      title: str = "llama8b-T32K workload") -> str:
    """HBM traffic per launch from two rocprofv3 --pmc runs (FETCH_SIZE, then
    WRITE_SIZE, KiB per dispatch), each scaled by what the counter reads for
    the plain device copy of copy_mib MiB that the same command ends with."""
    import csv
    import glob

    def load(d, counter):
        f = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)[0]
        rows = [r for r in csv.DictReader(open(f)) if r["Counter_Name"] == counter]
        rows.sort(key=lambda r: int(r["Dispatch_Id"]))
        copies = [float(r["Counter_Value"]) for r in rows if "copyBuffer" in r["Kernel_Name"]]
        per = {}
        for r in rows:
            k = kernel_short(r["Kernel_Name"])
            if k.split("<")[0] in OUR_KERNELS:
                per.setdefault(k, []).append(float(r["Counter_Value"]))
        return copies[-3:], {k: statistics.fmean(v) for k, v in per.items()}

    copy_bytes = copy_mib << 20
    cf, fetch = load(fetch_dir, "FETCH_SIZE")
    cw, write = load(write_dir, "WRITE_SIZE")
    f_fac = copy_bytes / (statistics.fmean(cf) * 1024.0)
    w_fac = copy_bytes / (statistics.fmean(cw) * 1024.0)
    lines = [f"# HBM traffic per launch, {title} (rocprofv3 FETCH_SIZE / WRITE_SIZE)",
             f"command = {command}",
             f"sources_sha256 = {sources_sha256()}",
             f"copy_bytes = {copy_bytes}",
             f"copy_fetch_kib = {statistics.fmean(cf):.1f}",
             f"copy_write_kib = {statistics.fmean(cw):.1f}",
             f"fetch_factor = {f_fac:.4f}",
             f"write_factor = {w_fac:.4f}"]
    call_bytes = step_bytes = 0.0
    for k in sorted(set(fetch) | set(write)):
        fb = fetch.get(k, 0.0) * 1024.0 * f_fac
        wb = write.get(k, 0.0) * 1024.0 * w_fac
        lines.append(f"{k} = fetch {fb:.0f} write {wb:.0f} bytes per launch")
        if is_step_kernel(k):
            step_bytes += fb + wb
        elif k.split("<")[0] in VERIFY_KERNELS and not is_paged(k):
            call_bytes += fb + wb
    lines.append(f"verify_call_traffic_bytes = {call_bytes:.0f}")
    if step_bytes:
        lines.append(f"decode_step_kernel_traffic_bytes = {step_bytes:.0f}")
    return "\n".join(lines) + "\n"


def summarize_mfma(d: str, command: str) -> str:
    """MFMA use per launch from a rocprofv3 --pmc MfmaUtil MfmaFlopsBF16 run:
    the share of SIMD cycles the matrix cores were busy, and the bf16 MFMA
    flops one launch issues."""
    import csv
    import glob
    f = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)[0]
    per = {}
    for r in csv.DictReader(open(f)):
        k = kernel_short(r["Kernel_Name"])
        if k.split("<")[0] in OUR_KERNELS:
            per.setdefault(k, {}).setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
    lines = ["# MFMA use per launch, llama8b-T32K workload (rocprofv3 MfmaUtil, MfmaFlopsBF16)",
             f"command = {command}",
             f"sources_sha256 = {sources_sha256()}"]
    for k in sorted(per):
        c = per[k]
        util = statistics.fmean(c.get("MfmaUtil", [0.0]))
        flops = statistics.fmean(c.get("MfmaFlopsBF16", [0.0]))
        lines.append(f"{k} = mfma busy {util:.2f} % of SIMD cycles, bf16 MFMA flops {flops:.0f} per launch")
    return "\n".join(lines) + "\n"


def measured_traffic():
    """Traffic per verify call from the committed summary, if it was taken on
    the current sources; else None."""
    try:
        kv = {}
        for line in open(TRAFFIC_FILE):
            if " = " in line and not line.startswith("#"):
                k, v = line.split(" = ", 1)
                kv[k.strip()] = v.strip()
        if kv.get("sources_sha256") != sources_sha256():
            return None
        return float(kv["verify_call_traffic_bytes"])
    except (OSError, KeyError, ValueError):
        return None


MFMA_FILE = os.path.join(REPO, "profiles", "verify_mfma_llama8b_T32K.txt")
MFMA_PEAK_TFLOPS = 2500.0   # dense bf16


def measured_mfma(kernel: str, avg_us: float):
    """MFMA use of one launch of ``kernel`` from the committed counter summary,
    if it was taken on the current sources; else None."""
    try:
        kv = {}
        for line in open(MFMA_FILE):
            if " = " in line and not line.startswith("#"):
                k, v = line.split(" = ", 1)
                kv[k.strip()] = v.strip()
        if kv.get("sources_sha256") != sources_sha256() or kernel not in kv:
            return None
        words = kv[kernel].split()
        busy, flops = float(words[2]), float(words[10])
        tflops = flops / (avg_us * 1e-6) / 1e12
        return {"kernel": kernel, "bf16_flops_per_launch": flops, "tflops": round(tflops, 1),
                "peak_tflops": MFMA_PEAK_TFLOPS, "frac": round(tflops / MFMA_PEAK_TFLOPS, 4),
                "busy_pct_of_simd_cycles": busy}
    except (OSError, ValueError, IndexError):
        return None


def cpu_baseline(w, seconds: float):
    import numpy as np
    import oracle
    threads = min(len(os.sched_getaffinity(0)), 16)
    oracle.set_num_threads(threads)
    times = []
    t_start = time.perf_counter()
    while True:
        t0 = time.perf_counter()
        _, s = oracle.verify(w)
        idx, n_idx = oracle.select(w, s)
        oracle.draft(w, np.maximum(idx, 0), n_idx)
        times.append(time.perf_counter() - t0)
        if time.perf_counter() - t_start >= seconds or len(times) >= 200:
            break
    units = w.batch * w.n_kv_heads
    return {"value": statistics.median(times) * 1e6, "unit": "us/step",
            "cores": min(threads, units), "kind": "oracle",
            "sample": f"the full workload step (verify over all {units} KV-head units, select, "
                      f"draft), repeated {len(times)} times; median; fp64 C, OpenMP over "
                      f"units with {threads} threads available"}


def oracle_times(w, threads: int, repeats: int):
    """The oracle's verify, select and draft on the workload, each timed on its
    own (median of ``repeats``), with ``threads`` OpenMP threads."""
    import numpy as np
    import oracle
    oracle.set_num_threads(threads)
    tv, ts, td = [], [], []
    for _ in range(repeats):
        t0 = time.perf_counter()
        _, s = oracle.verify(w)
        t1 = time.perf_counter()
        idx, n_idx = oracle.select(w, s)
        t2 = time.perf_counter()
        oracle.draft(w, np.maximum(idx, 0), n_idx)
        t3 = time.perf_counter()
        tv.append(t1 - t0)
        ts.append(t2 - t1)
        td.append(t3 - t2)
    med = lambda x: round(statistics.median(x) * 1e6, 1)
    return {"threads": threads, "repeats": repeats, "verify_us": med(tv), "select_us": med(ts),
            "draft_us": med(td),
            "step_us": round(statistics.median([a + b + c for a, b, c in zip(tv, ts, td)]) * 1e6, 1)}


def workload_entry(B, n: int, steps: int, warmup: int, torch, np, cpu: bool):
    """One named workload measured on its own: bare steps back to back (wall
    clock), per-call durations from HIP events between the calls (median, p10,
    p90), each call's average launch from ``steps`` back-to-back calls between
    two events (GB/s and fraction of the HBM peak from its algorithmic bytes),
    and the CPU oracle's per-kernel times on the host."""
    from paper_2607_27735_amd.workloads import make_config
    t_gen = time.perf_counter()
    w = make_config(n)
    t_gen = time.perf_counter() - t_gen
    dev = torch.device("cuda:0")

    def up(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16).copy()).view(
            torch.bfloat16).to(dev)

    q, qd = up(w.q), up(w.q_draft)
    k0, v0 = up(w.k), up(w.v)
    kv_bytes = k0.numel() * 2 * 2
    n_copies = kv_copies(w, kv_bytes)
    kvs = [(k0, v0)] + [(k0.clone(), v0.clone()) for _ in range(n_copies - 1)]
    params = B.make_params(w.sm_scale, window=w.window, k_sink=w.k_sink, k_recent=w.k_recent,
                           budget=w.budget, out_fp32=False)
    out = torch.empty(q.shape, dtype=torch.bfloat16, device=dev)
    scores = torch.zeros((w.batch, w.n_kv_heads, w.max_ctx), dtype=torch.float32, device=dev)
    idx = torch.zeros((w.batch, w.n_kv_heads, w.budget), dtype=torch.int32, device=dev)
    n_idx = torch.zeros(w.batch, dtype=torch.int32, device=dev)
    dout = torch.empty(qd.shape, dtype=torch.bfloat16, device=dev)
    stream = torch.cuda.current_stream()
    sts = [B.PreparedStep(q, k, v, qd, w.ctx_len, w.q_len, params, out, scores, idx, n_idx, dout,
                          stream=stream) for (k, v) in kvs]
    vshape = B.verify_shape(q, k0)
    schedule, vchunk, vitems = B.verify_plan(vshape, params, w.ctx_len, w.q_len)
    sel_one, _, sel_parts = B.select_plan(vshape, params, w.ctx_len)
    gc.collect()
    gc.disable()   # (as in the headline passes)
    for i in range(max(warmup, n_copies)):
        sts[i % n_copies].step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        sts[i % n_copies].step()
    torch.cuda.synchronize()
    step_us = (time.perf_counter() - t0) * 1e6 / steps
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
    for e in ev:   # (created at their first record: not inside the pass)
        for x in e:
            x.record(stream)
    for c in ("verify", "select", "draft"):   # (first launches load kernels: not inside the pass)
        getattr(sts[-1], c)()
    torch.cuda.synchronize()
    for i in range(steps):
        st, e = sts[i % n_copies], ev[i]
        e[0].record(stream)
        st.verify()
        e[1].record(stream)
        st.select()
        e[2].record(stream)
        st.draft()
        e[3].record(stream)
    torch.cuda.synchronize()
    calls = ("verify", "select", "draft")
    b2b = {}
    for c in calls:
        b2b[c] = back_to_back_us(lambda i, c=c: getattr(sts[i % n_copies], c)(), steps, stream, torch)
    gc.enable()
    nbytes, _ = algorithmic_bytes(w, out_bytes=2)
    entry = {"name": w.name, "batch": w.batch, "n_q_heads": w.n_q_heads,
             "n_kv_heads": w.n_kv_heads, "ctx_len": list(map(int, w.ctx_len)),
             "q_len": list(map(int, w.q_len)), "budget": w.budget,
             "verify_schedule": {B.VERIFY_ONE_SWEEP: "one-sweep", B.VERIFY_TWO_SWEEP: "two-sweep",
                                 B.VERIFY_ONE_SWEEP_PERSISTENT: "one-sweep persistent"}[schedule],
             "verify_items": vitems, "select_schedule": "one kernel" if sel_one else "three kernels",
             "select_partitions_per_unit": sel_parts,
             "step_call": "one kernel" if sts[0].one_kernel else "verify, then select_draft",
             "step_us": round(step_us, 3), "step_alg_bytes": sum(nbytes.values()),
             "step_hbm_frac": round(sum(nbytes.values()) / (step_us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
             "steps": steps, "kv_copies_rotated": n_copies, "calls": {}}
    for j, c in enumerate(calls):
        per = [ev[i][j].elapsed_time(ev[i][j + 1]) * 1e3 for i in range(steps)]
        gbps = nbytes[c] / (b2b[c] * 1e-6) / 1e9
        entry["calls"][c] = {"median_us": round(statistics.median(per), 3),
                             "p10_us": round(float(np.percentile(per, 10)), 3),
                             "p90_us": round(float(np.percentile(per, 90)), 3),
                             "back_to_back_us": round(b2b[c], 3), "alg_bytes": nbytes[c],
                             "gbps": round(gbps, 1), "hbm_frac": round(gbps / HBM_PEAK_GBPS, 4)}
    assert B.exchange_status(stream) == 0, "an exchange wait gave up"
    del sts, kvs, q, qd, k0, v0, out, scores, idx, n_idx, dout
    torch.cuda.empty_cache()
    if cpu:
        threads = min(len(os.sched_getaffinity(0)), 16)
        entry["oracle"] = oracle_times(w, threads, 3 if n <= 2 else 1)
        if n == 1:
            entry["oracle_single_thread"] = oracle_times(w, 1, 3)
            import oracle
            oracle.set_num_threads(threads)
    entry["input_generation_s"] = round(t_gen, 1)
    return entry


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", type=int, default=2, help="named workload 1..5 (default 2)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-draft-round", action="store_true",
                    help="skip the draft-round and vocabulary-side measurements printed "
                         "beside the headline")
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip the per-workload table (all five named workloads)")
    ap.add_argument("--mode", choices=["eager", "graph"], default="eager")
    ap.add_argument("--no-graph-step", action="store_true",
                    help="skip the captured-step figure printed beside the eager headline")
    ap.add_argument("--verify-mode", choices=["auto", "two-sweep", "one-sweep"], default="auto")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="end with three plain device copies of this size (counter calibration)")
    ap.add_argument("--summarize-trace", metavar="DIR",
                    help="print a summary of a rocprofv3 --kernel-trace --stats output and exit")
    ap.add_argument("--summarize-traffic", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="print HBM traffic per launch from two rocprofv3 --pmc outputs and exit")
    ap.add_argument("--summarize-mfma", metavar="DIR",
                    help="print MFMA use per launch from a rocprofv3 --pmc MfmaUtil MfmaFlopsBF16 "
                         "output and exit")
    ap.add_argument("--command-text", default="", help="the profiling command, for summaries")
    ap.add_argument("--title", default="", help="the workload a summary covers, for its title")
    args = ap.parse_args()
    if args.summarize_trace:
        sys.stdout.write(summarize_trace(args.summarize_trace, args.command_text, args.title))
        return 0
    if args.summarize_mfma:
        sys.stdout.write(summarize_mfma(args.summarize_mfma, args.command_text))
        return 0
    if args.summarize_traffic:
        sys.stdout.write(summarize_traffic(*args.summarize_traffic, args.copy_calibration_mib,
                                           args.command_text,
                                           args.title or "llama8b-T32K workload"))
        return 0
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (the hot path runs on one GPU; see the design "
              f"notes for how it would shard); --gpus {args.gpus} is not supported",
              file=sys.stderr)
        return 2

    import numpy as np
    import torch
    from paper_2607_27735_amd import binding as B
    from paper_2607_27735_amd.workloads import make_config, CONFIGS

    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        return 1
    B.load()
    w = make_config(args.workload)
    dev = torch.device("cuda:0")

    def up(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16).copy()).view(
            torch.bfloat16).to(dev)

    q, qd = up(w.q), up(w.q_draft)
    k0, v0 = up(w.k), up(w.v)
    kv_bytes = k0.numel() * 2 * 2
    n_copies = kv_copies(w, kv_bytes)
    kvs = [(k0, v0)] + [(k0.clone(), v0.clone()) for _ in range(n_copies - 1)]
    vmode = {"auto": B.VERIFY_AUTO, "two-sweep": B.VERIFY_TWO_SWEEP,
             "one-sweep": B.VERIFY_ONE_SWEEP}[args.verify_mode]
    params = B.make_params(w.sm_scale, window=w.window, k_sink=w.k_sink, k_recent=w.k_recent,
                           budget=w.budget, out_fp32=False, verify_mode=vmode)
    out = torch.empty(q.shape, dtype=torch.bfloat16, device=dev)
    scores = torch.zeros((w.batch, w.n_kv_heads, w.max_ctx), dtype=torch.float32, device=dev)
    idx = torch.zeros((w.batch, w.n_kv_heads, w.budget), dtype=torch.int32, device=dev)
    n_idx = torch.zeros(w.batch, dtype=torch.int32, device=dev)
    dout = torch.empty(qd.shape, dtype=torch.bfloat16, device=dev)

    vshape = B.Shape(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, w.max_ctx, w.max_q)
    schedule, vchunk, vitems = B.verify_plan(vshape, params, w.ctx_len, w.q_len)
    sched_name = {B.VERIFY_ONE_SWEEP: "one-sweep", B.VERIFY_TWO_SWEEP: "two-sweep",
                  B.VERIFY_ONE_SWEEP_PERSISTENT: "one-sweep persistent"}[schedule]
    verify_kernels = {B.VERIFY_ONE_SWEEP: "verify_fused_kernel",
                      B.VERIFY_ONE_SWEEP_PERSISTENT: "verify_pipe_kernel",
                      B.VERIFY_TWO_SWEEP: "verify_stats_kernel + verify_main_kernel + verify_combine_kernel"}[schedule]

    stream = torch.cuda.current_stream()
    steps = [B.PreparedStep(q, k, v, qd, w.ctx_len, w.q_len, params, out, scores, idx, n_idx,
                            dout, stream=stream) for (k, v) in kvs]
    # The timed passes run with Python's garbage collector paused, so that a
    # collection cannot stall the host between two launches; the collection
    # runs before the warm-up, not between it and the timed steps.
    gc.collect()
    gc.disable()
    for i in range(args.warmup):
        steps[i % n_copies].step()
    torch.cuda.synchronize()

    calls = ("verify", "select", "draft")
    graphs = None
    step_graphs = []
    if args.mode == "graph":
        # Per KV copy, one graph per call (events between their replays time
        # each call) and one graph of the whole step (the headline).
        graphs = []
        cap = torch.cuda.Stream()
        cap.wait_stream(stream)
        for (k, v) in kvs:
            with torch.cuda.stream(cap):
                st = B.PreparedStep(q, k, v, qd, w.ctx_len, w.q_len, params, out, scores, idx,
                                    n_idx, dout, stream=cap)
            with torch.cuda.stream(cap):   # eager warm-up on the capture stream
                st.step()
            gs = []
            for name in calls:
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g, stream=cap):
                    getattr(st, name)()
                gs.append(g)
            sg = torch.cuda.CUDAGraph()   # the whole step, for the headline
            with torch.cuda.graph(sg, stream=cap):
                st.step()
            graphs.append(gs)
            step_graphs.append((sg, st))
        stream.wait_stream(cap)
        for i in range(args.warmup):
            for g in graphs[i % n_copies]:
                g.replay()
        torch.cuda.synchronize()

    # Headline: exactly K steps back to back, nothing else on the stream.
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        if graphs is not None:
            step_graphs[i % n_copies][0].replay()
        else:
            steps[i % n_copies].step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()

    # Breakdown: K more steps with HIP events between the calls (on the stream
    # the kernels run on) for the per-call durations and the roofline.
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    for e in ev:   # (torch creates an event's HIP event at its first record: not inside the pass)
        for x in e:
            x.record(stream)
    if graphs is None:   # each call's first launch loads its kernels: not inside the pass
        for c in calls:
            getattr(steps[-1], c)()
    torch.cuda.synchronize()
    for i in range(args.steps):
        e = ev[i]
        if graphs is not None:
            gs = graphs[i % n_copies]
            e[0].record(stream)
            gs[0].replay()
            e[1].record(stream)
            gs[1].replay()
            e[2].record(stream)
            gs[2].replay()
            e[3].record(stream)
        else:
            st = steps[i % n_copies]
            e[0].record(stream)
            st.verify()
            e[1].record(stream)
            st.select()
            e[2].record(stream)
            st.draft()
            e[3].record(stream)
    torch.cuda.synchronize()

    # Roofline: K verify calls back to back (a different KV copy each) between
    # two events, i.e. the call's average launch duration in steady state.
    # The same for select and draft: each call's bandwidth figures below come
    # from these back-to-back averages, which a host stall between two launches
    # of the event-bracketed pass above cannot inflate.
    b2b = {}
    for j, c in enumerate(calls):
        if graphs is not None:
            b2b[c] = back_to_back_us(lambda i, j=j: graphs[i % n_copies][j].replay(), args.steps, stream, torch)
        else:
            b2b[c] = back_to_back_us(lambda i, c=c: getattr(steps[i % n_copies], c)(), args.steps, stream, torch)
    v_iso = b2b["verify"]

    gc.enable()
    per = {c: [ev[i][j].elapsed_time(ev[i][j + 1]) * 1e3 for i in range(args.steps)]
           for j, c in enumerate(calls)}
    step_us = [ev[i][0].elapsed_time(ev[i][3]) * 1e3 for i in range(args.steps)]
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    nbytes, n_list = algorithmic_bytes(w, out_bytes=2)
    kernels = {}
    for c in calls:
        avg = statistics.fmean(per[c])
        kernels[c] = {"back_to_back_us": round(b2b[c], 3),
                      "avg_us": round(avg, 3), "median_us": round(statistics.median(per[c]), 3),
                      "p10_us": round(float(np.percentile(per[c], 10)), 3),
                      "p90_us": round(float(np.percentile(per[c], 90)), 3),
                      "alg_bytes": nbytes[c],
                      "gbps": round(nbytes[c] / (b2b[c] * 1e-6) / 1e9, 1),
                      "hbm_frac": round(nbytes[c] / (b2b[c] * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4)}
    v_avg = round(v_iso, 3)
    step_total = sum(nbytes.values())
    result = {
        "metric": METRIC,
        "value": round(ms_per_step * 1e3, 3),
        "unit": "us/step",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 6),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{w.name}: batch {w.batch}, {w.n_q_heads} query / "
                               f"{w.n_kv_heads} KV heads, head_dim {w.head_dim}, context "
                               f"{list(map(int, w.ctx_len))}, k+1 = {list(map(int, w.q_len))}, "
                               f"B = {w.budget}, K_sink {w.k_sink}, K_recent {w.k_recent}, "
                               f"W {w.window}",
                   "batch": w.batch, "n_q_heads": w.n_q_heads, "n_kv_heads": w.n_kv_heads,
                   "head_dim": w.head_dim, "ctx_len": list(map(int, w.ctx_len)),
                   "q_len": list(map(int, w.q_len)), "budget": w.budget,
                   "launch": args.mode, "kv_copies_rotated": n_copies,
                   "verify_schedule": sched_name, "verify_chunk": vchunk,
                   "verify_items": vitems,
                   "step_call": "ssl_decode_step (" + ("one kernel: verify, select and the first "
                                "draft step" if steps[0].one_kernel else
                                "verify, then select_draft") + ")"},
        "gpu_step_us_median": round(statistics.median(step_us), 3),
        "step_alg_bytes": step_total,
        "step_hbm_gbps": round(step_total / (ms_per_step * 1e-3) / 1e9, 1),
        "roofline": {"bound": "hbm", "kernel": f"ssl_verify_attn ({verify_kernels})",
                     "achieved": round(nbytes["verify"] / (v_avg * 1e-6) / 1e9, 1),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(nbytes["verify"] / (v_avg * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
                     "traffic": (measured_traffic() if (args.workload == 2 and args.mode == "eager"
                                                        and args.verify_mode == "auto") else None),
                     "bytes_per_launch": nbytes["verify"],
                     "avg_launch_us": v_avg,
                     "timing": "K back-to-back verify calls between two HIP events on the launch stream, after one untimed call"},
        "kernels": kernels,
        "kernels_timing": "back_to_back_us: K calls of one kind back to back between two HIP events "
                          "(after one untimed call), which gbps and hbm_frac use; avg, median, p10, "
                          "p90: each call bracketed by events inside K whole steps",
    }
    if args.workload == 2 and args.mode == "eager" and args.verify_mode == "auto":
        result["mfma"] = measured_mfma("verify_fused_kernel<2, true, false, false>", v_avg)
    if args.mode == "eager" and not args.no_graph_step:
        result["graph_step"] = graph_step_bench(B, kvs, q, qd, w, params, out, scores, idx, n_idx,
                                                dout, stream, args.steps, torch)
    if not args.no_draft_round:
        result["draft_round"] = draft_round_bench(B, w, kvs, qd, params, scores, stream,
                                                  args.steps, torch, np)
        result["vocab_side"] = vocab_side_bench(B, w, stream, args.steps, torch, np)
        result["paged"] = paged_bench(B, w, kvs, q, qd, params, stream, args.steps, torch, np)
    # every cross-workgroup exchange of the timed calls completed
    result["exchange_status"] = B.exchange_status(stream)
    # sanity: score mass of every KV head equals min(W, q) * group
    s = scores.double().sum(dim=2).cpu().numpy()
    want = np.array([min(w.window, int(x)) * w.group for x in w.q_len])[:, None]
    result["score_mass_max_rel_err"] = float(np.abs(s - want).max() / want.max())
    if args.copy_calibration_mib > 0:
        # a plain device copy of known size, for scaling the traffic counters
        src = torch.empty(args.copy_calibration_mib << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
    if not args.no_workloads:
        del steps, kvs
        torch.cuda.empty_cache()
        result["workloads"] = {}
        for n in sorted(CONFIGS):
            print(f"[bench] workload {n}", file=sys.stderr, flush=True)
            result["workloads"][str(n)] = workload_entry(
                B, n, args.steps if n <= 2 else min(args.steps, 20), args.warmup, torch, np,
                cpu=not args.no_cpu_baseline)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
