"""Calls captured in a HIP graph and replayed with new contents in the
captured input buffers.  Each replay must equal the eager calls on the same
inputs, bit for bit: the kernels are deterministic (fixed merge orders, no
floating-point atomics).  The whole decode step (one kernel: verify, select
and the first draft step), the separate calls, a draft-round step and the
logit statistics exchange partial results between workgroups behind
tags, and a replay reuses the call tag fixed at capture; the workspace epochs
must give every replay a new one, or a replay could take the previous
replay's partials as its own.  Replays alternate with eager calls and
synchronisations, and every replay is checked."""
import pytest
import torch

from paper_2607_27735_amd import binding as B

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU visible", allow_module_level=True)

BATCH, HQ, HKV, D = 1, 32, 8, 128
T, QLEN, MAX_CTX, BUDGET = 16384, 7, 16392, 1024
K_ROUND, ROUND_STEP = 3, 2
N_LOGIT_ROWS, VOCAB = 6, 128256
REPLAYS = 4


def _refill(gen, *ts):
    for t in ts:
        t.copy_(torch.randn(t.shape, generator=gen, device=t.device, dtype=torch.float32).to(t.dtype))


def test_graph_replays_match_eager_calls():
    dev = torch.device("cuda:0")
    gen = torch.Generator(device=dev)
    gen.manual_seed(2607)
    q = torch.empty(BATCH, QLEN, HQ, D, dtype=torch.bfloat16, device=dev)
    k = torch.empty(BATCH, HKV, MAX_CTX, D, dtype=torch.bfloat16, device=dev)
    v = torch.empty_like(k)
    qd = torch.empty(BATCH, HQ, D, dtype=torch.bfloat16, device=dev)
    logits = torch.empty(N_LOGIT_ROWS, VOCAB, dtype=torch.bfloat16, device=dev)
    _refill(gen, q, k, v, qd, logits)
    params = B.make_params(D ** -0.5, budget=BUDGET, out_fp32=True)
    ctx, ql = [T], [QLEN]
    n_idx_host = B.index_count(T, params.k_sink, params.k_recent, BUDGET)

    out = torch.empty(BATCH, QLEN, HQ, D, dtype=torch.float32, device=dev)
    scores = torch.empty(BATCH, HKV, MAX_CTX, dtype=torch.float32, device=dev)
    idx = torch.empty(BATCH, HKV, BUDGET, dtype=torch.int32, device=dev)
    n_idx = torch.empty(BATCH, dtype=torch.int32, device=dev)
    dout = torch.empty(BATCH, HQ, D, dtype=torch.float32, device=dev)
    rout = torch.empty(BATCH, HQ, D, dtype=torch.float32, device=dev)

    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    st = B.PreparedStep(q, k, v, qd, ctx, ql, params, out, scores, idx, n_idx, dout, stream=cap)
    rnd = B.PreparedRound(qd, k, v, idx, ctx, K_ROUND, params, rout, stream=cap)
    assert B.verify_plan(st.shape, params, ctx, ql)[0] == B.VERIFY_ONE_SWEEP
    assert st.one_kernel
    with torch.cuda.stream(cap):   # eager warm-up: one-time launcher set-up stays out of the graph
        st.step()
        rnd.step(ROUND_STEP)
        B.logit_stats(logits)
    torch.cuda.synchronize()

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=cap):
        st.step()
        rnd.step(ROUND_STEP)
        ent_g, am_g = B.logit_stats(logits)
    torch.cuda.synchronize()

    for r in range(REPLAYS):
        print(f"[graph] replay {r}: new inputs, replay, eager reference", flush=True)
        _refill(gen, q, k, v, qd, logits)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()

        # the step is one call (one kernel here): its eager run, then the
        # separate calls, whose outputs, scores and index sets it must equal
        out_e, scores_e, idx_e, n_idx_e, dout_e = B.decode_step(q, k, v, qd, ctx, ql, params)
        out_v, scores_v = B.verify_attn(q, k, v, ctx, ql, params)
        idx_s, n_idx_s = B.select_topb(scores_v, ctx, params)
        torch.cuda.synchronize()
        assert torch.equal(out_e, out_v) and torch.equal(scores_e[:, :, :T], scores_v[:, :, :T])
        assert torch.equal(n_idx_e, n_idx_s) and torch.equal(idx_e[:, :, :n_idx_host],
                                                             idx_s[:, :, :n_idx_host])
        rout_e = torch.empty_like(rout)
        B.PreparedRound(qd, k, v, idx_e, ctx, K_ROUND, params, rout_e).step(ROUND_STEP)
        ent_e, am_e = B.logit_stats(logits)
        torch.cuda.synchronize()

        assert torch.equal(out, out_e), f"replay {r}: verify output"
        assert torch.equal(scores[:, :, :T], scores_e[:, :, :T]), f"replay {r}: scores"
        assert torch.equal(n_idx, n_idx_e), f"replay {r}: n_idx"
        assert torch.equal(idx[:, :, :n_idx_host], idx_e[:, :, :n_idx_host]), f"replay {r}: idx"
        assert torch.equal(dout, dout_e), f"replay {r}: draft output"
        assert torch.equal(rout, rout_e), f"replay {r}: draft-round step output"
        assert torch.equal(am_g, am_e), f"replay {r}: argmax"
        assert torch.equal(ent_g, ent_e), f"replay {r}: entropy"
        # the inputs changed, so a replay that returned the previous results fails
        if r > 0:
            assert not torch.equal(out, prev_out), f"replay {r}: output did not change"
        prev_out = out.clone()


def test_graph_with_one_shared_workspace():
    """verify -> select (three kernels: more than 256 partitions) -> draft as
    separate calls, captured with ONE workspace for the calls, replayed with new inputs.
    Every layout keeps its exchange epochs in the same leading words, so the
    select histograms never land on the draft's epochs."""
    dev = torch.device("cuda:0")
    gen = torch.Generator(device=dev)
    gen.manual_seed(2608)
    batch, t, max_ctx = 3, 16384, 16392
    q = torch.empty(batch, QLEN, HQ, D, dtype=torch.bfloat16, device=dev)
    k = torch.empty(batch, HKV, max_ctx, D, dtype=torch.bfloat16, device=dev)
    v = torch.empty_like(k)
    qd = torch.empty(batch, HQ, D, dtype=torch.bfloat16, device=dev)
    _refill(gen, q, k, v, qd)
    params = B.make_params(D ** -0.5, budget=BUDGET, out_fp32=True)
    ctx, ql = [t] * batch, [QLEN] * batch
    n_idx_host = B.index_count(t, params.k_sink, params.k_recent, BUDGET)
    out = torch.empty(batch, QLEN, HQ, D, dtype=torch.float32, device=dev)
    scores = torch.empty(batch, HKV, max_ctx, dtype=torch.float32, device=dev)
    idx = torch.empty(batch, HKV, BUDGET, dtype=torch.int32, device=dev)
    n_idx = torch.empty(batch, dtype=torch.int32, device=dev)
    dout = torch.empty(batch, HQ, D, dtype=torch.float32, device=dev)
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    st = B.PreparedStep(q, k, v, qd, ctx, ql, params, out, scores, idx, n_idx, dout, stream=cap,
                        shared_workspace=True)
    # (three sequences of 16K: 384 chunks, so the persistent one-sweep form)
    assert B.verify_plan(st.shape, params, ctx, ql)[0] == B.VERIFY_ONE_SWEEP_PERSISTENT
    assert B.select_plan(st.shape, params, ctx)[0] is False
    with torch.cuda.stream(cap):
        st.step_separate()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=cap):
        st.step_separate()
    torch.cuda.synchronize()
    for r in range(REPLAYS):
        print(f"[graph, shared workspace] replay {r}", flush=True)
        _refill(gen, q, k, v, qd)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        out_e, scores_e = B.verify_attn(q, k, v, ctx, ql, params)
        idx_e, n_idx_e = B.select_topb(scores_e, ctx, params)
        dout_e = B.draft_attn(qd, k, v, idx_e, [n_idx_host] * batch, params)
        torch.cuda.synchronize()
        assert torch.equal(out, out_e), f"replay {r}: verify output"
        assert torch.equal(scores[:, :, :t], scores_e[:, :, :t]), f"replay {r}: scores"
        assert torch.equal(idx[:, :, :n_idx_host], idx_e[:, :, :n_idx_host]), f"replay {r}: idx"
        assert torch.equal(dout, dout_e), f"replay {r}: draft output"
    assert B.exchange_status() == 0
