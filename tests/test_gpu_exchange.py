"""Exchange health on the GPU.

Kernels whose workgroups exchange partial results (one-sweep verify, one-kernel
select, draft and draft-round steps, logit statistics) wait for each other
with bounded polls.  These tests force every such wait to give up from the
host (ssl_test_exchange_faults: a small poll limit and published tags that no
wait accepts), so that no kernel is broken on purpose: every kernel must still
finish, leave the outputs it could not complete unwritten, and raise its bit
of the device's exchange status word; under graph capture a workspace whose
exchange gave up must keep failing, loudly, until it is filled with zeros.
Plans under a reduced CU budget must keep the results right."""
import numpy as np
import pytest
import torch

import oracle
from gpu_common import Dev, abs_v, check_outputs, check_scores, gpu_verify
from paper_2607_27735_amd import binding as B
from paper_2607_27735_amd.workloads import generate

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU visible", allow_module_level=True)

BATCH, HQ, HKV, D = 2, 32, 8, 128
T, QLEN, MAX_CTX, BUDGET = 8192, 5, 8200, 512
N_ROWS, VOCAB = 4, 40000           # five 8192-logit chunks per row
ALL = B.EXCHANGE_VERIFY | B.EXCHANGE_SELECT | B.EXCHANGE_DRAFT | B.EXCHANGE_LOGITS
SENT = -7.0


@pytest.fixture(autouse=True)
def _clean_state():
    torch.cuda.synchronize()
    B.test_exchange_faults(0, False)
    B.exchange_status()                      # start from a clear word
    yield
    B.test_exchange_faults(0, False)
    B.set_cu_budget(0)
    torch.cuda.synchronize()
    B.exchange_status()


class Inputs:
    def __init__(self, seed=5):
        dev = torch.device("cuda:0")
        g = torch.Generator(device=dev)
        g.manual_seed(seed)
        rnd = lambda *shape: torch.randn(*shape, generator=g, device=dev).to(torch.bfloat16)
        self.q = rnd(BATCH, QLEN, HQ, D)
        self.k = rnd(BATCH, HKV, MAX_CTX, D)
        self.v = rnd(BATCH, HKV, MAX_CTX, D)
        self.qd = rnd(BATCH, HQ, D)
        self.logits = rnd(N_ROWS, VOCAB)
        self.params = B.make_params(D ** -0.5, budget=BUDGET, out_fp32=True)
        self.ctx, self.ql = [T] * BATCH, [QLEN] * BATCH
        self.n_idx = [B.index_count(T, self.params.k_sink, self.params.k_recent, BUDGET)] * BATCH

    def run(self, idx_in=None):
        """verify -> select -> draft (on idx_in if given), a draft-round step and
        logit statistics into sentinel-filled outputs."""
        dev = self.q.device
        out = torch.full((BATCH, QLEN, HQ, D), SENT, dtype=torch.float32, device=dev)
        sc = torch.full((BATCH, HKV, MAX_CTX), SENT, dtype=torch.float32, device=dev)
        B.verify_attn(self.q, self.k, self.v, self.ctx, self.ql, self.params, out=out, scores=sc)
        idx = torch.full((BATCH, HKV, BUDGET), -7, dtype=torch.int32, device=dev)
        n_idx = torch.full((BATCH,), -1, dtype=torch.int32, device=dev)
        B.select_topb(sc if idx_in is None else torch.ones_like(sc), self.ctx, self.params,
                      idx=idx, n_idx=n_idx)
        src = idx if idx_in is None else idx_in
        dout = torch.full((BATCH, HQ, D), SENT, dtype=torch.float32, device=dev)
        B.draft_attn(self.qd, self.k, self.v, src, self.n_idx, self.params, out=dout)
        rout = torch.full((BATCH, HQ, D), SENT, dtype=torch.float32, device=dev)
        B.draft_step(self.qd, self.k, self.v, [T - 2] * BATCH, self.ctx, self.params, idx=src,
                     out=rout)
        ent, am = B.logit_stats(self.logits)
        # select and the first draft step in one kernel, on the verify scores
        idx2 = torch.full((BATCH, HKV, BUDGET), -7, dtype=torch.int32, device=dev)
        n_idx2 = torch.full((BATCH,), -1, dtype=torch.int32, device=dev)
        sdout = torch.full((BATCH, HQ, D), SENT, dtype=torch.float32, device=dev)
        B.select_draft(sc if idx_in is None else torch.ones_like(sc), self.ctx, self.params, self.qd,
                       self.k, self.v, idx=idx2, n_idx=n_idx2, out=sdout)
        # the whole step in one kernel
        step = (torch.full((BATCH, QLEN, HQ, D), SENT, dtype=torch.float32, device=dev),
                torch.full((BATCH, HKV, MAX_CTX), SENT, dtype=torch.float32, device=dev),
                torch.full((BATCH, HKV, BUDGET), -7, dtype=torch.int32, device=dev),
                torch.full((BATCH,), -1, dtype=torch.int32, device=dev),
                torch.full((BATCH, HQ, D), SENT, dtype=torch.float32, device=dev))
        B.decode_step(self.q, self.k, self.v, self.qd, self.ctx, self.ql, self.params, out=step[0],
                      scores=step[1], idx=step[2], n_idx=step[3], draft_out=step[4])
        torch.cuda.synchronize()
        return (out, sc, idx, n_idx, dout, rout, ent, am, idx2, n_idx2, sdout) + step


def test_plans_use_the_exchanging_schedules():
    x = Inputs()
    s = B.verify_shape(x.q, x.k)
    assert B.verify_plan(s, x.params, x.ctx, x.ql)[0] == B.VERIFY_ONE_SWEEP
    one_kernel, part, _ = B.select_plan(s, x.params, x.ctx)
    assert one_kernel is True and part <= 4096   # select_draft drafts inside the select kernel
    assert B.decode_step_plan(s, x.params, x.ctx, x.ql)   # the whole step is one kernel


def test_status_stays_clear_on_normal_calls():
    r = Inputs().run()
    assert B.exchange_status() == 0
    # the one-kernel step equals the separate calls on outputs, scores and index sets
    assert torch.equal(r[11], r[0]) and torch.equal(r[12], r[1])
    assert torch.equal(r[13], r[2]) and torch.equal(r[14], r[3])


def test_every_wait_gives_up_and_every_kernel_finishes():
    x = Inputs()
    good = x.run()
    assert B.exchange_status() == 0
    idx_good = good[2]
    B.test_exchange_faults(64, True)
    (out, sc, idx, n_idx, dout, rout, ent, am, idx2, n_idx2, sdout,
     st_out, st_sc, st_idx, st_n, st_dout) = x.run()
    flags = B.exchange_status()
    B.test_exchange_faults(0, False)
    assert flags == ALL, f"status {flags:#x}, expected {ALL:#x}"
    # nothing that needed an exchange was written
    assert torch.all(out == SENT) and torch.all(sc == SENT)
    assert torch.all(idx == -7) and torch.all(n_idx == -1)
    assert torch.all(dout == SENT) and torch.all(rout == SENT)
    assert torch.all(idx2 == -7) and torch.all(n_idx2 == -1) and torch.all(sdout == SENT)
    assert torch.all(st_out == SENT) and torch.all(st_sc == SENT) and torch.all(st_idx == -7)
    assert torch.all(st_n == -1) and torch.all(st_dout == SENT)
    # the draft kernels on a valid index set give up the same way
    out2 = x.run(idx_in=idx_good)
    B.test_exchange_faults(0, False)
    assert B.exchange_status() == 0           # read with the faults already off: nothing new
    B.test_exchange_faults(64, True)
    out2 = x.run(idx_in=idx_good)
    assert B.exchange_status() & B.EXCHANGE_DRAFT
    assert torch.all(out2[4] == SENT) and torch.all(out2[5] == SENT)
    B.test_exchange_faults(0, False)
    # afterwards the same calls give the same results as before, bit for bit
    again = x.run()
    assert B.exchange_status() == 0
    for a, b in zip(good, again):
        assert torch.equal(a, b)


def test_a_captured_call_that_gave_up_fails_until_its_workspace_is_cleared():
    x = Inputs()
    dev = x.q.device
    good = x.run()
    idx = good[2]
    ws = torch.empty(B.draft_workspace_bytes(B.Shape(BATCH, HQ, HKV, D, MAX_CTX, 1), x.params,
                                             x.n_idx), dtype=torch.uint8, device=dev)
    ws.zero_()
    dout = torch.full((BATCH, HQ, D), SENT, dtype=torch.float32, device=dev)
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cap):   # eager warm-up outside the graph
        B.draft_attn(x.qd, x.k, x.v, idx, x.n_idx, x.params, out=dout, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(dout, good[4]) and B.exchange_status() == 0

    B.test_exchange_faults(64, True)
    g_bad = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g_bad, stream=cap):
        B.draft_attn(x.qd, x.k, x.v, idx, x.n_idx, x.params, out=dout, workspace=ws)
    B.test_exchange_faults(0, False)
    g_ok = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g_ok, stream=cap):
        B.draft_attn(x.qd, x.k, x.v, idx, x.n_idx, x.params, out=dout, workspace=ws)
    torch.cuda.synchronize()

    dout.fill_(SENT)
    g_ok.replay()
    torch.cuda.synchronize()
    assert torch.equal(dout, good[4]) and B.exchange_status() == 0
    print("[exchange] replaying the graph captured with mismatched tags", flush=True)
    dout.fill_(SENT)
    g_bad.replay()
    torch.cuda.synchronize()
    assert B.exchange_status() == B.EXCHANGE_DRAFT and torch.all(dout == SENT)
    # the clean graph now finds the workspace's epochs marked: it gives up at once
    for _ in range(2):
        g_ok.replay()
        torch.cuda.synchronize()
        assert B.exchange_status() == B.EXCHANGE_DRAFT and torch.all(dout == SENT)
    ws.zero_()
    g_ok.replay()
    torch.cuda.synchronize()
    assert B.exchange_status() == 0 and torch.equal(dout, good[4])


@pytest.mark.parametrize("budget", [8, 24])
def test_small_cu_budget_keeps_results_right(budget):
    """Planned for a few CUs, verify takes the persistent one sweep (a grid of
    the budget) or two sweeps, and select three kernels (or smaller groups);
    the results still match the oracle."""
    w = generate(211, name="budget", batch=2, n_q_heads=32, n_kv_heads=8, ctx_len=[6000, 2500],
                 q_len=[5, 3], budget=300)
    B.set_cu_budget(budget)
    d = Dev(w)
    shape = B.verify_shape(d.q, d.k)
    p = B.make_params(w.sm_scale, budget=w.budget)
    print(f"[budget {budget}] verify plan {B.verify_plan(shape, p, w.ctx_len, w.q_len)}, "
          f"select plan {B.select_plan(shape, p, w.ctx_len)}", flush=True)
    out, s = gpu_verify(d)
    out_ref, s_ref = oracle.verify(w)
    oabs, _ = oracle.verify(w, v=abs_v(w))
    mask = np.arange(w.max_q)[None, :, None] < w.q_len[:, None, None] * np.ones((1, 1, w.n_q_heads), bool)
    check_outputs(out, out_ref, oabs, mask)
    check_scores(s, s_ref, w.ctx_len)
    assert B.exchange_status() == 0
