"""ssl_verify_attn_static, the verify entry point that allocates nothing (its
workspace is the library's own device scratch), against ssl_verify_attn on the
same inputs: two calls in a row, the second with a smaller input, must give
the outputs and scores of the workspace entry point bit for bit (same plan,
same kernels, deterministic merge orders)."""
import pytest
import torch

from paper_2607_27735_amd import binding as B

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU visible", allow_module_level=True)


def _case(seed, batch, hq, hkv, ctx, ql, max_ctx, budget):
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev)
    g.manual_seed(seed)
    rnd = lambda *shape: torch.randn(*shape, generator=g, device=dev).to(torch.bfloat16)
    q = rnd(batch, max(ql), hq, 128)
    k = rnd(batch, hkv, max_ctx, 128)
    v = rnd(batch, hkv, max_ctx, 128)
    return q, k, v, ctx, ql, B.make_params(128 ** -0.5, budget=budget, out_fp32=False)


CASES = [
    # the 32K Llama-3-8B-shaped layer (one sweep, 256 workgroups)
    dict(seed=31, batch=1, hq=32, hkv=8, ctx=[32768], ql=[7], max_ctx=32768, budget=2048),
    # smaller: two ragged sequences of a 16/4-head layer
    dict(seed=32, batch=2, hq=16, hkv=4, ctx=[4096, 1500], ql=[5, 3], max_ctx=4100, budget=256),
]


def test_static_scratch_matches_the_workspace_entry_point():
    refs, results = [], []
    for c in CASES:
        q, k, v, ctx, ql, p = _case(**c)
        refs.append(B.verify_attn(q, k, v, ctx, ql, p))
    torch.cuda.synchronize()
    for c in CASES:      # two calls in a row on the shared scratch, the second smaller
        print(f"[no-alloc] ssl_verify_attn_static on {c}", flush=True)
        q, k, v, ctx, ql, p = _case(**c)
        out = torch.full(q.shape, -7.0, dtype=torch.bfloat16, device=q.device)
        sc = torch.full((k.shape[0], k.shape[1], k.shape[2]), -1.0, dtype=torch.float32,
                        device=q.device)
        B.verify_attn_static(q, k, v, ctx, ql, p, out=out, scores=sc)
        results.append((out, sc))
    torch.cuda.synchronize()
    for c, (o_ref, s_ref), (o, s) in zip(CASES, refs, results):
        for b, (t, n) in enumerate(zip(c["ctx"], c["ql"])):
            assert torch.equal(o[b, :n], o_ref[b, :n]), f"outputs differ ({c})"
            assert torch.equal(s[b, :, :t], s_ref[b, :, :t]), f"scores differ ({c})"
    assert B.exchange_status() == 0
