"""GPU parity of the token statistics around the path (the draft entropies
that feed the length controller, and greedy acceptance over verify logits)
against the oracle.  Argmax, acceptance counts and tokens are integers:
bit-exact.  Entropy: fp32 accumulation of e^(x - M) and x e^(x - M) over at
most 524288 logits (32 per thread in sequence, then a merge tree) against
fp64; the bound allowed is 2e-5 * (1 + max |x|) nats per row.  Padding
columns past vocab hold values that would win the argmax if they were read."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_27735_amd import binding as B
from paper_2607_27735_amd.workloads import f32_to_bf16_bits

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU visible", allow_module_level=True)


def _logits(rng, n_rows, vocab, stride, dtype, scale):
    x = rng.standard_normal((n_rows, vocab)).astype(np.float32) * np.float32(scale)
    if n_rows > 1:
        x[1, rng.integers(vocab)] += np.float32(6.0 * max(scale, 1.0))   # a peaked row
    if n_rows > 2:   # a row of few distinct values: ties at the max
        x[2] = np.round(rng.standard_normal(vocab) * 2.0).astype(np.float32)
    full = np.full((n_rows, stride), 1.0e4, dtype=np.float32)
    full[:, :vocab] = x
    if dtype == "bf16":
        return f32_to_bf16_bits(full)
    return full


def _dev(arr):
    if arr.dtype == np.uint16:
        return torch.from_numpy(arr.view(np.int16).copy()).view(torch.bfloat16).cuda()
    return torch.from_numpy(arr.copy()).cuda()


CASES = [  # (n_rows, vocab, row_stride, dtype, scale)
    (7, 128256, 128256, "bf16", 1.0),
    (6, 128256, 128256, "f32", 3.0),
    (13, 50257, 50264, "bf16", 0.5),
    (5, 32000, 32004, "f32", 8.0),
    (3, 8, 8, "bf16", 1.0),
    (4, 8193, 8200, "bf16", 2.0),
    (2, 524288, 524288, "bf16", 1.0),
    (1, 1, 8, "bf16", 1.0),
]


@pytest.mark.parametrize("case", CASES, ids=[f"{c[0]}x{c[1]}-{c[3]}" for c in CASES])
def test_logit_stats_matches_oracle(case):
    n_rows, vocab, stride, dtype, scale = case
    rng = np.random.default_rng(n_rows * 1000 + vocab % 997)
    x = _logits(rng, n_rows, vocab, stride, dtype, scale)
    print(f"[logit stats] {n_rows} rows, vocab {vocab}, stride {stride}, {dtype}", flush=True)
    H_ref, a_ref = oracle.row_stats(x, vocab=vocab)
    H, a = B.logit_stats(_dev(x), vocab=vocab)
    torch.cuda.synchronize()
    H, a = H.cpu().numpy().astype(np.float64), a.cpu().numpy()
    assert np.array_equal(a, a_ref), (a, a_ref)
    xs = (x.astype(np.uint32) << 16).view(np.float32) if x.dtype == np.uint16 else x
    bound = 2e-5 * (1.0 + np.abs(xs[:, :vocab]).max(axis=1))
    err = np.abs(H - H_ref)
    assert np.all(err <= bound), (err, bound)
    print(f"  worst |dH| = {err.max():.2e} nats")
    # each output alone
    H2, none = B.logit_stats(_dev(x), vocab=vocab, argmax=False)
    none2, a2 = B.logit_stats(_dev(x), vocab=vocab, entropy=False)
    torch.cuda.synchronize()
    assert none is None and none2 is None
    assert np.array_equal(H2.cpu().numpy().astype(np.float64), H)
    assert np.array_equal(a2.cpu().numpy(), a)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_greedy_accept_matches_oracle(dtype):
    rng = np.random.default_rng(91 if dtype == "bf16" else 92)
    batch, max_k, vocab = 8, 10, 128256
    k_len = np.array([10, 0, 3, 7, 10, 1, 5, 9], dtype=np.int32)
    x = _logits(rng, batch * (max_k + 1), vocab, vocab, dtype, 2.0).reshape(batch, max_k + 1, vocab)
    _, t = oracle.row_stats(x.reshape(batch * (max_k + 1), vocab))
    t = t.reshape(batch, max_k + 1)
    draft = t[:, :max_k].copy()
    plant = [None, None, 1, 6, None, 0, 2, 4]        # where a drafted token disagrees
    for b, j in enumerate(plant):
        if j is not None and j < k_len[b]:
            draft[b, j] = (t[b, j] + 1 + rng.integers(vocab - 1)) % vocab
    draft[7, 8] = (t[7, 8] + 5) % vocab               # sequence 7: a second mismatch later
    m_ref, n_ref = oracle.greedy_accept(x, draft, k_len)
    m, n = B.greedy_accept(_dev(x), torch.from_numpy(draft.astype(np.int32)).cuda(), k_len)
    torch.cuda.synchronize()
    assert np.array_equal(m.cpu().numpy(), m_ref), (m.cpu().numpy(), m_ref)
    assert np.array_equal(n.cpu().numpy(), n_ref)
    assert list(m_ref) == [10, 0, 1, 6, 10, 0, 2, 4]  # the planted structure


def test_greedy_accept_random_drafts():
    rng = np.random.default_rng(93)
    batch, max_k, vocab = 64, 63, 4000
    k_len = rng.integers(0, max_k + 1, size=batch).astype(np.int32)
    # few distinct logit values per row: agreement happens by chance, ties are common
    x = np.round(rng.standard_normal((batch, max_k + 1, vocab)) * 1.5).astype(np.float32)
    x[..., :4] += 3.0                                 # argmax among the first few tokens
    xb = f32_to_bf16_bits(x)
    _, t = oracle.row_stats(xb.reshape(-1, vocab))
    t = t.reshape(batch, max_k + 1)
    draft = np.where(rng.random((batch, max_k)) < 0.85, t[:, :max_k],
                     rng.integers(0, vocab, size=(batch, max_k))).astype(np.int32)
    m_ref, n_ref = oracle.greedy_accept(xb, draft, k_len)
    m, n = B.greedy_accept(_dev(xb), torch.from_numpy(draft).cuda(), k_len)
    torch.cuda.synchronize()
    assert np.array_equal(m.cpu().numpy(), m_ref)
    assert np.array_equal(n.cpu().numpy(), n_ref)
