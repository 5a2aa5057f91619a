"""GPU parity of speculative sampling (ssl_spec_accept) against the oracle.

The GPU works in fp32 (row statistics, probabilities, chunk masses, the scan
that inverts the CDF), the oracle in fp64 on the same logits and uniforms.
An integer result that a floating-point comparison decides may differ only
where that comparison lies within rounding of its boundary, so for every
sequence: n_accepted must equal the oracle's, unless the first position
where they differ has |u q - p| <= 1e-5 max(p, q); the token must be the
oracle's, unless the drawn distribution's cumulative mass at one of the
token's edges lies within 1e-4 of u times the total (and the token must
carry mass).  Most sequences must match exactly.  Padding columns past vocab
hold values that would dominate if they were read."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_27735_amd import binding as B
from paper_2607_27735_amd.workloads import f32_to_bf16_bits

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("no GPU visible", allow_module_level=True)


def _dev(arr):
    if arr.dtype == np.uint16:
        return torch.from_numpy(arr.view(np.int16).copy()).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(arr)).cuda()


def _as_f32(arr):
    return (arr.astype(np.uint32) << 16).view(np.float32) if arr.dtype == np.uint16 else arr


def _inputs(seed, batch, max_k, vocab, stride, dtype, scale, noise):
    rng = np.random.default_rng(seed)
    t = np.full((batch, max_k + 1, stride), 1.0e4, np.float32)
    t[:, :, :vocab] = rng.standard_normal((batch, max_k + 1, vocab)) * scale
    d = np.full((batch, max_k, stride), 1.0e4, np.float32)
    d[:, :, :vocab] = t[:, :max_k, :vocab] + rng.standard_normal((batch, max_k, vocab)) * noise
    if dtype == "bf16":
        t, d = f32_to_bf16_bits(t), f32_to_bf16_bits(d)
    # drafted tokens: drawn from the drafter's rows (as a drafter would), a few arbitrary
    dv = _as_f32(d)[:, :, :vocab].astype(np.float64)
    x = np.zeros((batch, max_k), np.int32)
    for b in range(batch):
        for j in range(max_k):
            pr = np.exp(dv[b, j] - dv[b, j].max())
            x[b, j] = rng.choice(vocab, p=pr / pr.sum()) if rng.random() < 0.9 else rng.integers(vocab)
    k_len = rng.integers(0, max_k + 1, batch).astype(np.int32)
    k_len[0] = max_k
    u_acc = rng.random((batch, max(max_k, 0))).astype(np.float32)
    u_smp = rng.random(batch).astype(np.float32)
    return t, d, x, k_len, u_acc, u_smp


def _probs(row, tau):
    z = row.astype(np.float64) / tau
    p = np.exp(z - z.max())
    return p / p.sum()


def _check(t, d, x, k_len, u_acc, u_smp, tau, vocab, m, nxt):
    tf, df = _as_f32(t), _as_f32(d)
    m_ref, n_ref = oracle.spec_accept(tf, df, x, k_len, tau, u_acc.astype(np.float64),
                                      u_smp.astype(np.float64), vocab=vocab)
    exact = 0
    for b in range(len(k_len)):
        if m[b] != m_ref[b]:
            j = min(m[b], m_ref[b])   # the first position decided differently
            p = _probs(tf[b, j, :vocab], tau)[x[b, j]]
            q = _probs(df[b, j, :vocab], tau)[x[b, j]]
            assert abs(u_acc[b, j] * q - p) <= 1e-5 * max(p, q), (b, m[b], m_ref[b], p, q)
            continue
        if nxt[b] == n_ref[b]:
            exact += 1
            continue
        mm = m[b]
        p = _probs(tf[b, mm, :vocab], tau)
        w = np.maximum(p - _probs(df[b, mm, :vocab], tau), 0.0) if mm < k_len[b] else p
        if not w.sum() > 0:
            w = p
        c = np.cumsum(w)
        tgt = float(u_smp[b]) * c[-1]
        y = int(nxt[b])
        assert 0 <= y < vocab and w[y] > 0, (b, y)
        edges = [c[y - 1] if y > 0 else 0.0, c[y]]
        assert min(abs(e - tgt) for e in edges) <= 1e-4 * c[-1], (b, y, n_ref[b])
    return exact


CASES = [  # (seed, batch, max_k, vocab, row_stride, dtype, temperature, scale, noise)
    (1, 8, 6, 128256, 128256, "bf16", 1.0, 2.0, 0.7),
    (2, 6, 10, 32000, 32004, "f32", 0.7, 1.5, 1.0),
    (3, 4, 0, 50257, 50264, "bf16", 1.3, 3.0, 0.5),
    (4, 3, 63, 4000, 4000, "f32", 1.0, 4.0, 0.3),
    (5, 16, 4, 8193, 8200, "bf16", 2.0, 2.0, 2.0),
    (6, 5, 3, 17, 24, "f32", 1.0, 1.0, 1.0),
    (7, 2, 5, 524288, 524288, "bf16", 1.0, 2.0, 0.5),
]


@pytest.mark.parametrize("case", CASES, ids=[f"b{c[1]}-k{c[2]}-V{c[3]}-{c[5]}" for c in CASES])
def test_spec_accept_matches_oracle(case):
    seed, batch, max_k, vocab, stride, dtype, tau, scale, noise = case
    t, d, x, k_len, u_acc, u_smp = _inputs(seed, batch, max_k, vocab, stride, dtype, scale, noise)
    print(f"[spec accept] batch {batch}, max_k {max_k}, vocab {vocab}, {dtype}, tau {tau}", flush=True)
    m, nxt = B.spec_accept(_dev(t), _dev(d) if max_k > 0 else _dev(t)[:, :0],
                           torch.from_numpy(x).cuda(), k_len, tau,
                           torch.from_numpy(u_acc).cuda(), torch.from_numpy(u_smp).cuda(),
                           vocab=vocab)
    torch.cuda.synchronize()
    m, nxt = m.cpu().numpy(), nxt.cpu().numpy()
    exact = _check(t, d, x, k_len, u_acc, u_smp, tau, vocab, m, nxt)
    assert exact >= batch - 1, f"only {exact} of {batch} sequences match exactly"
    assert np.all(m <= k_len)


def test_spec_accept_identical_drafter_takes_everything():
    """A drafter equal to the target passes every token and draws the bonus
    from the last target row."""
    rng = np.random.default_rng(11)
    batch, max_k, V = 6, 5, 20000
    t = (rng.standard_normal((batch, max_k + 1, V)) * 2).astype(np.float32)
    d = t[:, :max_k].copy()
    x = rng.integers(0, V, (batch, max_k)).astype(np.int32)
    k_len = np.array([5, 4, 0, 1, 5, 3], np.int32)
    u_acc = (rng.random((batch, max_k)) * 0.999).astype(np.float32)
    u_smp = rng.random(batch).astype(np.float32)
    m, nxt = B.spec_accept(_dev(t), _dev(d), torch.from_numpy(x).cuda(), k_len, 1.0,
                           torch.from_numpy(u_acc).cuda(), torch.from_numpy(u_smp).cuda())
    torch.cuda.synchronize()
    assert np.array_equal(m.cpu().numpy(), k_len)
    _check(t, d, x, k_len, u_acc, u_smp, 1.0, V, m.cpu().numpy(), nxt.cpu().numpy())


def test_spec_accept_empirical_distribution():
    """Many sequences with the same rows and independent uniforms: the
    committed first token's histogram follows the target p0 (chi-square-like
    bound on a small vocabulary), whatever the drafter."""
    rng = np.random.default_rng(12)
    n, V = 8192, 8
    p_logits = rng.standard_normal(V).astype(np.float32) * 1.5
    q_logits = rng.standard_normal(V).astype(np.float32) * 1.5
    stride = 8
    t = np.tile(np.stack([p_logits, p_logits]), (n, 1, 1)).astype(np.float32)
    d = np.tile(q_logits[None], (n, 1, 1)).astype(np.float32)
    q = _probs(q_logits, 1.0)
    x = rng.choice(V, size=(n, 1), p=q).astype(np.int32)
    k_len = np.ones(n, np.int32)
    m_all, tok_all = [], []
    for s in range(0, n, 64):   # the kernels take at most 64 sequences a call
        sl = slice(s, s + 64)
        m, nxt = B.spec_accept(_dev(t[sl]), _dev(d[sl]), torch.from_numpy(x[sl]).cuda(),
                               k_len[sl], 1.0,
                               torch.from_numpy(rng.random((64, 1)).astype(np.float32)).cuda(),
                               torch.from_numpy(rng.random(64).astype(np.float32)).cuda())
        torch.cuda.synchronize()
        m_all.append(m.cpu().numpy())
        tok_all.append(nxt.cpu().numpy())
    m, nxt = np.concatenate(m_all), np.concatenate(tok_all)
    first = np.where(m == 1, x[:, 0], nxt)
    freq = np.bincount(first, minlength=V) / n
    p = _probs(p_logits, 1.0)
    assert np.all(np.abs(freq - p) <= 5 * np.sqrt(p * (1 - p) / n) + 1e-3), (freq, p)
    assert stride == V
