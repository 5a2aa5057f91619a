"""Pins that tie the CPU oracle to facts outside itself.

Each ``pin_*`` function takes a loaded oracle library and raises
``AssertionError`` when the oracle disagrees with:

* a library routine computing the same definition independently
  (``torch.nn.functional.scaled_dot_product_attention`` in fp64, whose GQA
  convention is query head h -> KV head h // (Hq/Hkv); ``numpy.lexsort``);
* a closed form (K = 0 gives uniform attention, V = 1 gives O = 1, constant
  acceptance probability gives a geometric series, ...);
* an invariant (probability rows sum to one, so the Eq. 3 scores of one KV
  head sum to min(W, q) * group; index sets are sorted, unique, contain
  sink and recent);
* brute force on tiny inputs (every subset of the middle span).

``test_oracle_pins.py`` runs them on the real oracle (all must pass) and
``test_oracle_mutants.py`` on copies of the oracle with a planted mistake
(at least one must fail for each mistake).
"""
from __future__ import annotations

import itertools
import math
import statistics

import numpy as np
import torch
import torch.nn.functional as F

import oracle
from paper_2607_27735_amd.workloads import generate, f32_to_bf16_bits


def _bf16_to_t64(bits: np.ndarray) -> torch.Tensor:
    """Library widening of bf16 bit patterns to float64 (torch's own bf16 type)."""
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16).copy())
    return t.view(torch.bfloat16).to(torch.float64)


def _tiny(seed, *, hq=8, hkv=2, d=128, ctx=(40,), ql=(5,), B=16, window=16,
          k_sink=4, k_recent=8):
    return generate(seed, name="tiny", batch=len(ctx), n_q_heads=hq, n_kv_heads=hkv,
                    ctx_len=list(ctx), q_len=list(ql), head_dim=d, budget=B,
                    window=window, k_sink=k_sink, k_recent=k_recent)


def _sdpa_verify(w, q_bits=None, k_bits=None, v_bits=None):
    """Verify output from torch SDPA with an explicit bottom-right causal mask."""
    q = _bf16_to_t64(w.q if q_bits is None else q_bits)
    k = _bf16_to_t64(w.k if k_bits is None else k_bits)
    v = _bf16_to_t64(w.v if v_bits is None else v_bits)
    out = torch.zeros(q.shape, dtype=torch.float64)
    for b in range(w.batch):
        T, nq = int(w.ctx_len[b]), int(w.q_len[b])
        qb = q[b, :nq].permute(1, 0, 2).unsqueeze(0)           # [1, Hq, nq, d]
        kb = k[b, :, :T].unsqueeze(0)                            # [1, Hkv, T, d]
        vb = v[b, :, :T].unsqueeze(0)
        pos = torch.arange(T)
        rows = torch.arange(nq) + (T - nq)
        mask = pos[None, :] <= rows[:, None]
        o = F.scaled_dot_product_attention(qb, kb, vb, attn_mask=mask, scale=w.sm_scale,
                                           enable_gqa=True)
        out[b, :nq] = o[0].permute(1, 0, 2)
    return out.numpy()


def _softmax_scores(w, q_bits=None, k_bits=None):
    """Eq. 3 scores from torch.softmax weights (per KV head, summed over the group)."""
    q = _bf16_to_t64(w.q if q_bits is None else q_bits)
    k = _bf16_to_t64(w.k if k_bits is None else k_bits)
    g = w.group
    S = np.zeros((w.batch, w.n_kv_heads, w.max_ctx))
    for b in range(w.batch):
        T, nq = int(w.ctx_len[b]), int(w.q_len[b])
        wn = min(w.window, nq)
        for c in range(w.n_kv_heads):
            qb = q[b, nq - wn:nq, c * g:(c + 1) * g, :]          # [wn, g, d]
            logits = torch.einsum("jhd,td->jht", qb, k[b, c, :T]) * w.sm_scale
            pos = torch.arange(T)
            rows = torch.arange(nq - wn, nq) + (T - nq)
            mask = pos[None, None, :] <= rows[:, None, None]
            P = torch.softmax(logits.masked_fill(~mask, -math.inf), dim=-1)
            S[b, c, :T] = P.sum(dim=(0, 1)).numpy()
    return S


# ---------------------------------------------------------------------------
# verify: output O
# ---------------------------------------------------------------------------

def pin_verify_matches_sdpa(lib):
    for seed, kw in [(11, {}), (12, dict(hq=4, hkv=4, ctx=(33, 20), ql=(3, 7))),
                     (13, dict(hq=6, hkv=2, d=16, ctx=(9,), ql=(9,))),
                     (14, dict(hq=8, hkv=1, d=32, ctx=(64, 17, 5), ql=(4, 1, 2)))]:
        w = _tiny(seed, **kw)
        out, _ = oracle.verify(w, lib=lib)
        ref = _sdpa_verify(w)
        err = np.abs(out - ref).max()
        assert err < 1e-12, f"verify O vs SDPA (seed {seed}): {err}"


def pin_verify_value_one(lib):
    """V = 1 makes every output exactly 1: the probabilities of a row sum to one."""
    w = _tiny(21, ctx=(50, 31), ql=(6, 2))
    v = np.full_like(w.v, f32_to_bf16_bits(np.float32(1.0)))
    out, _ = oracle.verify(w, v=v, lib=lib)
    for b in range(w.batch):
        nq = int(w.q_len[b])
        assert np.abs(out[b, :nq] - 1.0).max() < 1e-12
        assert np.all(out[b, nq:] == 0.0)


def pin_verify_zero_keys_closed_form(lib):
    """K = 0 makes attention uniform over the visible prefix: row j of q (position
    p = T - q + j) outputs the mean of V rows 0..p, and the Eq. 3 score of key i
    is group * sum over window rows with p >= i of 1 / (p + 1)."""
    w = _tiny(22, ctx=(37, 12), ql=(5, 4), window=3)
    k0 = np.zeros_like(w.k)
    out, S = oracle.verify(w, k=k0, lib=lib)
    V = _bf16_to_t64(w.v).numpy()
    g = w.group
    for b in range(w.batch):
        T, nq = int(w.ctx_len[b]), int(w.q_len[b])
        for j in range(nq):
            p = T - nq + j
            for h in range(w.n_q_heads):
                ref = V[b, h // g, :p + 1].mean(axis=0)
                assert np.abs(out[b, j, h] - ref).max() < 1e-12
        wn = min(w.window, nq)
        for i in range(T):
            ref = g * sum(1.0 / (T - nq + j + 1) for j in range(nq - wn, nq) if T - nq + j >= i)
            for c in range(w.n_kv_heads):
                assert abs(S[b, c, i] - ref) < 1e-12, (b, c, i, S[b, c, i], ref)


def pin_verify_planted_key(lib):
    """A key aligned with every query at huge scale takes all the attention:
    O equals that V row and its score equals min(W, q) * group."""
    w = _tiny(23, hq=4, hkv=2, ctx=(30,), ql=(4,))
    q = _bf16_to_t64(w.q).numpy()
    k = _bf16_to_t64(w.k).numpy().copy()
    i_star = 7
    for c in range(w.n_kv_heads):
        direction = q[0, :4, 2 * c:2 * c + 2].reshape(-1, w.head_dim).sum(axis=0)
        k[0, c, i_star] = 200.0 * direction / np.linalg.norm(direction)
    kb = f32_to_bf16_bits(k.astype(np.float32))
    out, S = oracle.verify(w, k=kb, lib=lib)
    V = _bf16_to_t64(w.v).numpy()
    for j in range(4):
        for h in range(4):
            assert np.abs(out[0, j, h] - V[0, h // 2, i_star]).max() < 1e-6
    for c in range(2):
        assert abs(S[0, c, i_star] - 4 * 2) < 1e-6
        assert S[0, c, :30].sum() - S[0, c, i_star] < 1e-6


# ---------------------------------------------------------------------------
# verify: scores S (Eq. 3)
# ---------------------------------------------------------------------------

def pin_scores_match_softmax(lib):
    for seed, kw in [(31, {}), (32, dict(ctx=(45, 23), ql=(7, 3), window=4)),
                     (33, dict(hq=12, hkv=3, d=16, ctx=(18,), ql=(18,), window=16))]:
        w = _tiny(seed, **kw)
        _, S = oracle.verify(w, lib=lib)
        ref = _softmax_scores(w)
        err = np.abs(S - ref).max()
        assert err < 1e-12, f"scores vs torch.softmax (seed {seed}): {err}"


def pin_scores_total_mass(lib):
    """Each window row's probabilities sum to 1, so a KV head's scores sum to
    min(W, q) * group; every score lies in [0, min(W, q) * group]."""
    for window in (16, 2, 1):
        w = _tiny(41, hq=8, hkv=2, ctx=(60, 25, 9), ql=(6, 3, 9), window=window)
        _, S = oracle.verify(w, lib=lib)
        for b in range(w.batch):
            T, nq = int(w.ctx_len[b]), int(w.q_len[b])
            wn = min(window, nq)
            for c in range(w.n_kv_heads):
                assert abs(S[b, c, :T].sum() - wn * w.group) < 1e-11
                assert S[b, c, :T].min() >= 0.0
                assert S[b, c, :T].max() <= wn * w.group + 1e-12
                assert np.all(S[b, c, T:] == 0.0)


def pin_scores_permutation(lib):
    """Keys visible to every verify row are exchangeable: permuting them permutes
    their scores and leaves the outputs unchanged."""
    w = _tiny(42, ctx=(40,), ql=(5,))
    T, nq = 40, 5
    perm = np.random.default_rng(0).permutation(T - nq + 1)
    k = w.k.copy(); v = w.v.copy()
    k[0, :, :T - nq + 1] = w.k[0][:, perm]
    v[0, :, :T - nq + 1] = w.v[0][:, perm]
    out0, S0 = oracle.verify(w, lib=lib)
    out1, S1 = oracle.verify(w, k=k, v=v, lib=lib)
    assert np.abs(out0 - out1).max() < 1e-12
    assert np.abs(S1[0, :, :T - nq + 1] - S0[0][:, perm]).max() < 1e-12
    assert np.abs(S1[0, :, T - nq + 1:T] - S0[0, :, T - nq + 1:T]).max() < 1e-12


# ---------------------------------------------------------------------------
# select (Eq. 4)
# ---------------------------------------------------------------------------

def _spans(T, ks, kr):
    s_end = min(ks, T)
    r_start = max(T - kr, s_end)
    return s_end, r_start


def _select_lexsort(scores_row, T, ks, kr, B):
    s_end, r_start = _spans(T, ks, kr)
    mid = np.arange(s_end, r_start)
    take = min(B - ks - kr, len(mid))
    order = np.lexsort((mid, -scores_row[mid]))       # primary -score, then position
    chosen = set(mid[order[:take]].tolist())
    keep = sorted(set(range(s_end)) | chosen | set(range(r_start, T)))
    return np.array(keep, dtype=np.int32)


def _check_index_properties(row, n, S, T, ks, kr, B):
    sel = row[:n]
    assert np.all(np.diff(sel) > 0), "not strictly ascending"
    assert sel.min() >= 0 and sel.max() < T
    s_end, r_start = _spans(T, ks, kr)
    sset = set(sel.tolist())
    assert set(range(s_end)) <= sset and set(range(r_start, T)) <= sset
    mid_sel = [i for i in sel if s_end <= i < r_start]
    mid_out = [i for i in range(s_end, r_start) if i not in sset]
    assert len(mid_sel) == min(B - ks - kr, r_start - s_end)
    for a in mid_sel:          # defining property of TopK with the tie rule
        for b in mid_out:
            assert S[a] > S[b] or (S[a] == S[b] and a < b), (a, b)


def pin_select_lexsort(lib):
    rng = np.random.default_rng(51)
    for T, ks, kr, B in [(40, 4, 8, 16), (200, 4, 32, 64), (37, 0, 5, 12), (64, 3, 0, 10),
                         (500, 4, 32, 100)]:
        batch, hkv = 2, 3
        S = np.zeros((batch, hkv, T + 3))
        S[:, :, :T] = rng.random((batch, hkv, T))
        S[0, 1, 10:20] = 0.25                       # ties across the boundary
        w = _tiny(0, hq=3, hkv=3, d=8, ctx=(T, T), ql=(1, 1), B=B, k_sink=ks, k_recent=kr)
        idx, n_idx = oracle.select(w, S, ctx_len=np.array([T, T]), lib=lib)
        for b in range(batch):
            for c in range(hkv):
                ref = _select_lexsort(S[b, c], T, ks, kr, B)
                assert n_idx[b] == len(ref)
                assert np.array_equal(idx[b, c, :n_idx[b]], ref), (T, b, c)
                _check_index_properties(idx[b, c], n_idx[b], S[b, c], T, ks, kr, B)
                assert np.all(idx[b, c, n_idx[b]:] == -1), "wrote past n_idx"


def pin_select_bruteforce_subsets(lib):
    """Tiny spans: among all subsets of the middle span of size K_mid, the chosen
    one has the largest score sum, and among equal sums the smallest sorted
    positions (integer-valued scores make ties exact)."""
    rng = np.random.default_rng(52)
    for trial in range(30):
        T = int(rng.integers(6, 13)); ks, kr = 1, 2; kmid = int(rng.integers(1, 5)); B = ks + kr + kmid
        S = np.zeros((1, 1, T))
        S[0, 0] = rng.integers(0, 4, size=T).astype(np.float64)
        w = _tiny(0, hq=1, hkv=1, d=8, ctx=(T,), ql=(1,), B=B, k_sink=ks, k_recent=kr)
        idx, n_idx = oracle.select(w, S, lib=lib)
        s_end, r_start = _spans(T, ks, kr)
        mid = list(range(s_end, r_start))
        take = min(kmid, len(mid))
        best = max(itertools.combinations(mid, take),
                   key=lambda sub: (sum(S[0, 0, i] for i in sub), [-i for i in sub]))
        ref = sorted(set(range(s_end)) | set(best) | set(range(r_start, T)))
        assert list(idx[0, 0, :n_idx[0]]) == ref, (S[0, 0], ref, idx[0, 0, :n_idx[0]])


def pin_select_special_cases(lib):
    rng = np.random.default_rng(53)
    T = 50
    S = np.zeros((1, 1, T)); S[0, 0] = rng.random(T)
    w = _tiny(0, hq=1, hkv=1, d=8, ctx=(T,), ql=(1,))
    # budget >= T: every position
    idx, n = oracle.select(w, S, k_sink=4, k_recent=8, budget=T, lib=lib)
    assert n[0] == T and np.array_equal(idx[0, 0, :T], np.arange(T))
    idx, n = oracle.select(w, S, k_sink=4, k_recent=8, budget=T + 17, lib=lib)
    assert n[0] == T and np.array_equal(idx[0, 0, :T], np.arange(T))
    # K_mid = 0: sink and recent only
    idx, n = oracle.select(w, S, k_sink=4, k_recent=8, budget=12, lib=lib)
    assert list(idx[0, 0, :n[0]]) == list(range(4)) + list(range(T - 8, T))
    # all scores equal: the lowest K_mid middle positions
    S1 = np.ones((1, 1, T))
    idx, n = oracle.select(w, S1, k_sink=4, k_recent=8, budget=20, lib=lib)
    assert list(idx[0, 0, :n[0]]) == list(range(12)) + list(range(T - 8, T))
    # T shorter than the sink
    idx, n = oracle.select(w, S, ctx_len=np.array([3]), k_sink=4, k_recent=8, budget=20,
                           lib=lib)
    assert list(idx[0, 0, :n[0]]) == [0, 1, 2]
    # recent overlapping the sink
    idx, n = oracle.select(w, S, ctx_len=np.array([10]), k_sink=4, k_recent=8, budget=13,
                           lib=lib)
    assert list(idx[0, 0, :n[0]]) == list(range(10))
    # index counts
    for T_, ks, kr, B in [(50, 4, 8, 20), (3, 4, 8, 20), (10, 4, 8, 13), (4096, 4, 32, 256),
                          (32768, 4, 32, 2048)]:
        cnt = oracle.index_count(T_, ks, kr, B, lib=lib)
        s_end, r_start = _spans(T_, ks, kr)
        assert cnt == s_end + min(B - ks - kr, r_start - s_end) + (T_ - r_start)
    assert oracle.index_count(32768, 4, 32, 2048, lib=lib) == 2048
    assert oracle.index_count(100, 4, 32, 2048, lib=lib) == 100


# ---------------------------------------------------------------------------
# draft (Eq. 5)
# ---------------------------------------------------------------------------

def pin_draft_matches_sdpa(lib):
    rng = np.random.default_rng(61)
    w = _tiny(62, hq=8, hkv=2, ctx=(70, 33), ql=(1, 1), B=24)
    idx = np.zeros((2, 2, 24), dtype=np.int32)
    n_idx = np.array([24, 19], dtype=np.int32)
    for b in range(2):
        for c in range(2):
            idx[b, c, :n_idx[b]] = np.sort(rng.choice(int(w.ctx_len[b]), n_idx[b], replace=False))
    out = oracle.draft(w, idx, n_idx, lib=lib)
    q = _bf16_to_t64(w.q_draft); k = _bf16_to_t64(w.k); v = _bf16_to_t64(w.v)
    for b in range(2):
        n = int(n_idx[b])
        for h in range(8):
            c = h // 4
            I = torch.from_numpy(idx[b, c, :n].astype(np.int64))
            o = F.scaled_dot_product_attention(q[b, h][None, None, None], k[b, c, I][None, None],
                                               v[b, c, I][None, None], scale=w.sm_scale)
            assert (out[b, h] - o[0, 0, 0].numpy()).__abs__().max() < 1e-12


def pin_draft_full_equals_dense(lib):
    """With every position selected, draft attention is dense attention: it equals
    verify with a single query row (no causal restriction then applies)."""
    w = _tiny(63, hq=8, hkv=2, ctx=(45,), ql=(1,), B=45)
    T = 45
    idx = np.arange(T, dtype=np.int32)[None, None, :].repeat(2, axis=1)
    n_idx = np.array([T], dtype=np.int32)
    qv = w.q.copy()
    qv[0, 0] = w.q_draft[0]
    out_d = oracle.draft(w, idx, n_idx, lib=lib)
    out_v, _ = oracle.verify(w, q=qv, lib=lib)
    assert np.abs(out_d[0] - out_v[0, 0]).max() < 1e-12
    ref = _sdpa_verify(w, q_bits=qv)
    assert np.abs(out_d[0] - ref[0, 0]).max() < 1e-12


def pin_draft_permutation(lib):
    rng = np.random.default_rng(64)
    w = _tiny(65, hq=4, hkv=2, ctx=(60,), ql=(1,), B=20)
    idx = np.zeros((1, 2, 20), dtype=np.int32)
    for c in range(2):
        idx[0, c] = rng.choice(60, 20, replace=False)
    n_idx = np.array([20], dtype=np.int32)
    o1 = oracle.draft(w, idx, n_idx, lib=lib)
    o2 = oracle.draft(w, idx[:, :, ::-1].copy(), n_idx, lib=lib)
    assert np.abs(o1 - o2).max() < 1e-12
    # V = 1 gives 1
    v1 = np.full_like(w.v, f32_to_bf16_bits(np.float32(1.0)))
    o3 = oracle.draft(w, idx, n_idx, v=v1, lib=lib)
    assert np.abs(o3 - 1.0).max() < 1e-12


# ---------------------------------------------------------------------------
# draft round (Sec. 3.1 drafting loop over the Eq. 5 view, recent window slid)
# ---------------------------------------------------------------------------

def pin_draft_step_first_matches_sdpa(lib):
    """Before any token is drafted the step is Eq. 5 over the select output:
    SDPA over exactly those rows."""
    rng = np.random.default_rng(71)
    w = _tiny(72, hq=8, hkv=2, ctx=(90, 41), ql=(1, 1), B=24, k_sink=3, k_recent=6)
    scores = rng.random((2, 2, w.max_ctx))
    idx, n_idx = oracle.select(w, scores, lib=lib)
    out = oracle.draft_step(w, idx, w.ctx_len, w.ctx_len, lib=lib)
    q = _bf16_to_t64(w.q_draft); k = _bf16_to_t64(w.k); v = _bf16_to_t64(w.v)
    for b in range(2):
        for h in range(8):
            c = h // 4
            I = torch.from_numpy(idx[b, c, :n_idx[b]].astype(np.int64))
            o = F.scaled_dot_product_attention(q[b, h][None, None, None], k[b, c, I][None, None],
                                               v[b, c, I][None, None], scale=w.sm_scale)
            assert np.abs(out[b, h] - o[0, 0, 0].numpy()).max() < 1e-12


def pin_draft_step_worked_example(lib):
    """Hand-worked sets.  T = 20, K_sink = 2, K_recent = 4, budget 9 (K_mid = 3),
    middle span [2, 16) with the three largest scores at 5, 9, 13: the index set
    is {0, 1, 5, 9, 13, 16..19}.  After i drafted tokens the recent window is
    [16 + i, 20 + i).  A second sequence with T = 3 has sink {0, 1}, recent {2}
    and window [max(2, T + i - 4), T + i): it grows to four positions and then
    drops position 2.  With K = 0 the attention is uniform and with one-hot V
    rows (row t = e_t) the output is 1/|S| exactly on the step's set."""
    w = _tiny(73, hq=2, hkv=1, ctx=(24, 24), ql=(1, 1), B=9, k_sink=2, k_recent=4)
    scores = np.full((2, 1, 24), 0.1)
    scores[0, 0, [5, 9, 13]] = [0.9, 0.8, 0.7]
    idx, n_idx = oracle.select(w, scores, ctx_len=np.array([20, 3]), lib=lib)
    assert list(idx[0, 0, :n_idx[0]]) == [0, 1, 5, 9, 13, 16, 17, 18, 19]
    assert list(idx[1, 0, :n_idx[1]]) == [0, 1, 2]
    k0 = np.zeros_like(w.k)
    v1 = np.zeros_like(w.v)
    one = f32_to_bf16_bits(np.float32(1.0))
    for t in range(24):
        v1[:, :, t, t] = one
    expect = {(0, 20): [0, 1, 5, 9, 13, 16, 17, 18, 19],
              (0, 21): [0, 1, 5, 9, 13, 17, 18, 19, 20],
              (0, 22): [0, 1, 5, 9, 13, 18, 19, 20, 21],
              (0, 24): [0, 1, 5, 9, 13, 20, 21, 22, 23],
              (1, 3): [0, 1, 2], (1, 5): [0, 1, 2, 3, 4], (1, 6): [0, 1, 2, 3, 4, 5],
              (1, 7): [0, 1, 3, 4, 5, 6]}
    for cur0, cur1 in ((20, 3), (21, 5), (22, 6), (24, 7)):
        out = oracle.draft_step(w, idx, [20, 3], [cur0, cur1], k=k0, v=v1, lib=lib)
        for b, cur in ((0, cur0), (1, cur1)):
            want = np.zeros(128)
            S = expect[(b, cur)]
            want[S] = 1.0 / len(S)
            for h in range(2):
                assert np.abs(out[b, h] - want).max() < 1e-15, (b, cur, h)
    # a drafted tail longer than the recent window, or shorter than T, is rejected
    for cur in ([25, 3], [19, 3]):
        try:
            oracle.draft_step(w, idx, [20, 3], cur, lib=lib)
        except ValueError:
            continue
        raise AssertionError(f"cur_len {cur} accepted")


def pin_draft_step_value_one(lib):
    """Softmax weights sum to one: V = 1 gives 1 at every step of a round."""
    rng = np.random.default_rng(74)
    w = _tiny(75, hq=4, hkv=2, ctx=(64, 64), ql=(1, 1), B=20, k_sink=2, k_recent=5)
    scores = rng.random((2, 2, 64))
    base = np.array([50, 17], dtype=np.int32)
    idx, _ = oracle.select(w, scores, ctx_len=base, lib=lib)
    v1 = np.full_like(w.v, f32_to_bf16_bits(np.float32(1.0)))
    for i in range(6):
        o = oracle.draft_step(w, idx, base, base + i, v=v1, lib=lib)
        assert np.abs(o - 1.0).max() < 1e-12


def pin_draft_step_heads(lib):
    """The draft-round step with one index set per query head: (1) when every
    head of a group carries its KV head's set it is the per-KV-head step;
    (2) before any drafted token it is the per-head Eq. 5 draft over those
    sets; (3) hand-worked sets: with K = 0 and one-hot V rows each head's output
    is uniform exactly on its own fixed rows plus the shared slid window."""
    rng = np.random.default_rng(94)
    w = _tiny(95, hq=8, hkv=2, ctx=(64, 64), ql=(1, 1), B=20, k_sink=2, k_recent=5)
    base = np.array([50, 17], dtype=np.int32)
    idx_kv, _ = oracle.select(w, rng.random((2, 2, 64)), ctx_len=base, lib=lib)
    shared = np.repeat(idx_kv, 4, axis=1)                        # [2][8][B]
    for i in range(6):
        a = oracle.draft_step(w, shared, base, base + i, per_head=True, lib=lib)
        b = oracle.draft_step(w, idx_kv, base, base + i, lib=lib)
        assert np.abs(a - b).max() < 1e-15
    # per-head sets from per-head scores (a select over the query heads as units)
    wh = _tiny(95, hq=8, hkv=8, ctx=(64, 64), ql=(1, 1), B=20, k_sink=2, k_recent=5)
    idx_h, n_h = oracle.select(wh, rng.random((2, 8, 64)), ctx_len=base, lib=lib)
    assert len(set(map(tuple, idx_h[0, :, :n_h[0]].tolist()))) > 1      # the sets differ
    first = oracle.draft_step(w, idx_h, base, base, per_head=True, lib=lib)
    assert np.abs(first - oracle.draft_heads(w, idx_h, n_h, lib=lib)).max() < 1e-15
    # hand-worked: T = 20, sink 2, recent 4, budget 8 (K_mid 2); head 0 keeps
    # {5, 9}, head 1 {7, 13}; after i drafted tokens the window is [16+i, 20+i)
    w2 = _tiny(96, hq=2, hkv=1, ctx=(24,), ql=(1,), B=8, k_sink=2, k_recent=4)
    idx2 = np.array([[[0, 1, 5, 9, 16, 17, 18, 19], [0, 1, 7, 13, 16, 17, 18, 19]]],
                    dtype=np.int32)
    k0 = np.zeros_like(w2.k)
    v1 = np.zeros_like(w2.v)
    one = f32_to_bf16_bits(np.float32(1.0))
    for t in range(24):
        v1[:, :, t, t] = one
    for i in (0, 1, 4):
        out = oracle.draft_step(w2, idx2, [20], [20 + i], k=k0, v=v1, per_head=True, lib=lib)
        for h, fixed in ((0, [0, 1, 5, 9]), (1, [0, 1, 7, 13])):
            S = fixed + list(range(16 + i, 20 + i))
            want = np.zeros(128)
            want[S] = 1.0 / len(S)
            assert np.abs(out[0, h] - want).max() < 1e-15, (h, i)


# ---------------------------------------------------------------------------
# per-query-head scores and draft (Eq. 3 / Eq. 5 per attention head)
# ---------------------------------------------------------------------------

def pin_head_scores_match_softmax(lib):
    """Per-head Eq. 3 against torch.softmax weights of each query head, the
    per-head mass min(W, q), and the group sum against the per-KV-head scores."""
    w = _tiny(91, hq=8, hkv=2, ctx=(50, 33), ql=(5, 3), window=4)
    S = oracle.head_scores(w, lib=lib)
    q = _bf16_to_t64(w.q)
    k = _bf16_to_t64(w.k)
    g = w.group
    for b in range(w.batch):
        T, nq = int(w.ctx_len[b]), int(w.q_len[b])
        wn = min(w.window, nq)
        for h in range(w.n_q_heads):
            c = h // g
            logits = (q[b, nq - wn:nq, h, :] @ k[b, c, :T].T) * w.sm_scale     # [wn, T]
            rows = torch.arange(nq - wn, nq) + (T - nq)
            mask = torch.arange(T)[None, :] <= rows[:, None]
            P = torch.softmax(logits.masked_fill(~mask, -math.inf), dim=-1)
            assert np.abs(S[b, h, :T] - P.sum(dim=0).numpy()).max() < 1e-12
            assert abs(S[b, h, :T].sum() - wn) < 1e-10
    _, Skv = oracle.verify(w, lib=lib)
    Sg = S.reshape(w.batch, w.n_kv_heads, g, w.max_ctx).sum(axis=2)
    assert np.abs(Sg - Skv).max() < 1e-12


def pin_draft_heads(lib):
    """Per-head draft against SDPA per head; with one set shared by a group's
    heads it is the per-KV-head draft."""
    rng = np.random.default_rng(92)
    w = _tiny(93, hq=8, hkv=2, ctx=(70, 40), ql=(1, 1), B=16)
    n_idx = np.array([16, 11], dtype=np.int32)
    idx = np.zeros((2, 8, 16), dtype=np.int32)
    for b in range(2):
        for h in range(8):
            idx[b, h, :n_idx[b]] = np.sort(rng.choice(int(w.ctx_len[b]), n_idx[b], replace=False))
    out = oracle.draft_heads(w, idx, n_idx, lib=lib)
    qd = _bf16_to_t64(w.q_draft); k = _bf16_to_t64(w.k); v = _bf16_to_t64(w.v)
    for b in range(2):
        for h in range(8):
            c = h // 4
            I = torch.from_numpy(idx[b, h, :n_idx[b]].astype(np.int64))
            o = F.scaled_dot_product_attention(qd[b, h][None, None, None], k[b, c, I][None, None],
                                               v[b, c, I][None, None], scale=w.sm_scale)
            assert np.abs(out[b, h] - o[0, 0, 0].numpy()).max() < 1e-12
    shared = idx.reshape(2, 2, 4, 16)[:, :, 0, :]                  # head 4c's set for the group
    per_head = np.repeat(shared, 4, axis=1)
    o1 = oracle.draft_heads(w, per_head, n_idx, lib=lib)
    o2 = oracle.draft(w, shared, n_idx, lib=lib)
    assert np.abs(o1 - o2).max() < 1e-12


# ---------------------------------------------------------------------------
# around the path: token entropy and greedy acceptance
# ---------------------------------------------------------------------------

def pin_row_stats_library(lib):
    """Entropy against scipy (softmax, then Shannon entropy in nats) and argmax
    against numpy (first occurrence), for bf16 and fp32 logits of several scales."""
    from scipy.special import softmax
    from scipy.stats import entropy
    rng = np.random.default_rng(81)
    V = 1000
    x = rng.standard_normal((6, V)) * np.array([0.1, 1.0, 3.0, 10.0, 30.0, 1.0])[:, None]
    x[5, 17] = 40.0                                      # a peaked row
    for logits in (f32_to_bf16_bits(x.astype(np.float32)), x.astype(np.float32)):
        H, a = oracle.row_stats(logits, lib=lib)
        xs = (logits.astype(np.uint32) << 16).view(np.float32).astype(np.float64) \
            if logits.dtype == np.uint16 else logits.astype(np.float64)
        for r in range(6):
            want = entropy(softmax(xs[r]))
            assert abs(H[r] - want) <= 1e-12 * max(1.0, want), (r, H[r], want)
            assert a[r] == int(np.argmax(xs[r]))
    # only the first vocab entries of a row count
    xpad = np.concatenate([x.astype(np.float32), np.full((6, 8), 99.0, np.float32)], axis=1)
    H2, a2 = oracle.row_stats(xpad, vocab=V, lib=lib)
    H1, a1 = oracle.row_stats(x.astype(np.float32), lib=lib)
    assert np.array_equal(a1, a2) and np.abs(H1 - H2).max() < 1e-12


def pin_row_stats_closed_forms(lib):
    V = 4096
    x = np.zeros((3, V), dtype=np.float32)              # uniform: ln V, ties to index 0
    c = 5.0
    x[1, 100] = c                                        # one raised logit
    x[2, [9, 5, 3000]] = [2.0, 2.0, 1.0]                 # tie at the max: the lower index
    H, a = oracle.row_stats(x, lib=lib)
    assert abs(H[0] - math.log(V)) < 1e-12 and a[0] == 0
    p1 = math.exp(c) / (math.exp(c) + V - 1)
    want = -p1 * math.log(p1) - (1 - p1) * math.log((1 - p1) / (V - 1))
    assert abs(H[1] - want) < 1e-11 and a[1] == 100     # (a 4096-term fp64 sum)
    assert a[2] == 5


def pin_greedy_accept_worked(lib):
    """Row j's argmax is planted at t_j; the drafts agree with the first m rows."""
    V, max_k = 300, 5
    rng = np.random.default_rng(82)
    t = rng.integers(0, V, size=(4, max_k + 1))
    x = rng.standard_normal((4, max_k + 1, V)).astype(np.float32)
    for b in range(4):
        for j in range(max_k + 1):
            x[b, j, t[b, j]] = 10.0
    draft = t[:, :max_k].copy()
    draft[0, 3] = (t[0, 3] + 1) % V                      # disagrees at 3: m = 3, next t_3
    k_len = np.array([5, 5, 2, 0])                       # seq 1 agrees everywhere: bonus t_5
    draft[2, 2:] = -1                                    # past k: never read
    m, nxt = oracle.greedy_accept(x, draft, k_len, lib=lib)
    assert list(m) == [3, 5, 2, 0]
    assert list(nxt) == [t[0, 3], t[1, 5], t[2, 2], t[3, 0]]
    # a tie at the max is read as its lower index
    x[1, 1, :] = 0.0
    x[1, 1, [7, 250]] = 10.0
    draft[1, 1] = 250
    m, nxt = oracle.greedy_accept(x, draft, k_len, lib=lib)
    assert m[1] == 1 and nxt[1] == 7


# ---------------------------------------------------------------------------
# speculative sampling (the distribution-preserving verification rule)
# ---------------------------------------------------------------------------

def _log_rows(*probs):
    return np.log(np.array(probs, dtype=np.float64)).astype(np.float32)


def pin_spec_accept_worked(lib):
    """Hand-worked: V = 3, two drafted tokens.  Target rows p0 = (.5, .3, .2),
    p1 = (.1, .6, .3), p2 = (.2, .2, .6); drafter rows q0 = (.25, .5, .25),
    q1 = (.3, .3, .4); drafted tokens 1 (p/q = .6) and 2 (p/q = .75)."""
    t = _log_rows([.5, .3, .2], [.1, .6, .3], [.2, .2, .6])[None]
    d = _log_rows([.25, .5, .25], [.3, .3, .4])[None]
    x = np.array([[1, 2]])
    def run(u_acc, u_smp, k=2):
        m, n = oracle.spec_accept(t, d, x, [k], 1.0, np.array([u_acc]), np.array([u_smp]), lib=lib)
        return int(m[0]), int(n[0])
    # both pass; bonus from p2 = (.2, .2, .6): cumulative (.2, .4, 1), .3 -> 1
    assert run([.5, .7], .3) == (2, 1)
    assert run([.5, .7], .41) == (2, 2)
    # the first fails (.65 >= .6): residual max(0, p0 - q0) = (.25, 0, 0) -> 0
    assert run([.65, .1], .99) == (0, 0)
    # the second fails (.8 >= .75): residual max(0, p1 - q1) = (0, .3, 0) -> 1,
    # even for u = 0 (the first index whose cumulative mass exceeds 0)
    assert run([.1, .8], .0) == (1, 1)
    assert run([.1, .8], .999) == (1, 1)
    # nothing drafted: the token comes from p0 = (.5, .3, .2): .9 -> 2, .5 -> 1
    assert run([.9, .9], .9, k=0) == (0, 2)
    assert run([.9, .9], .55, k=0) == (0, 1)
    assert run([.9, .9], .45, k=0) == (0, 0)


def pin_spec_accept_identical_distributions(lib):
    """A drafter equal to the target passes every token (u q < p = q for u < 1),
    and the bonus token is drawn from the last target row by inversion."""
    rng = np.random.default_rng(91)
    batch, max_k, V = 5, 4, 200
    t = (rng.standard_normal((batch, max_k + 1, V)) * 2).astype(np.float32)
    d = t[:, :max_k].copy()
    x = rng.integers(0, V, (batch, max_k))
    k_len = np.array([4, 3, 0, 1, 4])
    u_acc = rng.random((batch, max_k)) * 0.999
    u_smp = rng.random(batch)
    m, nxt = oracle.spec_accept(t, d, x, k_len, 0.7, u_acc, u_smp, lib=lib)
    assert np.array_equal(m, k_len)
    for b in range(batch):
        z = t[b, k_len[b]].astype(np.float64) / 0.7
        p = np.exp(z - z.max())
        c = np.cumsum(p / p.sum())
        assert nxt[b] == int(np.searchsorted(c, u_smp[b], side="right"))


def pin_spec_accept_preserves_target_distribution(lib):
    """The committed first token is distributed as the target's p0 whatever the
    drafter's q0.  Over a grid of N uniforms: a(x) = the fraction with which
    drafted token x passes, R(y) = the fraction of residual draws giving y
    (a drafted token that always fails, a grid of draw uniforms).  Then
    P(token = y) = sum_x q0(x) [a(x) [y = x] + (1 - a(x)) R(y)] must equal
    p0(y) to within the grid's resolution."""
    N = 4000
    grid = (np.arange(N) + 0.5) / N
    for seed in (92, 93, 94):
        rng = np.random.default_rng(seed)
        V = 6
        t = np.log(np.stack([rng.dirichlet(np.ones(V)), rng.dirichlet(np.ones(V))]))[None]
        t = t.astype(np.float32)
        d = np.log(rng.dirichlet(np.ones(V)))[None, None].astype(np.float32)
        p0 = np.exp(t[0, 0].astype(np.float64)); p0 /= p0.sum()
        q0 = np.exp(d[0, 0].astype(np.float64)); q0 /= q0.sum()
        tb, db, ones = np.repeat(t, N, axis=0), np.repeat(d, N, axis=0), np.ones(N, np.int32)
        a = np.zeros(V)
        for xv in range(V):
            m, _ = oracle.spec_accept(tb, db, np.full((N, 1), xv), ones, 1.0, grid[:, None],
                                      grid, lib=lib)
            a[xv] = m.mean()
        x_fail = int(np.argmin(p0 / q0))          # p0 < q0 there: u just below 1 fails
        m, y = oracle.spec_accept(tb, db, np.full((N, 1), x_fail), ones, 1.0,
                                  np.full((N, 1), 1.0 - 1e-12), grid, lib=lib)
        assert not m.any()
        R = np.bincount(y, minlength=V) / N
        prob = (q0 * a) + (q0 * (1 - a)).sum() * R
        assert np.abs(prob - p0).max() < 3.0 / N, (prob, p0)
        # and each part separately: the pass rate min(1, p/q), the residual's shape
        assert np.abs(a - np.minimum(1.0, p0 / q0)).max() < 1.5 / N
        r = np.maximum(p0 - q0, 0.0)
        assert np.abs(R - r / r.sum()).max() < 1.5 / N


def pin_spec_accept_temperature(lib):
    """Only logits / tau matter: (2 x, tau = 2) draws exactly what (x, tau = 1) does."""
    rng = np.random.default_rng(95)
    batch, max_k, V = 6, 5, 64
    t = rng.standard_normal((batch, max_k + 1, V)).astype(np.float32)
    d = (t[:, :max_k] + 0.7 * rng.standard_normal((batch, max_k, V))).astype(np.float32)
    x = rng.integers(0, V, (batch, max_k))
    k_len = np.array([5, 5, 3, 1, 0, 2])
    u_acc, u_smp = rng.random((batch, max_k)), rng.random(batch)
    a = oracle.spec_accept(t, d, x, k_len, 1.0, u_acc, u_smp, lib=lib)
    b = oracle.spec_accept(2 * t, 2 * d, x, k_len, 2.0, u_acc, u_smp, lib=lib)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    assert len(set(a[0].tolist())) > 1   # the draws differ between sequences


def pin_spec_accept_greedy_limit(lib):
    """As tau -> 0 both distributions become one-hot at their argmax: a drafted
    token equal to the drafter's argmax passes exactly when it is the target's
    argmax, and the next token is the target argmax: greedy verification."""
    rng = np.random.default_rng(96)
    batch, max_k, V = 8, 6, 50
    t = rng.standard_normal((batch, max_k + 1, V)).astype(np.float32)
    d = rng.standard_normal((batch, max_k, V)).astype(np.float32)
    am = t.argmax(axis=2)
    for b in range(batch):   # agree with the target on a prefix of random length
        for j in range(rng.integers(0, max_k + 1)):
            d[b, j, am[b, j]] = d[b, j].max() + 1.0
    x = d.argmax(axis=2)
    k_len = rng.integers(0, max_k + 1, batch)
    m, nxt = oracle.spec_accept(t, d, x, k_len, 1e-4, rng.random((batch, max_k)),
                                rng.random(batch), lib=lib)
    mg, ng = oracle.greedy_accept(t, x, k_len, lib=lib)
    assert np.array_equal(m, mg) and np.array_equal(nxt, ng)


# ---------------------------------------------------------------------------
# controller (Eq. 6-8)
# ---------------------------------------------------------------------------

def pin_controller_closed_forms(lib):
    # Eq. 6: n identical observations from m0: m_n = beta^n m0 + (1 - beta^n) H
    m, beta, H = 2.0, 0.9, 0.5
    for n in range(1, 8):
        m = oracle.ema(m, H, beta, lib=lib)
        assert abs(m - (beta ** n * 2.0 + (1 - beta ** n) * H)) < 1e-12
    # Eq. 7: equal distances -> 1/2; at the accepted center -> logistic of the gap
    assert abs(oracle.accept_prob(1.0, 0.5, 1.5, lib=lib) - 0.5) < 1e-15
    for gap in (0.1, 1.0, 3.0):
        p = oracle.accept_prob(0.7, 0.7, 0.7 + gap, lib=lib)
        assert abs(p - 1.0 / (1.0 + math.exp(-gap))) < 1e-12
        p = oracle.accept_prob(0.7 + gap, 0.7, 0.7 + gap, lib=lib)
        assert abs(p - 1.0 / (1.0 + math.exp(gap))) < 1e-12
    # far beyond both centers the distances differ by the gap: p = 1/(1+e^{gap})
    assert abs(oracle.accept_prob(10.0, 0.5, 1.5, lib=lib) - 1.0 / (1.0 + math.e)) < 1e-12
    assert oracle.accept_prob(0.0, 0.5, 1.5, lib=lib) > 0.5
    # constant p: geometric series p (1 - p^k) / (1 - p)
    for pc in (0.3, 0.5, 0.9):
        for k in range(0, 9):
            e = oracle.expected_accepted([pc] * max(k, 1), k, lib=lib)
            assert abs(e - pc * (1 - pc ** k) / (1 - pc)) < 1e-12
    # p = 1/2: objective (2 - 2^-k) / (k Cd + Cv)
    for k in range(1, 10):
        v = oracle.step_efficiency([0.5] * k, k, 0.3, 2.0, lib=lib)
        assert abs(v - (2 - 2.0 ** -k) / (k * 0.3 + 2.0)) < 1e-12
    # p = 1: Eq. 1 with alpha = 1 (times 1/Cv): (k + 1) / (k gamma + 1)
    for k in range(1, 10):
        v = oracle.step_efficiency([1.0] * k, k, 0.25, 1.0, lib=lib)
        assert abs(v - (k + 1) / (k * 0.25 + 1)) < 1e-12
    # non-uniform prefix product
    p = [0.9, 0.5, 0.2]
    assert abs(oracle.expected_accepted(p, 3, lib=lib) - (0.9 + 0.45 + 0.09)) < 1e-12
    assert abs(oracle.expected_accepted(p, 2, lib=lib) - (0.9 + 0.45)) < 1e-12


def pin_controller_observe(lib):
    """Eq. 6 over one verification: label means by drafting order, first
    observation sets a label's mean, a label without tokens keeps its state."""
    fresh = [123.0, -5.0, 0.0, 0.0]          # unseen labels: the stored values are stale
    H = [0.2, 0.4, 0.9, 3.0, 5.0]
    st = oracle.ctrl_observe(fresh, H, 3, 0.9, lib=lib)
    assert st[2] == 1.0 and st[3] == 1.0
    assert abs(st[0] - statistics.fmean(H[:3])) < 1e-15
    assert abs(st[1] - statistics.fmean(H[3:])) < 1e-15
    # the accepted tokens are the first ones drafted
    st = oracle.ctrl_observe(fresh, [0.0, 0.0, 0.0, 9.0, 9.0], 3, 0.5, lib=lib)
    assert st[:2] == [0.0, 9.0]
    # a label with no tokens keeps its mean and its seen flag
    st = oracle.ctrl_observe([1.5, 2.5, 1.0, 1.0], [7.0, 8.0], 0, 0.9, lib=lib)
    assert st[0] == 1.5 and abs(st[1] - (0.9 * 2.5 + 0.1 * 7.5)) < 1e-12
    st = oracle.ctrl_observe([1.5, 2.5, 1.0, 0.0], [7.0, 8.0], 2, 0.9, lib=lib)
    assert st[1:] == [2.5, 1.0, 0.0]
    assert oracle.ctrl_observe([1.5, 2.5, 1.0, 1.0], [], 0, 0.9, lib=lib) == [1.5, 2.5, 1.0, 1.0]
    # step response: a label first seen at x0, then n verifications whose
    # tokens of that label all have entropy y, sits at y + (x0 - y) beta^n
    for beta in (0.0, 0.6, 0.9, 1.0):
        st = oracle.ctrl_observe(fresh, [4.0, 4.0, 1.0], 2, beta, lib=lib)
        for n in range(1, 7):
            st = oracle.ctrl_observe(st, [0.5, 0.5, 0.5, 3.0], 3, beta, lib=lib)
            assert abs(st[0] - (0.5 + 3.5 * beta ** n)) < 1e-12
            assert abs(st[1] - (3.0 + (1.0 - 3.0) * beta ** n)) < 1e-12
    # a constant-entropy stream is a fixed point
    st = oracle.ctrl_observe(fresh, [0.7, 0.7], 1, 0.3, lib=lib)
    for _ in range(5):
        st = oracle.ctrl_observe(st, [0.7] * 6, 4, 0.3, lib=lib)
        assert st[:2] == [0.7, 0.7]
    try:
        oracle.ctrl_observe(fresh, [0.1, 0.2], 3, 0.9, lib=lib)
    except ValueError:
        pass
    else:
        raise AssertionError("more accepted than drafted tokens was not refused")


def pin_controller_argmax(lib):
    cands = list(range(1, 21))
    # free drafting with positive acceptance: the longest candidate wins
    assert oracle.choose_k([0.4] * 20, cands, 0.0, 1.0, lib=lib) == 20
    # near-zero acceptance: the shortest candidate wins
    assert oracle.choose_k([1e-9] * 20, cands, 0.1, 1.0, lib=lib) == 1
    # only candidates k <= n are considered
    assert oracle.choose_k([0.99] * 5, cands, 0.01, 1.0, lib=lib) == 5
    assert oracle.choose_k([0.9] * 3, [4, 8], 0.0, 1.0, lib=lib) == -1
    # exact tie (p = 0 beyond the first token, free drafting): the smaller k
    assert oracle.choose_k([0.5, 0.0, 0.0, 0.0], [1, 2, 3, 4], 0.0, 1.0, lib=lib) == 1
    # efficiency inversion: with constant p, extending k pays while the tail
    # acceptance p^k exceeds the marginal cost; compare with enumeration
    rng = np.random.default_rng(71)
    for _ in range(50):
        n = int(rng.integers(1, 21))
        p = rng.random(n)
        cd, cv = float(rng.random() * 0.5), 1.0 + float(rng.random())
        vals = []
        for k in cands:
            if k <= n:
                e = sum(float(np.prod(p[:m])) for m in range(1, k + 1))
                vals.append(((1 + e) / (k * cd + cv), -k))
        best = -max(vals)[1]
        assert oracle.choose_k(list(p), cands, cd, cv, lib=lib) == best
    # lower entropy -> larger accepted probability -> longer k (feedback direction)
    h_acc, h_rej = 0.5, 2.5
    p_lo = [oracle.accept_prob(0.4, h_acc, h_rej, lib=lib)] * 20
    p_hi = [oracle.accept_prob(2.4, h_acc, h_rej, lib=lib)] * 20
    assert oracle.choose_k(p_lo, cands, 0.05, 1.0, lib=lib) > \
        oracle.choose_k(p_hi, cands, 0.05, 1.0, lib=lib)


ALL_PINS = [pin_verify_matches_sdpa, pin_verify_value_one, pin_verify_zero_keys_closed_form,
            pin_verify_planted_key, pin_scores_match_softmax, pin_scores_total_mass,
            pin_scores_permutation, pin_select_lexsort, pin_select_bruteforce_subsets,
            pin_select_special_cases, pin_draft_matches_sdpa, pin_draft_full_equals_dense,
            pin_draft_permutation, pin_draft_step_first_matches_sdpa,
            pin_draft_step_worked_example, pin_draft_step_value_one, pin_draft_step_heads, pin_row_stats_library,
            pin_row_stats_closed_forms, pin_greedy_accept_worked, pin_spec_accept_worked,
            pin_spec_accept_identical_distributions, pin_spec_accept_preserves_target_distribution,
            pin_spec_accept_temperature, pin_spec_accept_greedy_limit, pin_head_scores_match_softmax,
            pin_draft_heads,
            pin_controller_closed_forms, pin_controller_observe, pin_controller_argmax]
