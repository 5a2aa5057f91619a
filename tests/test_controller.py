"""Host controller (Eq. 6-8) of the C library against the CPU oracle."""
import math

import numpy as np
import pytest

import oracle
from paper_2607_27735_amd import binding as B


@pytest.fixture(scope="module")
def lib():
    return B.load()


def test_cold_start_returns_default(lib):
    c = B.Controller(beta=0.9, candidates=range(1, 21), k_default=4)
    assert c.choose_k([0.1] * 20, 0.1, 1.0) == 4
    c.observe([0.2, 0.3], 2)             # accepted only
    assert c.choose_k([0.1] * 20, 0.1, 1.0) == 4
    assert c.accept_prob(0.2) == 0.5
    c.observe([0.2, 3.0], 1)             # now both classes seen
    assert c.choose_k([0.1] * 20, 0.1, 1.0) != -1


def test_observe_matches_oracle():
    """Eq. 6 with the label means of one verification (the oracle's
    oracle_ctrl_observe), over random verifications including empty labels."""
    rng = np.random.default_rng(1)
    beta = 0.85
    c = B.Controller(beta=beta)
    st_ref = [0.0, 0.0, 0.0, 0.0]
    for _ in range(60):
        n = int(rng.integers(0, 12))
        m = int(rng.integers(0, n + 1))
        H = list(rng.random(n) * 4)
        c.observe(H, m)
        st_ref = oracle.ctrl_observe(st_ref, H, m, beta)
        st = c.state()
        assert st[2] == bool(st_ref[2]) and st[3] == bool(st_ref[3])
        if st_ref[2]:
            assert abs(st[0] - st_ref[0]) < 1e-12
        if st_ref[3]:
            assert abs(st[1] - st_ref[1]) < 1e-12


def test_accept_prob_matches_oracle():
    c = B.Controller()
    for h_acc, h_rej in [(0.5, 2.0), (1.5, 0.2), (1.0, 1.0)]:
        c.set_state(h_acc, h_rej, True, True)
        for H in np.linspace(-1, 5, 61):
            assert abs(c.accept_prob(H) - oracle.accept_prob(H, h_acc, h_rej)) < 1e-12
    # far from both centers the printed ratio underflows; the library's form does not
    c.set_state(0.0, 1.0, True, True)
    p = c.accept_prob(2000.0)
    assert math.isfinite(p) and abs(p - 1 / (1 + math.e)) < 1e-12


def test_choose_k_matches_oracle():
    rng = np.random.default_rng(2)
    cands = list(range(1, 21))
    c = B.Controller(candidates=cands)
    for _ in range(200):
        h_acc, h_rej = float(rng.random() * 2), float(rng.random() * 2 + 1)
        c.set_state(h_acc, h_rej, True, True)
        n = int(rng.integers(1, 21))
        H = list(rng.random(n) * 3)
        cd, cv = float(rng.random() * 0.3), 1.0 + float(rng.random())
        k = c.choose_k(H, cd, cv)
        p = [oracle.accept_prob(h, h_acc, h_rej) for h in H]
        vals = {kk: oracle.step_efficiency(p, kk, cd, cv) for kk in cands if kk <= n}
        best = max(vals.values())
        assert k in vals and vals[k] >= best * (1 - 1e-12)
        ko = oracle.choose_k(p, cands, cd, cv)
        if abs(vals[ko] - sorted(vals.values())[-2 if len(vals) > 1 else -1]) > 1e-9:
            assert k == ko


def test_choose_k_errors_and_candidates():
    c = B.Controller(candidates=[4, 8, 12], k_default=8)
    c.set_state(0.5, 2.0, True, True)
    with pytest.raises(B.SSLError):
        c.choose_k([0.1, 0.1], 0.1, 1.0)            # no candidate <= 2
    assert c.choose_k([0.1] * 12, 0.0, 1.0) == 12    # free drafting, confident
    with pytest.raises(ValueError):
        B.Controller(candidates=[-1, 2])
    with pytest.raises(ValueError):
        B.Controller(beta=1.5)
    with pytest.raises(B.SSLError):
        c.observe([0.1, 0.2], 3)


@pytest.mark.parametrize("cd,cv", [(0.1, 0.0), (0.1, -1.0), (-0.1, 1.0), (float("nan"), 1.0),
                                   (0.1, float("nan")), (float("inf"), 1.0), (0.1, float("inf"))])
def test_choose_k_rejects_bad_costs(cd, cv):
    """Eq. 8 divides by k C_d + C_v: costs must be finite, C_d >= 0 and C_v > 0."""
    c = B.Controller(candidates=[1, 2, 4], k_default=2)
    c.set_state(0.5, 2.0, True, True)
    with pytest.raises(B.SSLError) as e:
        c.choose_k([0.1] * 4, cd, cv)
    assert e.value.status == B.SSL_ERR_SHAPE
    c.set_state(0.0, 0.0, False, False)            # also before both labels are seen
    with pytest.raises(B.SSLError):
        c.choose_k([0.1] * 4, cd, cv)


def test_feedback_direction():
    """Confident drafts (entropy near the accepted class) lengthen k*, uncertain
    ones shorten it (Sec. 3.3)."""
    c = B.Controller()
    c.set_state(0.3, 2.5, True, True)
    k_conf = c.choose_k([0.3] * 20, 0.05, 1.0)
    k_unsure = c.choose_k([2.4] * 20, 0.05, 1.0)
    assert k_conf > k_unsure
