"""Branch allocation of Section IV (Eq. 11-14): the oracle against the optimisation it
solves, and the library's integer allocation against the oracle."""
import itertools

import numpy as np
import pytest

import synth
from oracle import allocation as oa
from oracle import model as om
from paper_2609_02514_amd import allocation as al


@pytest.mark.parametrize("alpha,beta", [(0.8, 1.0), (0.6, 0.5), (0.95, 3.0)])
def test_real_allocation_is_the_constrained_optimum(alpha, beta):
    F = oa.real_allocation(24.0, 8, alpha, beta)
    assert abs(F.sum() - 24.0) < 1e-12
    lam = oa.stationarity_multipliers(F, alpha, beta)
    np.testing.assert_allclose(lam, lam[0], rtol=1e-12)           # KKT: one multiplier
    eta = alpha ** (1.0 / (beta + 1.0))
    np.testing.assert_allclose(F[1:] / F[:-1], eta, rtol=1e-12)   # geometric decay
    # budget-preserving perturbations lower the (Lagrangian's) objective
    J = lambda G: -np.sum(alpha ** np.arange(8) * (1 - alpha) * G ** (-beta))
    rng = np.random.default_rng(1)
    for _ in range(200):
        d = rng.normal(size=8) * 0.05
        d -= d.mean()
        assert J(F + d) <= J(F) + 1e-15


def test_uniform_limit_and_hand_vector():
    np.testing.assert_allclose(oa.real_allocation(12.0, 4, 1.0 - 1e-15, 1.0), 3.0, rtol=1e-9)
    # alpha 0.8, beta 1 (eta = 0.8944), B_alloc 24 over 8 depths:
    # real [4.29 3.84 3.43 3.07 2.75 2.46 2.20 1.97] -> floors sum 20 -> +1 at the four
    # largest remainders (depths 7, 1, 4, 5)
    assert oa.integer_allocation(oa.real_allocation(24, 8, 0.8, 1.0), 24) == \
        [4, 4, 3, 3, 3, 3, 2, 2]


def test_library_allocation_matches_oracle():
    for b, g, a, be in itertools.product(range(0, 61, 3), range(1, 11), (0.5, 0.8, 0.95),
                                         (0.5, 1.0, 2.0)):
        f = al.branch_allocation(b, g, al.decay_factor(a, be))
        assert f == oa.integer_allocation(oa.real_allocation(b, g, a, be), b), (b, g, a, be)
        assert sum(f) == b and all(x >= 0 for x in f)
        assert all(f[k] >= f[k + 1] for k in range(g - 1))        # never deeper-heavy
        real = oa.real_allocation(b, g, a, be)
        assert np.all(np.abs(np.array(f) - real) < 1.0)


def test_budget_rule():
    # inverse latency: 2 ms per node -> B = floor((RTT + T_verify) / 2 ms), capped at B_max
    inv = lambda t: t / 2e-3
    assert al.budget(64, inv, 0.050, 0.010) == 30
    assert al.budget(16, inv, 0.050, 0.010) == 16


def test_geometric_workload_tree():
    w = synth.get("8b-geometric")
    assert list(w.fanout) == al.branch_allocation(24, 8, al.decay_factor(0.8, 1.0))
    parents = synth.tree_parents(w)
    assert len(parents) - 1 == 8 + 24
    ch = synth.children_lists(parents)
    main = [0]
    for k, fk in enumerate(w.fanout):
        kids = ch[main[-1]]
        assert len(kids) == 1 + fk                  # main child + F_k alternatives
        main.append(kids[0])
    assert max(om.tree_depths(parents)) == 8
