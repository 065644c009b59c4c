"""The paper's own protocol (scalar q-hat uplink, k-sparse downlink, edge-side resampling,
Algorithm 1): pins of the oracle's reading, and the edge resampler (product code,
CPU by design) against it."""
import numpy as np
import pytest

from oracle import verify as ov
from paper_2609_02514_amd import edge


def test_edge_resample_hand_vector():
    # payload ids [3, 0, 1] with probs [.5, .3, .2]; draft q: q(0)=.4, q(1)=.1, q(3)=.2
    # residual on the payload: {0: 0, 1: .1, 3: .3} -> law {1: .25, 3: .75} (ids ascending)
    ids, probs = [3, 0, 1], [0.5, 0.3, 0.2]
    q = np.array([0.4, 0.1, 0.3, 0.2, 0.0])
    assert ov.edge_resample(ids, probs, q, 0.2) == 1
    assert ov.edge_resample(ids, probs, q, 0.3) == 3
    # full acceptance: P_hat itself, ids ascending [0, 1, 3], running mass .3 .5 1.0
    assert ov.edge_resample(ids, probs, q, 0.2, rejected=False) == 0
    assert ov.edge_resample(ids, probs, q, 0.4, rejected=False) == 1
    assert ov.edge_resample(ids, probs, q, 0.6, rejected=False) == 3


def _nucleus_payload(p, k):
    order = ov.sorted_order(p)
    ids = order[:k]
    w = p[ids]
    return ids, w / w.sum()


def test_edge_resample_is_exact_when_the_payload_covers_the_support():
    """With every id of non-zero p in the payload, the sparse residual law equals the exact
    residual law max(0, p - q)/sum (midpoint grid of uniforms through the oracle code)."""
    rng = np.random.default_rng(5)
    M = 4000
    for _ in range(20):
        V = 8
        p = rng.dirichlet(np.ones(V) * 0.7)
        p[rng.integers(V)] = 0.0
        p /= p.sum()
        q = rng.dirichlet(np.ones(V))
        ids, probs = _nucleus_payload(p, V)
        law = np.zeros(V)
        for m in range(M):
            law[ov.edge_resample(ids, probs, q, (m + 0.5) / M)] += 1.0 / M
        np.testing.assert_allclose(law, ov.exact_residual_law(p, q), atol=2.0 / M)


def test_truncated_payload_has_a_measurable_gap():
    """A payload smaller than the support changes the law (the paper is silent on this);
    the total-variation gap is what the GPU test reports on real rows."""
    p = np.array([0.4, 0.3, 0.2, 0.1])
    q = np.array([0.1, 0.1, 0.1, 0.7])
    ids, probs = _nucleus_payload(p, 2)                 # {0: 4/7, 1: 3/7}
    sid, w = edge.residual_law(ids, probs, q)
    sparse = np.zeros(4)
    sparse[sid] = w
    tv = 0.5 * np.abs(sparse - ov.exact_residual_law(p, q)).sum()
    assert tv > 0.05
    ids4, probs4 = _nucleus_payload(p, 4)
    sid, w = edge.residual_law(ids4, probs4, q)
    full = np.zeros(4)
    full[sid] = w
    assert 0.5 * np.abs(full - ov.exact_residual_law(p, q)).sum() < 1e-12


def test_accept_scalar_matches_dense_accept():
    rng = np.random.default_rng(9)
    for _ in range(200):
        p = rng.dirichlet(np.ones(6))
        q = rng.dirichlet(np.ones(6))
        x, u = int(rng.integers(6)), float(rng.random())
        assert ov.accept_scalar(p, x, float(q[x]), u) == ov.accept_token(p, q, x, u)


@pytest.mark.parametrize("rejected", [True, False])
def test_edge_module_matches_oracle(rejected):
    rng = np.random.default_rng(11 + rejected)
    for _ in range(300):
        V, k = 50, int(rng.integers(1, 12))
        p = rng.dirichlet(np.ones(V) * 0.3)
        q = rng.dirichlet(np.ones(V) * 0.3)
        ids, probs = _nucleus_payload(p, k)
        u = float(rng.random())
        assert edge.resample(ids, probs, q, u, rejected) == \
            ov.edge_resample(ids, probs, q, u, rejected)
