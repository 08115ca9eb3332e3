"""The oracle against its pins (hand-worked examples, closed forms, invariants,
brute force), plus property tests over random shapes and permutations."""
import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import tpdq_oracle as o
from tests import pins


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda p: p.__name__)
def test_pin(pin):
    pin(o)


@settings(max_examples=40, deadline=None)
@given(ng=st.integers(1, 24), g8=st.integers(1, 6), seed=st.integers(0, 2**31 - 1))
def test_reorder_properties(ng, g8, seed):
    """P3 over random K, G (G | K, 8 | G) and random phi."""
    G = 8 * g8
    K = ng * G
    phi = np.random.default_rng(seed).permutation(K)
    g = o.g_idx_actorder(phi, G)
    o.check_groups(g, G)
    P, gs = o.reorder(g)
    assert np.array_equal(gs, o.g_idx_naive(K, G))
    assert np.array_equal(g[P], gs)
    assert np.array_equal(np.sort(P), np.arange(K))


@settings(max_examples=15, deadline=None)
@given(ng=st.integers(1, 6), g8=st.integers(1, 4), n8=st.integers(1, 6), M=st.integers(1, 5),
       seed=st.integers(0, 2**31 - 1))
def test_ordered_equals_actorder_properties(ng, g8, n8, M, seed):
    """P7 over random shapes."""
    from paper_2402_04925_amd import inputs
    G = 8 * g8
    K = ng * G
    N = 8 * n8
    w1, _ = inputs.make_custom(K, N, 0, G, seed % 100000)
    X = inputs.random_activations(M, K, np.random.default_rng(seed))
    ref = o.w4a16_gemm(X, w1.qweight, w1.scales, w1.qzeros, w1.g_idx, round_fp16=False)
    P, gs = o.reorder(w1.g_idx)
    ws = o.permute_rows(dict(qweight=w1.qweight, scales=w1.scales, qzeros=w1.qzeros), P)
    Y = o.w4a16_gemm(X, ws["qweight"], ws["scales"], ws["qzeros"], gs, x_perm=P, round_fp16=False)
    assert np.max(np.abs(Y - ref)) <= 1e-12 * max(1e-30, np.max(np.abs(ref)))


def test_generator_matches_eq3():
    """The input generator's g_idx is Eq. 3 of its phi, for every workload."""
    from paper_2402_04925_amd import inputs
    for name in ("tiny_gemm",):
        w = inputs.WORKLOADS[name]
        w1, _ = inputs.make_workload(w)
        assert np.array_equal(o.g_idx_actorder(w1.phi, w.G), w1.g_idx)
        o.check_groups(w1.g_idx, w.G)


def test_generator_deterministic():
    from paper_2402_04925_amd import inputs
    a, _ = inputs.make_custom(64, 16, 0, 16, 5)
    b, _ = inputs.make_custom(64, 16, 0, 16, 5)
    for f in ("qweight", "scales", "qzeros", "g_idx"):
        assert np.array_equal(getattr(a, f), getattr(b, f))
