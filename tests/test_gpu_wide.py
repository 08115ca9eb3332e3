"""GPU wide decode kernel (ordered path, tiled weights of at least 64M
elements, or of 16M with row-major X and M > 16; X too large to stage whole in LDS: 8 waves over 128 columns share
the activations through LDS, K split over workgroups when the columns alone
give too few) against the oracle on sampled columns."""
import numpy as np
import pytest

from oracle import tpdq_oracle as o
from paper_2402_04925_amd import inputs
from tests.gpu_util import TOL_FP16, layer_to_dev, log, np_of, sample_cols, to_dev, torch_dev

pytestmark = pytest.mark.gpu

# K, N, G, M: K split in 4 (64 workgroups of columns), ragged N (the last
# workgroup has one tile), two row tiles with G = 32, G = 256 with splits
# starting on odd blocks, and no split (224 workgroups)
SHAPES = [
    (8192, 8192, 128, 8), (8192, 8200, 64, 16), (4096, 16384, 32, 17), (16384, 4096, 256, 32),
    (8192, 28672, 128, 12),
    # 16M to 64M elements: row-major X with two or more row tiles only
    (8192, 3584, 128, 32), (3584, 8192, 128, 64), (6144, 6144, 128, 40),
    # 64M elements at M = 3 and 4, where X would fit in LDS (wide from 3 rows on)
    (8192, 8192, 128, 3), (8192, 8192, 128, 4),
]


@pytest.mark.parametrize("K,N,G,M", SHAPES)
def test_wide_gemm(K, N, G, M):
    """Sorted rows from the GPU reorder, with the X[:, P] gather (the
    prepared operand) and without it (X row-major), each called twice."""
    import torch
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    log(f"wide K={K} N={N} G={G} M={M}")
    w1, _ = inputs.make_custom(K, N, 0, G, seed=K + N + G + M)
    X = inputs.random_activations(M, K, np.random.default_rng(M + 21))
    P, _, _, _, wo, _ = tpdq.reorder(layer_to_dev(w1, dev), layout=tpdq.LAYOUT_TILED)
    Xd = to_dev(X, dev)
    cols = sample_cols(N, np.random.default_rng(K + M + 1))
    ref = o.w4a16_gemm(X, w1.qweight, w1.scales, w1.qzeros, w1.g_idx, cols=cols)
    eP, eg = o.reorder(w1.g_idx)
    ws = o.permute_rows(dict(qweight=w1.qweight, scales=w1.scales, qzeros=w1.qzeros), eP)
    ref2 = o.w4a16_gemm(X, ws["qweight"], ws["scales"], ws["qzeros"], eg, cols=cols)
    for _ in range(2):
        Y = tpdq.w4a16_gemm(Xd, wo, tpdq.PATH_ORDERED, x_perm=P)
        Y2 = tpdq.w4a16_gemm(Xd, wo, tpdq.PATH_ORDERED)
        torch.cuda.synchronize()
        assert o.rel_err(np_of(Y)[:, cols], ref) <= TOL_FP16
        assert o.rel_err(np_of(Y2)[:, cols], ref2) <= TOL_FP16


def test_wide_deterministic():
    """Split-K partials are added in a fixed order: two calls agree bit for bit."""
    import torch
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    K, N, G, M = 8192, 8192, 128, 16
    w1, _ = inputs.make_custom(K, N, 0, G, seed=5)
    X = to_dev(inputs.random_activations(M, K, np.random.default_rng(6)), dev)
    _, _, _, _, wo, _ = tpdq.reorder(layer_to_dev(w1, dev), layout=tpdq.LAYOUT_TILED)
    a = np_of(tpdq.w4a16_gemm(X, wo, tpdq.PATH_ORDERED))
    b = np_of(tpdq.w4a16_gemm(X, wo, tpdq.PATH_ORDERED))
    torch.cuda.synchronize()
    assert np.array_equal(a.view(np.uint16), b.view(np.uint16))
