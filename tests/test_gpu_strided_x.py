"""Activations with a leading dimension larger than K (X cut from a wider
buffer) on every route that gathers X[:, perm]: inside the decode kernel's
LDS (M <= 4), gathered once row-major on grids of more than 512 column tiles
(N = 8320, M <= 4), through the prepared operand (M > 4), through the M-tiled
kernel's row gather (M >= 256), and in the MLP shard. The contract is 16-byte
alignment and ldx % 8 == 0 on every path."""
import numpy as np
import pytest

from oracle import tpdq_oracle as o
from paper_2402_04925_amd import inputs
from tests.gpu_util import TOL_FP16, layer_to_dev, log, np_of, to_dev, torch_dev

pytestmark = pytest.mark.gpu


def _strided(X, dev, pad=8):
    import torch
    M, K = X.shape
    buf = torch.zeros(M, K + pad, dtype=torch.float16, device=dev)
    buf[:, :K] = to_dev(X, dev)
    v = buf[:, :K]
    assert v.stride(0) == K + pad and v.stride(1) == 1
    return v


@pytest.mark.parametrize("K,N,G,M", [(256, 128, 32, 3), (1024, 256, 128, 16), (512, 512, 64, 256),
                                     (8192, 512, 128, 4), (512, 8320, 64, 1), (1024, 8320, 128, 3)])
def test_gather_with_ldx(K, N, G, M):
    import torch
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    log(f"strided X gather K={K} N={N} G={G} M={M}")
    w1, _ = inputs.make_custom(K, N, 0, G, seed=K + M)
    X = inputs.random_activations(M, K, np.random.default_rng(M + 1))
    P, _, _, _, wo, _ = tpdq.reorder(layer_to_dev(w1, dev), layout=tpdq.LAYOUT_TILED)
    Xs = _strided(X, dev)
    Y = tpdq.w4a16_gemm(Xs, wo, tpdq.PATH_ORDERED, x_perm=P)
    torch.cuda.synchronize()
    ref = o.w4a16_gemm(X, w1.qweight, w1.scales, w1.qzeros, w1.g_idx)
    assert o.rel_err(np_of(Y), ref) <= TOL_FP16


@pytest.mark.parametrize("M", [2, 16])
@pytest.mark.parametrize("ordered", [True, False])
def test_mlp_with_ldx(M, ordered):
    import torch
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    K1, N1, N2, G, tp = 1024, 512, 256, 128, 2
    log(f"strided X mlp M={M} ordered={ordered}")
    w1, w2 = inputs.make_custom(K1, N1, N2, G, seed=40 + M)
    X = inputs.random_activations(M, K1, np.random.default_rng(M))
    d1, d2 = layer_to_dev(w1, dev), layer_to_dev(w2, dev)
    Xs = _strided(X, dev)
    eP2, _ = o.reorder(w2.g_idx)
    if ordered:
        P1, _, _, _, w1o, w2o = tpdq.reorder(d1, d2)
        y1, y2 = tpdq.mlp_shard(Xs, w1o.column_shard(0, tp), w2o.row_shard(0, tp, True),
                                tpdq.PATH_ORDERED, P1=P1)
    else:
        y1, y2 = tpdq.mlp_shard(Xs, d1.column_shard(0, tp), d2.row_shard(0, tp, False),
                                tpdq.PATH_ACTORDER)
    torch.cuda.synchronize()
    l1 = (w1.qweight, w1.scales, w1.qzeros, w1.g_idx)
    l2 = (w2.qweight, w2.scales, w2.qzeros, w2.g_idx)
    e1, e2 = o.mlp_rank_from_global(X, l1, l2, 0, tp, ordered, P2=eP2)
    assert o.rel_err(np_of(y1), e1) <= TOL_FP16
    assert o.rel_err(np_of(y2), e2) <= TOL_FP16
