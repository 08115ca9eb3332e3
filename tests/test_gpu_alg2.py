"""Alg. 2's local data flow on one GPU at TP = 1 (no collectives): Y1 =
X[:, P1] @ W1[P1] with W1's columns in place, then Y2 = Y1[:, P2] @ W2[P2],
through the same entry points (the Y1[:, P2] gather is GEMM2's x_perm).
Against the oracle's Alg. 2, and against Alg. 3 (W1[P1, P2], no gather
between the GEMMs) on the GPU: every output is the same dot product over the
same sorted rows, so the two agree bit for bit."""
import numpy as np
import pytest

from oracle import tpdq_oracle as o
from paper_2402_04925_amd import inputs
from tests.gpu_util import TOL_FP16, layer_to_dev, log, np_of, sample_cols, to_dev, torch_dev

pytestmark = pytest.mark.gpu


def _d(layer):
    return dict(qweight=layer.qweight, scales=layer.scales, qzeros=layer.qzeros)


def _both(tpdq, Xd, d1, d2):
    P1, _, P2, _, w1f, w2o = tpdq.reorder(d1, d2)       # Alg. 3 inputs (the fold)
    P1b, _, _, _, w1o, _ = tpdq.reorder(d1)              # W1[P1], columns in place
    P2b, _, _, _, w2b, _ = tpdq.reorder(d2)              # W2[P2]
    y1, y2 = tpdq.mlp_shard(Xd, w1f, w2o, tpdq.PATH_ORDERED, P1=P1)
    y1n = tpdq.w4a16_gemm(Xd, w1o, tpdq.PATH_ORDERED, x_perm=P1b)
    y2n = tpdq.w4a16_gemm(y1n, w2b, tpdq.PATH_ORDERED, x_perm=P2b)
    return (P1, P2, P1b, P2b), (y1, y2), (y1n, y2n)


@pytest.mark.parametrize("M", [1, 5, 16, 70])
def test_alg2_local_small(M):
    import torch
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    K1, N1, N2, G = 256, 512, 136, 32
    log(f"alg2 local small M={M}")
    w1, w2 = inputs.make_custom(K1, N1, N2, G, seed=40 + M)
    X = inputs.random_activations(M, K1, np.random.default_rng(M + 40))
    Xd = to_dev(X, dev)
    (P1, P2, P1b, P2b), (y1, y2), (y1n, y2n) = _both(tpdq, Xd, layer_to_dev(w1, dev),
                                                     layer_to_dev(w2, dev))
    torch.cuda.synchronize()
    assert torch.equal(P1, P1b) and torch.equal(P2, P2b)
    eP1, _ = o.reorder(w1.g_idx)
    eP2, _ = o.reorder(w2.g_idx)
    w1o = o.permute_rows(_d(w1), eP1)
    w2o = o.permute_rows(_d(w2), eP2)
    ref, _ = o.mlp_naive_algorithm(X, eP1, eP2, w1o, w2o, G, 1)
    assert o.rel_err(np_of(y2n), ref) <= TOL_FP16
    # Alg. 3's Y1 is Alg. 2's Y1 with its columns gathered by P2; Y2 is the same
    assert np.array_equal(np_of(y1n)[:, eP2].view(np.uint16), np_of(y1).view(np.uint16))
    assert np.array_equal(np_of(y2n).view(np.uint16), np_of(y2).view(np.uint16))


@pytest.mark.parametrize("M", [1, 16])
def test_alg2_local_llama_tp1(M):
    """The unsharded Llama-70B MLP (the paper's TP = 1 comparison): Alg. 2 and
    Alg. 3 agree bit for bit; Alg. 2 against the oracle on sampled columns."""
    import torch
    import paper_2402_04925_amd as tpdq
    from tests.gpu_util import workload_layers
    dev = torch_dev()
    wl = inputs.WORKLOADS["llama70b_tp1"]
    log(f"alg2 local llama70b_tp1 M={M}")
    w1, w2 = workload_layers(wl.name)
    X = inputs.make_x(wl, M)
    Xd = to_dev(X, dev)
    _, (y1, y2), (y1n, y2n) = _both(tpdq, Xd, layer_to_dev(w1, dev), layer_to_dev(w2, dev))
    torch.cuda.synchronize()
    eP2, _ = o.reorder(w2.g_idx)
    assert np.array_equal(np_of(y1n)[:, eP2].view(np.uint16), np_of(y1).view(np.uint16))
    assert np.array_equal(np_of(y2n).view(np.uint16), np_of(y2).view(np.uint16))
    cols = sample_cols(wl.N2, np.random.default_rng(M + 1))
    l1 = (w1.qweight, w1.scales, w1.qzeros, w1.g_idx)
    l2 = (w2.qweight, w2.scales, w2.qzeros, w2.g_idx)
    _, e2 = o.mlp_rank_from_global(X, l1, l2, 0, 1, True, P2=eP2, cols2=cols)
    assert o.rel_err(np_of(y2n)[:, cols], e2) <= TOL_FP16
