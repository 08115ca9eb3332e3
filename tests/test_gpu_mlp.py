"""GPU MLP shard (Alg. 3 per rank, and the act-order rank) against the oracle."""
import numpy as np
import pytest

from oracle import tpdq_oracle as o
from paper_2402_04925_amd import inputs
from tests.gpu_util import (TOL_FP16, layer_to_dev, log, np_of, sample_cols, to_dev, torch_dev,
                            workload_layers)

pytestmark = pytest.mark.gpu


def _l(layer):
    return (layer.qweight, layer.scales, layer.qzeros, layer.g_idx)


def _run_rank(tpdq, X, d1, d2, P1, w1o, w2o, rank, tp, ordered, path=None):
    if ordered:
        return tpdq.mlp_shard(X, w1o.column_shard(rank, tp), w2o.row_shard(rank, tp, True),
                              tpdq.PATH_ORDERED, P1=P1)
    return tpdq.mlp_shard(X, d1.column_shard(rank, tp), d2.row_shard(rank, tp, False),
                          tpdq.PATH_ACTORDER if path is None else path)


@pytest.mark.parametrize("tp", [1, 2, 4])
@pytest.mark.parametrize("ordered", [False, True])
def test_mlp_small_all_ranks(tp, ordered):
    """Every rank's partial against the oracle, and their sum (the simulated
    AllReduce) against the unsharded MLP."""
    import torch
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    K1, N1, N2, G, M = 256, 512, 136, 32, 5
    log(f"mlp small tp={tp} ordered={ordered}")
    w1, w2 = inputs.make_custom(K1, N1, N2, G, seed=20 + tp)
    X = inputs.random_activations(M, K1, np.random.default_rng(tp))
    d1, d2 = layer_to_dev(w1, dev), layer_to_dev(w2, dev)
    P1, _, P2, _, w1o, w2o = tpdq.reorder(d1, d2)
    eP2, _ = o.reorder(w2.g_idx)
    Xd = to_dev(X, dev)
    parts = []
    for r in range(tp):
        y1, y2 = _run_rank(tpdq, Xd, d1, d2, P1, w1o, w2o, r, tp, ordered)
        torch.cuda.synchronize()
        e1, e2 = o.mlp_rank_from_global(X, _l(w1), _l(w2), r, tp, ordered, P2=eP2)
        assert o.rel_err(np_of(y1), e1) <= TOL_FP16, r
        assert o.rel_err(np_of(y2), e2) <= TOL_FP16, r
        parts.append(np_of(y2))
    tot = o.all_reduce_sum(parts)
    ref = o.mlp_reference(X, dict(qweight=w1.qweight, scales=w1.scales, qzeros=w1.qzeros), w1.g_idx,
                          dict(qweight=w2.qweight, scales=w2.scales, qzeros=w2.qzeros), w2.g_idx)
    assert o.rel_err(tot, ref) <= 2 * TOL_FP16


CASES = [("llama70b_tp8", M) for M in (1, 4, 16)] + [("granite20b_tp4", M) for M in (1, 8, 16)] + \
        [("llama70b_tp1", M) for M in (1, 16, 64)]


@pytest.mark.parametrize("name,M", CASES)
def test_mlp_full_size(name, M):
    """Rank 0 at the paper's MLP problem sizes, both paths: Y1 in full,
    Y2_partial on sampled columns."""
    import torch
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    w = inputs.WORKLOADS[name]
    log(f"mlp full {name} M={M}")
    w1, w2 = workload_layers(name)
    X = inputs.make_x(w, M)
    d1, d2 = layer_to_dev(w1, dev), layer_to_dev(w2, dev)
    P1, _, P2, _, w1o, w2o = tpdq.reorder(d1, d2)
    eP2, _ = o.reorder(w2.g_idx)
    cols = sample_cols(w.N2, np.random.default_rng(M))
    Xd = to_dev(X, dev)
    t1, t2 = tpdq.pack_tiled(d1), tpdq.pack_tiled(d2)
    e_act = o.mlp_rank_from_global(X, _l(w1), _l(w2), 0, w.tp, False, P2=eP2, cols2=cols)
    e_ord = o.mlp_rank_from_global(X, _l(w1), _l(w2), 0, w.tp, True, P2=eP2, cols2=cols)
    for name, ordered, a1, a2, path in (
            ("actorder", False, d1, d2, tpdq.PATH_ACTORDER),
            ("actorder-global", False, d1, d2, tpdq.PATH_ACTORDER_GLOBAL),
            ("actorder-tiled", False, t1, t2, tpdq.PATH_ACTORDER),
            ("ordered", True, d1, d2, None)):
        y1, y2 = _run_rank(tpdq, Xd, a1, a2, P1, w1o, w2o, 0, w.tp, ordered, path)
        torch.cuda.synchronize()
        e1, e2 = e_ord if ordered else e_act
        assert o.rel_err(np_of(y1), e1) <= TOL_FP16, name
        assert o.rel_err(np_of(y2)[:, cols], e2) <= TOL_FP16, name
