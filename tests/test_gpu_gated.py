"""GPU gated MLP shard (silu(X W_gate) * (X W_up), then W_down; Alg. 3 with
P2 folded into both gate and up, and the act-order rank) against the oracle."""
import numpy as np
import pytest

from oracle import tpdq_oracle as o
from paper_2402_04925_amd import inputs
from tests.gpu_util import (TOL_BF16, TOL_FP16, layer_to_dev, log, np_of, sample_cols, to_dev,
                            torch_dev)

pytestmark = pytest.mark.gpu


def _l(layer, g=None):
    return (layer.qweight, layer.scales, layer.qzeros, layer.g_idx if g is None else g)


def _custom(K1, N1, N2, G, seed, scale_dtype=np.float16):
    gate, down = inputs.make_custom(K1, N1, N2, G, seed, scale_dtype=scale_dtype)
    up, _ = inputs.make_custom(K1, N1, 0, G, seed + 1000, scale_dtype=scale_dtype)
    up.g_idx = gate.g_idx   # one input, one act-order permutation
    return gate, up, down


def _run(tpdq, Xd, dev, gate, up, down, rank, tp, variant):
    dg, du, dd = layer_to_dev(gate, dev), layer_to_dev(up, dev), layer_to_dev(down, dev)
    if variant.startswith("ordered"):
        lay = tpdq.LAYOUT_GPTQ if variant.endswith("gptq") else tpdq.LAYOUT_TILED
        P1, _, P2, _, gf, do = tpdq.reorder(dg, dd, layout=lay)
        P1u, _, _, _, uf, _ = tpdq.reorder(du, dd, layout=lay)
        assert bool((P1 == P1u).all())
        if tp == 1:   # the whole layers (a tiled shard must cover whole 16-column tiles)
            return tpdq.gated_mlp_shard(Xd, gf, uf, do, tpdq.PATH_ORDERED, P1=P1)
        return tpdq.gated_mlp_shard(Xd, gf.column_shard(rank, tp), uf.column_shard(rank, tp),
                                    do.row_shard(rank, tp, True), tpdq.PATH_ORDERED, P1=P1)
    if variant == "actorder-tiled":
        dg, du, dd = tpdq.pack_tiled(dg), tpdq.pack_tiled(du), tpdq.pack_tiled(dd)
    path = tpdq.PATH_ACTORDER_GLOBAL if variant == "actorder-global" else tpdq.PATH_ACTORDER
    if tp == 1:
        return tpdq.gated_mlp_shard(Xd, dg, du, dd, path)
    return tpdq.gated_mlp_shard(Xd, dg.column_shard(rank, tp), du.column_shard(rank, tp),
                                dd.row_shard(rank, tp, False), path)


VARIANTS = ["ordered", "ordered-gptq", "actorder", "actorder-global", "actorder-tiled"]


@pytest.mark.parametrize("M", [1, 5, 16, 70])
@pytest.mark.parametrize("tp", [1, 2])
@pytest.mark.parametrize("variant", VARIANTS)
def test_gated_small(M, tp, variant):
    """Every rank's Y1 and Y2 partial against the oracle, and the ranks' sum
    against the unsharded act-order gated MLP."""
    import torch
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    K1, N1, N2, G = 256, 512, 136, 32
    log(f"gated small {variant} tp={tp} M={M}")
    gate, up, down = _custom(K1, N1, N2, G, 50 + tp)
    X = inputs.random_activations(M, K1, np.random.default_rng(M + 50))
    Xd = to_dev(X, dev)
    eP2, _ = o.reorder(down.g_idx)
    ordered = variant.startswith("ordered")
    parts = []
    for r in range(tp):
        y1, y2 = _run(tpdq, Xd, dev, gate, up, down, r, tp, variant)
        torch.cuda.synchronize()
        e1, e2 = o.gated_rank_from_global(X, _l(gate), _l(up, gate.g_idx), _l(down), r, tp, ordered,
                                          P2=eP2)
        assert o.rel_err(np_of(y1), e1) <= TOL_FP16, r
        assert o.rel_err(np_of(y2), e2) <= TOL_FP16, r
        parts.append(np_of(y2))
    d = lambda w: dict(qweight=w.qweight, scales=w.scales, qzeros=w.qzeros)
    ref = o.gated_mlp_reference(X, d(gate), d(up), gate.g_idx, d(down), down.g_idx)
    assert o.rel_err(o.all_reduce_sum(parts), ref) <= 2 * TOL_FP16


def test_gated_zero_up():
    """q == z in W_up: Y1 and Y2 are exactly 0 whatever the gate (fp16)."""
    import torch
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    gate, up, down = _custom(256, 512, 136, 32, 7)
    z = o.unpack_cols(up.qzeros)
    up.qweight = o.pack_rows(z[up.g_idx])
    X = to_dev(inputs.random_activations(16, 256, np.random.default_rng(7)), dev)
    for variant in ("ordered", "actorder"):
        y1, y2 = _run(tpdq, X, dev, gate, up, down, 0, 1, variant)
        torch.cuda.synchronize()
        assert np.all(np_of(y1) == 0) and np.all(np_of(y2) == 0), variant


@pytest.mark.parametrize("name,M,dtype", [("llama70b_tp8", 1, "fp16"), ("llama70b_tp8", 4, "fp16"),
                                          ("llama70b_tp8", 16, "fp16"), ("granite20b_tp4", 8, "fp16"),
                                          ("llama70b_tp8", 16, "bf16")])
def test_gated_full_size(name, M, dtype):
    """Rank 0 of the gated Llama-70B TP = 8 and Granite-20B TP = 4 shards, both
    paths: Y1 on sampled columns, Y2_partial on sampled columns."""
    import torch
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    w = inputs.WORKLOADS[name]
    log(f"gated full {name} M={M} {dtype}")
    bf = dtype == "bf16"
    gate, up, down = inputs.make_gated_workload(w, scale_dtype=inputs.BF16 if bf else np.float16)
    X = inputs.make_x(w, M, dtype=inputs.BF16 if bf else np.float16)
    Xd = to_dev(X, dev, bf16=bf)
    eP2, _ = o.reorder(down.g_idx)
    tol = TOL_BF16 if bf else TOL_FP16
    n1 = w.N1 // w.tp
    c1 = sample_cols(n1, np.random.default_rng(M))
    c2 = sample_cols(w.N2, np.random.default_rng(M + 1))
    for variant in ("ordered", "actorder"):
        y1, y2 = _run(tpdq, Xd, dev, gate, up, down, 0, w.tp, variant)
        torch.cuda.synchronize()
        ordered = variant == "ordered"
        sel = eP2[:n1] if ordered else np.arange(n1)
        e1 = o.gated_y1(X, _l(gate)[:3], _l(up)[:3], gate.g_idx, cols=sel[c1], dtype=dtype)
        assert o.rel_err(np_of(y1)[:, c1], e1) <= tol, variant
        # Y2 from the GPU's own Y1 (the oracle's GEMM2 on the same input)
        W2 = o.dequant(*_l(down), cols=c2)[sel]
        e2 = o.round_to(o.matmul(np_of(y1).astype(np.float64), W2), dtype)
        assert o.rel_err(np_of(y2)[:, c2], e2) <= tol, variant


@pytest.mark.parametrize("M", [3, 17])
@pytest.mark.parametrize("variant", ["ordered", "actorder"])
def test_gated_ragged(M, variant):
    """Ragged K and N (not multiples of 128 or 16) and G = 8: the ordered path
    takes the per-row gated kernel with groups floor(k / G)."""
    import torch
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    K1, N1, N2, G = 288, 200, 72, 8
    log(f"gated ragged {variant} M={M}")
    gate, up, down = _custom(K1, N1, N2, G, 60 + M)
    X = inputs.random_activations(M, K1, np.random.default_rng(M + 60))
    y1, y2 = _run(tpdq, to_dev(X, dev), dev, gate, up, down, 0, 1, variant)
    torch.cuda.synchronize()
    eP2, _ = o.reorder(down.g_idx)
    e1, e2 = o.gated_rank_from_global(X, _l(gate), _l(up, gate.g_idx), _l(down), 0, 1,
                                      variant == "ordered", P2=eP2)
    assert o.rel_err(np_of(y1), e1) <= TOL_FP16
    assert o.rel_err(np_of(y2), e2) <= TOL_FP16


def test_gated_deterministic():
    """Two calls give bit-identical outputs."""
    import torch
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    gate, up, down = _custom(1024, 512, 256, 128, 3)
    X = to_dev(inputs.random_activations(16, 1024, np.random.default_rng(3)), dev)
    a = [np_of(t) for t in _run(tpdq, X, dev, gate, up, down, 0, 1, "ordered")]
    b = [np_of(t) for t in _run(tpdq, X, dev, gate, up, down, 0, 1, "ordered")]
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert np.array_equal(x.view(np.uint16), y.view(np.uint16))
