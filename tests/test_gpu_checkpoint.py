"""GPTQ checkpoint conventions on the GPU against the oracle: the zero-point
offset (packers that store z - 1), a partial last group (G not dividing K,
Eq. 3's groups), and groups of unequal sizes (G = 0, the grouping given by
g_idx alone). Both paths (act-order through g_idx; ordered after the
reorder), both weight layouts, the decode, wide and M-tiled kernels, the
reorder itself (bit-exact), and the MLP shard."""
import numpy as np
import pytest

from oracle import tpdq_oracle as o
from paper_2402_04925_amd import inputs
from tests.gpu_util import TOL_BF16, TOL_FP16, layer_to_dev, log, np_of, sample_cols, to_dev, torch_dev

pytestmark = pytest.mark.gpu


def _gl(L, zo=0):
    return (L.qweight, L.scales, L.qzeros, L.g_idx, zo)


def _run_paths(tpdq, X, Xd, L, d, zo, cols=None, tol=TOL_FP16):
    """Every path on layer L (device d): act-order on GPTQ and tiled words,
    Fig. 1's global-metadata variant, and ordered after the GPU reorder (with
    and without the X[:, P] gather); each against the oracle."""
    import torch
    ref = o.w4a16_gemm(X, L.qweight, L.scales, L.qzeros, L.g_idx, cols=cols, zero_offset=zo)
    d.zero_offset = zo
    t = tpdq.pack_tiled(d)
    for name, w, path in (("actorder", d, tpdq.PATH_ACTORDER), ("actorder_tiled", t, tpdq.PATH_ACTORDER),
                          ("actorder_global", d, tpdq.PATH_ACTORDER_GLOBAL)):
        Y = tpdq.w4a16_gemm(Xd, w, path)
        torch.cuda.synchronize()
        y = np_of(Y) if cols is None else np_of(Y)[:, cols]
        assert o.rel_err(y, ref) <= tol, name
    for layout in (tpdq.LAYOUT_TILED, tpdq.LAYOUT_GPTQ):
        P, gs, _, _, wo, _ = tpdq.reorder(d, layout=layout)
        assert wo.zero_offset == zo
        Y = tpdq.w4a16_gemm(Xd, wo, tpdq.PATH_ORDERED, x_perm=P)
        torch.cuda.synchronize()
        y = np_of(Y) if cols is None else np_of(Y)[:, cols]
        assert o.rel_err(y, ref) <= tol, ("ordered", layout)
    eP, eg = o.reorder(L.g_idx)
    assert np.array_equal(np_of(P), eP) and np.array_equal(np_of(gs), eg)


# ------------------------------------------------------------ zero offset ---

@pytest.mark.parametrize("K,N,G,M", [(256, 128, 32, 1), (1024, 256, 128, 5), (1024, 520, 64, 16),
                                     (512, 256, 256, 64), (1024, 512, 128, 300)])
def test_zero_offset_gemm(K, N, G, M):
    """Stored zeros z' read as z' + 1 (z = 16 reachable) on every path and
    kernel: the decode kernels (M <= 64, X in LDS or from global memory) and
    the M-tiled kernel (M = 300)."""
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    log(f"zero offset K={K} N={N} G={G} M={M}")
    L, _ = inputs.make_custom(K, N, 0, G, seed=K + N + M)
    X = inputs.random_activations(M, K, np.random.default_rng(M))
    _run_paths(tpdq, X, to_dev(X, dev), L, layer_to_dev(L, dev), 1)


def test_zero_offset_bf16():
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    K, N, G, M = 1024, 256, 128, 16
    L, _ = inputs.make_custom(K, N, 0, G, seed=9, scale_dtype=inputs.BF16)
    X = inputs.random_activations(M, K, np.random.default_rng(9), dtype=inputs.BF16)
    _run_paths(tpdq, X, to_dev(X, dev, bf16=True), L, layer_to_dev(L, dev), 1, tol=TOL_BF16)


@pytest.mark.parametrize("M", [16, 40])
def test_zero_offset_large(M):
    """64M weights with row-major X and the offset: the wide kernel (M = 16)
    and the M-tiled kernel with K split (M = 40)."""
    import paper_2402_04925_amd as tpdq
    import torch
    dev = torch_dev()
    K, N, G = 8192, 8192, 128
    L, _ = inputs.make_custom(K, N, 0, G, seed=21)
    X = inputs.random_activations(M, K, np.random.default_rng(21))
    d = layer_to_dev(L, dev)
    d.zero_offset = 1
    _, _, _, _, wo, _ = tpdq.reorder(d)
    eP, eg = o.reorder(L.g_idx)
    cols = sample_cols(N, np.random.default_rng(3))
    ws = o.permute_rows(dict(qweight=L.qweight, scales=L.scales, qzeros=L.qzeros), eP)
    ref = o.w4a16_gemm(X, ws["qweight"], ws["scales"], ws["qzeros"], eg, cols=cols, zero_offset=1)
    Y = tpdq.w4a16_gemm(to_dev(X, dev), wo, tpdq.PATH_ORDERED)
    torch.cuda.synchronize()
    assert o.rel_err(np_of(Y)[:, cols], ref) <= TOL_FP16


@pytest.mark.parametrize("ordered", [True, False])
@pytest.mark.parametrize("M", [2, 16])
def test_zero_offset_mlp(ordered, M):
    import paper_2402_04925_amd as tpdq
    import torch
    dev = torch_dev()
    K1, N1, N2, G, tp = 1024, 512, 256, 128, 2
    w1, w2 = inputs.make_custom(K1, N1, N2, G, seed=33 + M)
    X = inputs.random_activations(M, K1, np.random.default_rng(M))
    d1, d2 = layer_to_dev(w1, dev), layer_to_dev(w2, dev)
    d1.zero_offset = d2.zero_offset = 1
    if ordered:
        P1, _, _, _, w1o, w2o = tpdq.reorder(d1, d2)
        y1, y2 = tpdq.mlp_shard(to_dev(X, dev), w1o.column_shard(0, tp), w2o.row_shard(0, tp, True),
                                tpdq.PATH_ORDERED, P1=P1)
    else:
        y1, y2 = tpdq.mlp_shard(to_dev(X, dev), d1.column_shard(0, tp), d2.row_shard(0, tp, False),
                                tpdq.PATH_ACTORDER)
    torch.cuda.synchronize()
    eP2, _ = o.reorder(w2.g_idx)
    e1, e2 = o.mlp_rank_from_global(X, _gl(w1, 1), _gl(w2, 1), 0, tp, ordered, P2=eP2)
    assert o.rel_err(np_of(y1), e1) <= TOL_FP16 and o.rel_err(np_of(y2), e2) <= TOL_FP16


def test_zero_offset_gated():
    import paper_2402_04925_amd as tpdq
    import torch
    dev = torch_dev()
    K1, N1, N2, G, M = 512, 256, 128, 64, 5
    gate, down = inputs.make_custom(K1, N1, N2, G, seed=44)
    up, _ = inputs.make_custom(K1, N1, 0, G, seed=45)
    up.g_idx = gate.g_idx
    X = inputs.random_activations(M, K1, np.random.default_rng(4))
    dg, du, dd = layer_to_dev(gate, dev), layer_to_dev(up, dev), layer_to_dev(down, dev)
    for w in (dg, du, dd):
        w.zero_offset = 1
    P1, _, _, _, go, do = tpdq.reorder(dg, dd)
    _, _, _, _, uo, _ = tpdq.reorder(du, dd)
    y1, y2 = tpdq.gated_mlp_shard(to_dev(X, dev), go, uo, do, tpdq.PATH_ORDERED, P1=P1)
    torch.cuda.synchronize()
    eP2, _ = o.reorder(down.g_idx)
    sel = eP2
    yg = o.matmul(X, o.dequant(gate.qweight, gate.scales, gate.qzeros, gate.g_idx, cols=sel, zero_offset=1))
    yu = o.matmul(X, o.dequant(up.qweight, up.scales, up.qzeros, gate.g_idx, cols=sel, zero_offset=1))
    e1 = o.to_fp16(o.silu(yg) * yu)
    e2 = o.to_fp16(o.matmul(e1, o.dequant(down.qweight, down.scales, down.qzeros, down.g_idx,
                                          zero_offset=1)[sel]))
    assert o.rel_err(np_of(y1), e1) <= TOL_FP16 and o.rel_err(np_of(y2), e2) <= TOL_FP16


# ---------------------------------------------------- partial last group ---

@pytest.mark.parametrize("K,N,G,M", [(1088, 128, 128, 1), (1088, 256, 128, 16), (1152, 136, 256, 4),
                                     (1064, 128, 32, 5), (1000, 264, 64, 33), (1088, 512, 128, 300)])
def test_partial_group_gemm(K, N, G, M):
    """G not dividing K: ceil(K/G) groups, the last partial (K = 1088 with
    G = 128: 64 rows; K = 1152 with G = 256: 128 rows; K = 1064 with G = 32:
    8 rows, K % 32 != 0), every path, the reorder bit-exact."""
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    log(f"partial group K={K} N={N} G={G} M={M}")
    L, _ = inputs.make_custom(K, N, 0, G, seed=K + G + M)
    assert L.scales.shape[0] == -(-K // G)
    X = inputs.random_activations(M, K, np.random.default_rng(M + 2))
    _run_paths(tpdq, X, to_dev(X, dev), L, layer_to_dev(L, dev), 0)


@pytest.mark.parametrize("K,M", [(8256, 16), (8200, 40)])
def test_partial_group_wide(K, M):
    """64M weights (N = 8192) on K = 8256 (a partial group of 64 rows) and
    K = 8200 (8 rows; the last 32-row step partly outside K): the wide kernel
    (M = 16) and the M-tiled kernel with K split (M = 40), with the gathered
    and the row-major activations (their per-octet loads)."""
    import paper_2402_04925_amd as tpdq
    import torch
    dev = torch_dev()
    N, G = 8192, 128
    L, _ = inputs.make_custom(K, N, 0, G, seed=K)
    X = inputs.random_activations(M, K, np.random.default_rng(K))
    d = layer_to_dev(L, dev)
    P, _, _, _, wo, _ = tpdq.reorder(d)
    cols = sample_cols(N, np.random.default_rng(K + 1))
    ref = o.w4a16_gemm(X, L.qweight, L.scales, L.qzeros, L.g_idx, cols=cols)
    Xd = to_dev(X, dev)
    Y = tpdq.w4a16_gemm(Xd, wo, tpdq.PATH_ORDERED, x_perm=P)
    torch.cuda.synchronize()
    assert o.rel_err(np_of(Y)[:, cols], ref) <= TOL_FP16
    # row-major X straight into the sorted rows (no gather): X multiplies W[P]
    Xs = X[:, np.asarray(o.reorder(L.g_idx)[0])]
    Y2 = tpdq.w4a16_gemm(to_dev(np.ascontiguousarray(Xs), dev), wo, tpdq.PATH_ORDERED)
    torch.cuda.synchronize()
    assert o.rel_err(np_of(Y2)[:, cols], ref) <= TOL_FP16


def test_partial_group_reorder_rejects():
    """A g_idx whose last group is not Eq. 3's (here 9 rows instead of 8)
    is refused by the reorder's validation."""
    import paper_2402_04925_amd as tpdq
    import torch
    dev = torch_dev()
    L, _ = inputs.make_custom(72, 32, 0, 32, seed=3)
    g = L.g_idx.copy()
    g[np.flatnonzero(g == 1)[0]] = 2
    d = layer_to_dev(L, dev)
    d.g_idx = to_dev(g.astype(np.int32), dev)
    with pytest.raises(tpdq.TpdqError, match="Eq. 3"):
        tpdq.reorder(d)
    torch.cuda.synchronize()


@pytest.mark.parametrize("ordered", [True, False])
@pytest.mark.parametrize("M", [1, 16])
def test_partial_group_mlp(ordered, M):
    """W1 8 x 128 + 64 rows deep and W2 with a partial last group (K2 = N1 =
    1088); TP = 1 on the ordered path (a sorted row shard must start on a
    group boundary), TP = 2 on the act-order path."""
    import paper_2402_04925_amd as tpdq
    import torch
    dev = torch_dev()
    K1, N1, N2, G = 1088, 1088, 256, 128
    tp = 1 if ordered else 2
    w1, w2 = inputs.make_custom(K1, N1, N2, G, seed=55 + M)
    X = inputs.random_activations(M, K1, np.random.default_rng(M + 7))
    d1, d2 = layer_to_dev(w1, dev), layer_to_dev(w2, dev)
    if ordered:
        P1, _, _, _, w1o, w2o = tpdq.reorder(d1, d2)
        y1, y2 = tpdq.mlp_shard(to_dev(X, dev), w1o, w2o, tpdq.PATH_ORDERED, P1=P1)
    else:
        y1, y2 = tpdq.mlp_shard(to_dev(X, dev), d1.column_shard(1, tp), d2.row_shard(1, tp, False),
                                tpdq.PATH_ACTORDER)
    torch.cuda.synchronize()
    eP2, _ = o.reorder(w2.g_idx)
    e1, e2 = o.mlp_rank_from_global(X, _gl(w1), _gl(w2), 0 if ordered else 1, tp, ordered, P2=eP2)
    assert o.rel_err(np_of(y1), e1) <= TOL_FP16 and o.rel_err(np_of(y2), e2) <= TOL_FP16


# ------------------------------------------------- groups of unequal size ---

@pytest.mark.parametrize("K,N,ng,M", [(256, 128, 5, 4), (1024, 264, 13, 16), (2048, 512, 40, 64),
                                      (1024, 256, 9, 300)])
def test_unequal_groups_gemm(K, N, ng, M):
    """Groups of unequal sizes (G = 0): the reorder sorts them (P and the
    sorted g_idx bit-exact), the act-order paths read g_idx, the ordered path
    reads the sorted g_idx (per-row metadata on sorted rows)."""
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    log(f"unequal groups K={K} N={N} ng={ng} M={M}")
    L = inputs.make_unequal_layer(K, N, ng, seed=K + ng)
    X = inputs.random_activations(M, K, np.random.default_rng(M + 3))
    d = layer_to_dev(L, dev)
    assert d.G == 0 and d.num_groups == ng
    _run_paths(tpdq, X, to_dev(X, dev), L, d, 0)


@pytest.mark.parametrize("tp", [1, 2, 4])
@pytest.mark.parametrize("ordered", [True, False])
def test_unequal_groups_mlp(tp, ordered):
    """The MLP with groups of unequal sizes in both layers: every rank against
    the oracle and the rank sum against the unsharded MLP (W2's sorted row
    shards keep every group's metadata and their rows' sorted groups)."""
    import paper_2402_04925_amd as tpdq
    import torch
    dev = torch_dev()
    K1, N1, N2, M = 512, 512, 256, 5
    w1 = inputs.make_unequal_layer(K1, N1, 11, seed=70, layer=0)
    w2 = inputs.make_unequal_layer(N1, N2, 7, seed=70, layer=1)
    X = inputs.random_activations(M, K1, np.random.default_rng(70))
    d1, d2 = layer_to_dev(w1, dev), layer_to_dev(w2, dev)
    Xd = to_dev(X, dev)
    eP2, _ = o.reorder(w2.g_idx)
    if ordered:
        P1, _, _, _, w1o, w2o = tpdq.reorder(d1, d2)
    parts = []
    for r in range(tp):
        if ordered:
            y1, y2 = tpdq.mlp_shard(Xd, w1o.column_shard(r, tp), w2o.row_shard(r, tp, True),
                                    tpdq.PATH_ORDERED, P1=P1)
        else:
            y1, y2 = tpdq.mlp_shard(Xd, d1.column_shard(r, tp), d2.row_shard(r, tp, False),
                                    tpdq.PATH_ACTORDER)
        torch.cuda.synchronize()
        e1, e2 = o.mlp_rank_from_global(X, _gl(w1), _gl(w2), r, tp, ordered, P2=eP2)
        assert o.rel_err(np_of(y1), e1) <= TOL_FP16 and o.rel_err(np_of(y2), e2) <= TOL_FP16, r
        parts.append(np_of(y2))
    d1o = dict(qweight=w1.qweight, scales=w1.scales, qzeros=w1.qzeros)
    d2o = dict(qweight=w2.qweight, scales=w2.scales, qzeros=w2.qzeros)
    ref = o.mlp_reference(X, d1o, w1.g_idx, d2o, w2.g_idx)
    assert o.rel_err(o.all_reduce_sum(parts), ref) <= 2 * TOL_FP16
