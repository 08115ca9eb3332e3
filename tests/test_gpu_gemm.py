"""GPU W4A16 GEMM (act-order and ordered paths) against the oracle."""
import numpy as np
import pytest

from oracle import tpdq_oracle as o
from paper_2402_04925_amd import inputs
from tests.gpu_util import (TOL_FP16, layer_to_dev, log, np_of, sample_cols, to_dev, torch_dev,
                            workload_layers)

pytestmark = pytest.mark.gpu

SHAPES = [  # K, N, G: config-0 size, ragged N and K, several tiles, small G (row-metadata kernel),
    # groups of 256 rows that span two 128-row blocks, split between waves
    (256, 128, 32), (288, 200, 32), (1024, 520, 128), (128, 72, 8), (192, 64, 64), (40, 24, 8),
    (2048, 1032, 128), (768, 48, 256), (2304, 96, 256),
]
MS = [1, 4, 16, 17, 64, 65]


def _d(layer):
    return dict(qweight=layer.qweight, scales=layer.scales, qzeros=layer.qzeros)


@pytest.mark.parametrize("K,N,G", SHAPES)
@pytest.mark.parametrize("M", MS)
@pytest.mark.parametrize("variant", ["lds", "global", "lds-tiled"])
def test_gemm_actorder(K, N, G, M, variant):
    import torch
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    path = tpdq.PATH_ACTORDER_GLOBAL if variant == "global" else tpdq.PATH_ACTORDER
    log(f"gemm actorder-{variant} K={K} N={N} G={G} M={M}")
    w1, _ = inputs.make_custom(K, N, 0, G, seed=K + N + G)
    X = inputs.random_activations(M, K, np.random.default_rng(M))
    dw = layer_to_dev(w1, dev)
    if variant == "lds-tiled":
        dw = tpdq.pack_tiled(dw)
    Y = tpdq.w4a16_gemm(to_dev(X, dev), dw, path)
    torch.cuda.synchronize()
    ref = o.w4a16_gemm(X, w1.qweight, w1.scales, w1.qzeros, w1.g_idx)
    assert o.rel_err(np_of(Y), ref) <= TOL_FP16


@pytest.mark.parametrize("K,N,G,M", [(K, N, G, M) for (K, N, G) in SHAPES for M in (2, 3)] +
                         [(8192, 256, 128, M) for M in (2, 3, 4)] + [(6144, 4352, 128, 2)])
@pytest.mark.parametrize("layout", ["tiled", "gptq"])
def test_gemm_ordered_gather_rows(K, N, G, M, layout):
    """The X[:, P] gather from the column-major LDS copy of X (2 <= M <= 4):
    ragged shapes, the Llama-70B K with one and two octets per thread, and
    4 waves with three octets per thread (over 256 column tiles)."""
    import torch
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    log(f"gemm ordered gather K={K} N={N} G={G} M={M} {layout}")
    w1, _ = inputs.make_custom(K, N, 0, G, seed=K + N + G + M)
    X = inputs.random_activations(M, K, np.random.default_rng(M + 7))
    lay = tpdq.LAYOUT_TILED if layout == "tiled" else tpdq.LAYOUT_GPTQ
    P, _, _, _, wo, _ = tpdq.reorder(layer_to_dev(w1, dev), layout=lay)
    Y = tpdq.w4a16_gemm(to_dev(X, dev), wo, tpdq.PATH_ORDERED, x_perm=P)
    torch.cuda.synchronize()
    ref = o.w4a16_gemm(X, w1.qweight, w1.scales, w1.qzeros, w1.g_idx)
    assert o.rel_err(np_of(Y), ref) <= TOL_FP16


@pytest.mark.parametrize("K,N,G", SHAPES)
@pytest.mark.parametrize("M", MS)
@pytest.mark.parametrize("layout", ["tiled", "gptq"])
def test_gemm_ordered(K, N, G, M, layout):
    """Sorted rows from the GPU reorder, the activation gather X[:, P] in the
    call; equal to the act-order product by the reorder invariant."""
    import torch
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    log(f"gemm ordered K={K} N={N} G={G} M={M} {layout}")
    w1, _ = inputs.make_custom(K, N, 0, G, seed=K + N + G)
    X = inputs.random_activations(M, K, np.random.default_rng(M))
    lay = tpdq.LAYOUT_TILED if layout == "tiled" else tpdq.LAYOUT_GPTQ
    P, gs, _, _, wo, _ = tpdq.reorder(layer_to_dev(w1, dev), layout=lay)
    Xd = to_dev(X, dev)
    Y = tpdq.w4a16_gemm(Xd, wo, tpdq.PATH_ORDERED, x_perm=P)
    torch.cuda.synchronize()
    ref = o.w4a16_gemm(X, w1.qweight, w1.scales, w1.qzeros, w1.g_idx)
    assert o.rel_err(np_of(Y), ref) <= TOL_FP16
    # without the gather: X multiplies the sorted rows directly
    Y2 = tpdq.w4a16_gemm(Xd, wo, tpdq.PATH_ORDERED)
    torch.cuda.synchronize()
    eP, eg = o.reorder(w1.g_idx)
    ws = o.permute_rows(_d(w1), eP)
    ref2 = o.w4a16_gemm(X, ws["qweight"], ws["scales"], ws["qzeros"], eg)
    assert o.rel_err(np_of(Y2), ref2) <= TOL_FP16


def test_gemm_deterministic():
    import torch
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    w1, _ = inputs.make_custom(4096, 1024, 0, 128, seed=3)
    X = to_dev(inputs.random_activations(16, 4096, np.random.default_rng(3)), dev)
    dw = layer_to_dev(w1, dev)
    P, _, _, _, wo, _ = tpdq.reorder(dw)
    for path, w, perm in ((tpdq.PATH_ACTORDER, dw, None), (tpdq.PATH_ORDERED, wo, P)):
        a = tpdq.w4a16_gemm(X, w, path, x_perm=perm).clone()
        b = tpdq.w4a16_gemm(X, w, path, x_perm=perm).clone()
        torch.cuda.synchronize()
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))


def test_gemm_zero_codes_special_case():
    """q == z everywhere -> Y == 0 exactly; G = K (one group)."""
    import torch
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    K, N = 256, 64
    z = np.random.default_rng(1).integers(0, 16, size=(1, N))
    qz = o.pack_cols(z)
    qw = o.pack_rows(np.repeat(z, K, axis=0))
    s = inputs.random_scales((1, N), np.random.default_rng(2))
    g = np.zeros(K, dtype=np.int32)
    w = tpdq.QuantWeight.from_tensors(to_dev(qw, dev), to_dev(s, dev), to_dev(qz, dev), to_dev(g, dev), K)
    X = to_dev(inputs.random_activations(4, K, np.random.default_rng(3)), dev)
    for path in (tpdq.PATH_ACTORDER, tpdq.PATH_ORDERED):
        Y = tpdq.w4a16_gemm(X, w, path)
        torch.cuda.synchronize()
        assert np.all(np_of(Y) == 0)


def test_gemm_clamps_out_of_range_gidx():
    """Act-order g_idx values outside [0, num_groups) are clamped in the kernel
    (no fault); the result equals the oracle with the clamped g_idx."""
    import torch
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    w1, _ = inputs.make_custom(256, 64, 0, 32, seed=5)
    g = w1.g_idx.copy()
    g[3], g[100] = 1000, -7
    w1.g_idx = g
    X = inputs.random_activations(4, 256, np.random.default_rng(5))
    Y = tpdq.w4a16_gemm(to_dev(X, dev), layer_to_dev(w1, dev), tpdq.PATH_ACTORDER)
    torch.cuda.synchronize()
    gc = np.where(g < 0, 7, g).clip(0, 7)
    ref = o.w4a16_gemm(X, w1.qweight, w1.scales, w1.qzeros, gc)
    assert o.rel_err(np_of(Y), ref) <= TOL_FP16


@pytest.mark.parametrize("name,which,M", [
    ("llama70b_tp8", 1, 1), ("llama70b_tp8", 1, 16), ("llama70b_tp8", 2, 4), ("llama70b_tp8", 2, 64),
    ("granite20b_tp4", 1, 8), ("granite20b_tp4", 2, 16), ("llama70b_tp1", 1, 16), ("llama70b_tp1", 2, 1),
])
def test_gemm_full_size_shards(name, which, M):
    """Rank 0's shard of the global layer at the paper's sizes (act-order:
    W2's row shard keeps global g_idx values and all metadata), both paths,
    on sampled output columns."""
    import torch
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    w = inputs.WORKLOADS[name]
    log(f"gemm full {name} W{which} M={M}")
    w1, w2 = workload_layers(name)
    L = w1 if which == 1 else w2
    K = L.K // (1 if which == 1 else w.tp)
    X = inputs.random_activations(M, K, np.random.default_rng(M))
    Xd = to_dev(X, dev)
    dl = layer_to_dev(L, dev)
    rng = np.random.default_rng(1)
    if which == 1:
        sh = dl.column_shard(0, w.tp)
        ncols = L.N // w.tp
        cols = sample_cols(ncols, rng)
        ref = o.w4a16_gemm(X, L.qweight, L.scales, L.qzeros, L.g_idx, cols=cols)
    else:
        sh = dl.row_shard(0, w.tp, sorted_rows=False)
        cols = sample_cols(L.N, rng)
        ref = o.w4a16_gemm(X, L.qweight[:K // 8], L.scales, L.qzeros, L.g_idx[:K], cols=cols)
    Y = tpdq.w4a16_gemm(Xd, sh, tpdq.PATH_ACTORDER)
    torch.cuda.synchronize()
    assert o.rel_err(np_of(Y)[:, cols], ref) <= TOL_FP16
    # act-order on the tiled storage order
    dlt = tpdq.pack_tiled(dl)
    sht = dlt.column_shard(0, w.tp) if which == 1 else dlt.row_shard(0, w.tp, sorted_rows=False)
    Yt = tpdq.w4a16_gemm(Xd, sht, tpdq.PATH_ACTORDER)
    torch.cuda.synchronize()
    assert o.rel_err(np_of(Yt)[:, cols], ref) <= TOL_FP16
    # ordered: the reordered global layer, same shard position
    P, gs, _, _, wo, _ = tpdq.reorder(dl)
    eP, eg = o.reorder(L.g_idx)
    if which == 1:
        sho = wo.column_shard(0, w.tp)
        Yo = tpdq.w4a16_gemm(Xd, sho, tpdq.PATH_ORDERED, x_perm=P)
        refo = ref   # X[:, P] @ W[P] has the same terms as X @ W
    else:
        sho = wo.row_shard(0, w.tp, sorted_rows=True)
        Yo = tpdq.w4a16_gemm(Xd, sho, tpdq.PATH_ORDERED)
        Wd = o.dequant(L.qweight, L.scales, L.qzeros, L.g_idx, cols=cols)[eP[:K]]
        refo = o.to_fp16(o.matmul(X, Wd))
    torch.cuda.synchronize()
    assert o.rel_err(np_of(Yo)[:, cols], refo) <= TOL_FP16


def test_gemm_interleaved_shapes_share_workspace():
    """Calls of different shapes and paths, one after another on one stream and
    one workspace, each equal to its own oracle result."""
    import torch
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    ws = tpdq.Workspace(dev)
    cases = [(256, 64, 32, 3), (2048, 3584, 128, 16), (512, 1032, 64, 1), (2048, 512, 128, 40)]
    outs = []
    for K, N, G, M in cases * 2:
        w1, _ = inputs.make_custom(K, N, 0, G, seed=K + N)
        X = inputs.random_activations(M, K, np.random.default_rng(K))
        dw = layer_to_dev(w1, dev)
        P, _, _, _, wo, _ = tpdq.reorder(dw, workspace=ws)
        Yo = tpdq.w4a16_gemm(to_dev(X, dev), wo, tpdq.PATH_ORDERED, x_perm=P, workspace=ws)
        Ya = tpdq.w4a16_gemm(to_dev(X, dev), dw, tpdq.PATH_ACTORDER, workspace=ws)
        outs.append((X, w1, Yo, Ya))
    torch.cuda.synchronize()
    for X, w1, Yo, Ya in outs:
        ref = o.w4a16_gemm(X, w1.qweight, w1.scales, w1.qzeros, w1.g_idx)
        assert o.rel_err(np_of(Yo), ref) <= TOL_FP16
        assert o.rel_err(np_of(Ya), ref) <= TOL_FP16


# degenerate shapes: one group (G = K), the smallest N (half a 16-column
# tile), the smallest K (one 8-row word), a single row
DEGENERATE = [(256, 64, 256, 5), (128, 8, 128, 1), (8, 8, 8, 1), (8, 24, 8, 3), (512, 8, 32, 16)]


@pytest.mark.parametrize("K,N,G,M", DEGENERATE)
def test_gemm_degenerate(K, N, G, M):
    """Every path and layout on degenerate shapes, against the oracle."""
    import torch
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    log(f"gemm degenerate K={K} N={N} G={G} M={M}")
    w1, _ = inputs.make_custom(K, N, 0, G, seed=K * 7 + N + G)
    X = inputs.random_activations(M, K, np.random.default_rng(K + M))
    Xd = to_dev(X, dev)
    dw = layer_to_dev(w1, dev)
    ref = o.w4a16_gemm(X, w1.qweight, w1.scales, w1.qzeros, w1.g_idx)
    for path in (tpdq.PATH_ACTORDER, tpdq.PATH_ACTORDER_GLOBAL):
        for w in (dw, tpdq.pack_tiled(dw)):
            Y = tpdq.w4a16_gemm(Xd, w, path)
            torch.cuda.synchronize()
            assert o.rel_err(np_of(Y), ref) <= TOL_FP16, path
    for lay in (tpdq.LAYOUT_TILED, tpdq.LAYOUT_GPTQ):
        P, _, _, _, wo, _ = tpdq.reorder(dw, layout=lay)
        Y = tpdq.w4a16_gemm(Xd, wo, tpdq.PATH_ORDERED, x_perm=P)
        torch.cuda.synchronize()
        assert o.rel_err(np_of(Y), ref) <= TOL_FP16, lay
