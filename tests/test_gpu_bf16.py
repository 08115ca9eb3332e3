"""bf16 activations, scales and outputs on every GEMM kernel family and the
MLP shard, against the oracle's bf16 results (one rounding of the float64
product)."""
import numpy as np
import pytest

from oracle import tpdq_oracle as o
from paper_2402_04925_amd import inputs
from tests.gpu_util import TOL_BF16, layer_to_dev, log, np_of, sample_cols, to_dev, torch_dev

pytestmark = pytest.mark.gpu

BF = inputs.BF16

# K, N, G: ragged N and K, small G (per-row metadata for the ordered path),
# groups of 256 rows spanning two 128-row blocks
SHAPES = [(256, 128, 32), (288, 200, 32), (1024, 520, 128), (128, 72, 8), (768, 48, 256),
          (2304, 96, 256)]
MS = [1, 5, 16, 33, 64, 65]


def _layer(K, N, G, seed):
    w1, _ = inputs.make_custom(K, N, 0, G, seed=seed, scale_dtype=BF)
    return w1


def _sorted_ref(w1, X, cols=None):
    eP, eg = o.reorder(w1.g_idx)
    ws = o.permute_rows(dict(qweight=w1.qweight, scales=w1.scales, qzeros=w1.qzeros), eP)
    return o.w4a16_gemm(X, ws["qweight"], ws["scales"], ws["qzeros"], eg, cols=cols, dtype="bf16")


@pytest.mark.parametrize("K,N,G", SHAPES)
@pytest.mark.parametrize("M", MS)
@pytest.mark.parametrize("variant", ["ordered-tiled", "ordered-gptq", "actorder", "actorder-global",
                                     "actorder-tiled"])
def test_bf16_gemm(K, N, G, M, variant):
    import torch
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    log(f"bf16 gemm {variant} K={K} N={N} G={G} M={M}")
    w1 = _layer(K, N, G, K + N + G + 1)
    X = inputs.random_activations(M, K, np.random.default_rng(M + 3), dtype=BF)
    Xd = to_dev(X, dev, bf16=True)
    dw = layer_to_dev(w1, dev)
    ref = o.w4a16_gemm(X, w1.qweight, w1.scales, w1.qzeros, w1.g_idx, dtype="bf16")
    if variant.startswith("ordered"):
        lay = tpdq.LAYOUT_TILED if variant.endswith("tiled") else tpdq.LAYOUT_GPTQ
        P, _, _, _, wo, _ = tpdq.reorder(dw, layout=lay)
        Y = tpdq.w4a16_gemm(Xd, wo, tpdq.PATH_ORDERED, x_perm=P)
        torch.cuda.synchronize()
        assert Y.dtype == torch.bfloat16
        assert o.rel_err(np_of(Y), ref) <= TOL_BF16
        Y2 = tpdq.w4a16_gemm(Xd, wo, tpdq.PATH_ORDERED)
        torch.cuda.synchronize()
        assert o.rel_err(np_of(Y2), _sorted_ref(w1, X)) <= TOL_BF16
    else:
        path = tpdq.PATH_ACTORDER_GLOBAL if variant == "actorder-global" else tpdq.PATH_ACTORDER
        if variant == "actorder-tiled":
            dw = tpdq.pack_tiled(dw)
        Y = tpdq.w4a16_gemm(Xd, dw, path)
        torch.cuda.synchronize()
        assert Y.dtype == torch.bfloat16
        assert o.rel_err(np_of(Y), ref) <= TOL_BF16


def test_bf16_exact_weights_ordered():
    """The ordered decode kernel keeps q - z exact (128 + q against the group
    sum of X) and scales in fp32, so its only rounding is the output's: within
    2^-8 of each output's magnitude plus the fp32 accumulation."""
    import torch
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    K, N, G, M = 2048, 520, 128, 16
    w1 = _layer(K, N, G, 5)
    X = inputs.random_activations(M, K, np.random.default_rng(6), dtype=BF)
    P, _, _, _, wo, _ = tpdq.reorder(layer_to_dev(w1, dev), layout=tpdq.LAYOUT_TILED)
    Y = np_of(tpdq.w4a16_gemm(to_dev(X, dev, bf16=True), wo, tpdq.PATH_ORDERED, x_perm=P))
    torch.cuda.synchronize()
    Y64 = o.w4a16_gemm(X, w1.qweight, w1.scales, w1.qzeros, w1.g_idx, round_fp16=False)
    err = np.abs(Y.astype(np.float64) - Y64)
    assert np.all(err <= np.exp2(-8) * np.abs(Y64) + 1e-5 * np.max(np.abs(Y64)))


def test_bf16_zero_codes():
    """q == z everywhere: the exact product is 0. The ordered bf16 kernels
    form it as sum x (128 + z) - (128 + z) sum x from two fp32 MFMA
    accumulations, so what is left is their rounding: far below 2^-16 of the
    largest group term 143 s sum |x| (fp32 keeps 24 bits)."""
    import torch
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    K, N, M = 512, 256, 16
    z = np.random.default_rng(1).integers(0, 16, size=(K // 128, N))
    qz = o.pack_cols(z)
    qw = o.pack_rows(np.repeat(z, 128, axis=0))
    s = inputs.random_scales((K // 128, N), np.random.default_rng(2), dtype=BF)
    X = to_dev(inputs.random_activations(M, K, np.random.default_rng(3), dtype=BF), dev, bf16=True)
    w = tpdq.QuantWeight.from_tensors(to_dev(qw, dev), to_dev(s, dev, bf16=True), to_dev(qz, dev),
                                      None, 128)
    Xh = inputs.random_activations(M, K, np.random.default_rng(3), dtype=BF)
    bound = np.exp2(-16) * 143.0 * float(np.max(s)) * float(np.max(np.sum(np.abs(Xh), axis=1)))
    for dw in (w, tpdq.pack_tiled(w)):
        Y = tpdq.w4a16_gemm(X, dw, tpdq.PATH_ORDERED)
        torch.cuda.synchronize()
        assert np.max(np.abs(np_of(Y))) <= bound


# K, N, G, M: the M-tiled kernel (prefill tiles; split-K tiles on large weights)
# and the wide decode kernel (large weights, X too large for LDS)
LARGE = [("prefill", 1024, 1032, 128, 257), ("prefill", 2048, 512, 256, 512),
         ("mtile", 8192, 8200, 128, 40), ("wide", 8192, 8200, 64, 16), ("wide", 4096, 16384, 32, 17)]


@pytest.mark.parametrize("kind,K,N,G,M", LARGE)
def test_bf16_large(kind, K, N, G, M):
    """Sorted rows, tiled weights, with the gather and without, on sampled
    columns (tile edges, the ragged tail, random ones)."""
    import torch
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    log(f"bf16 {kind} K={K} N={N} G={G} M={M}")
    w1 = _layer(K, N, G, K + N + M)
    X = inputs.random_activations(M, K, np.random.default_rng(M + 9), dtype=BF)
    Xd = to_dev(X, dev, bf16=True)
    P, _, _, _, wo, _ = tpdq.reorder(layer_to_dev(w1, dev), layout=tpdq.LAYOUT_TILED)
    cols = sample_cols(N, np.random.default_rng(K + M)) if K * N >= (1 << 26) else np.arange(N)
    ref = o.w4a16_gemm(X, w1.qweight, w1.scales, w1.qzeros, w1.g_idx, cols=cols, dtype="bf16")
    for _ in range(2):
        Y = tpdq.w4a16_gemm(Xd, wo, tpdq.PATH_ORDERED, x_perm=P)
        torch.cuda.synchronize()
        assert o.rel_err(np_of(Y)[:, cols], ref) <= TOL_BF16
    Y2 = tpdq.w4a16_gemm(Xd, wo, tpdq.PATH_ORDERED)
    torch.cuda.synchronize()
    assert o.rel_err(np_of(Y2)[:, cols], _sorted_ref(w1, X, cols)) <= TOL_BF16


def _l(layer):
    return (layer.qweight, layer.scales, layer.qzeros, layer.g_idx)


@pytest.mark.parametrize("name,M", [("llama70b_tp8", 1), ("llama70b_tp8", 16), ("granite20b_tp4", 8)])
def test_bf16_mlp_full_size(name, M):
    """Rank 0 of the paper's MLP problem sizes with bf16 activations and
    scales, ordered (Alg. 3) and act-order: Y1 in full, Y2_partial on sampled
    columns."""
    import torch
    import paper_2402_04925_amd as tpdq
    dev = torch_dev()
    w = inputs.WORKLOADS[name]
    log(f"bf16 mlp {name} M={M}")
    w1, w2 = inputs.make_workload(w, scale_dtype=BF)
    X = inputs.make_x(w, M, dtype=BF)
    d1, d2 = layer_to_dev(w1, dev), layer_to_dev(w2, dev)
    P1, _, P2, _, w1o, w2o = tpdq.reorder(d1, d2)
    eP2, _ = o.reorder(w2.g_idx)
    cols = sample_cols(w.N2, np.random.default_rng(M))
    Xd = to_dev(X, dev, bf16=True)
    for ordered in (False, True):
        if ordered:
            y1, y2 = tpdq.mlp_shard(Xd, w1o.column_shard(0, w.tp), w2o.row_shard(0, w.tp, True),
                                    tpdq.PATH_ORDERED, P1=P1)
        else:
            y1, y2 = tpdq.mlp_shard(Xd, d1.column_shard(0, w.tp), d2.row_shard(0, w.tp, False),
                                    tpdq.PATH_ACTORDER)
        torch.cuda.synchronize()
        e1, e2 = o.mlp_rank_from_global(X, _l(w1), _l(w2), 0, w.tp, ordered, P2=eP2, cols2=cols,
                                        dtype="bf16")
        assert o.rel_err(np_of(y1), e1) <= TOL_BF16, ordered
        assert o.rel_err(np_of(y2)[:, cols], e2) <= TOL_BF16, ordered
