"""CPU oracle for TP-aware dequantization (arXiv 2402.04925).

TEST INFRASTRUCTURE ONLY. Nothing in the product path imports this module; only
the tests, the smoke check and the CPU-baseline leg of the benchmark do. It is a
plain, slow, obviously correct restatement of what the paper computes, written
with numpy and sharing no code with the HIP kernels.

Precision: dequantized weights are formed exactly in float64 (an fp16 or
bf16 scale times a small integer is exact), GEMMs accumulate in float64 (or
float32 when asked), and every tensor the paper's experiments hold in FP16
(Y1, Y2) is rounded to fp16 with round-to-nearest-even (numpy's float64 ->
float16 cast rounds once, correctly). With dtype="bf16" (not in the paper:
the activations and scales are bfloat16) Y1 and Y2 are rounded to bfloat16
instead, also once and to nearest even (to_bf16).

Readings of the paper taken here (the paper is silent on them):
  * dequant is asymmetric: w = s * (q - z) with q the stored int4 code and z
    the stored zero code plus the layer's zero offset (0 by default; 1 for
    packers that store z - 1, so that z = 16 is reachable);
  * groups: Eq. 3 with a permutation phi gives every group G rows except a
    partial last group of K - (ng - 1) G rows when G does not divide K
    (ng = ceil(K / G)); a checkpoint may also carry groups of unequal sizes
    (G = 0 here), given by g_idx alone;
  * storage: qweight int32 [K/8][N], nibble j of word [r][n] is row 8r+j;
    qzeros int32 [K/G][N/8], nibble j of word [g][c] is column 8c+j;
  * the argsort of Alg. 1 is stable (ties by ascending row index) and
    ascending; M[P] is a gather (new index j takes old index P[j]);
  * P2 is global over all N1 = K2 rows and the shards are cut afterwards;
  * no activation between the two GEMMs (single up_proj then down_proj).
"""
from __future__ import annotations

import numpy as np

# ----------------------------------------------------------------------------
# Storage format: int4 codes packed eight to an int32 word.
# ----------------------------------------------------------------------------


def unpack_rows(qweight: np.ndarray) -> np.ndarray:
    """Codes q[k][n] of a K x N int4 weight stored as int32 [K/8][N] (group
    quantization of a K x N weight, section 1.1)."""
    w = np.asarray(qweight).view(np.uint32)
    kw, n = w.shape
    q = np.empty((kw * 8, n), dtype=np.int64)
    for j in range(8):
        q[j::8, :] = (w >> np.uint32(4 * j)) & np.uint32(0xF)
    return q


def pack_rows(q: np.ndarray) -> np.ndarray:
    """Inverse of unpack_rows: codes [K][N] (0..15) -> int32 [K/8][N]."""
    q = np.asarray(q, dtype=np.uint32)
    k, n = q.shape
    if k % 8:
        raise ValueError("K must be a multiple of 8")
    if q.max(initial=0) > 15:
        raise ValueError("codes must be 0..15")
    w = np.zeros((k // 8, n), dtype=np.uint32)
    for j in range(8):
        w |= q[j::8, :] << np.uint32(4 * j)
    return w.view(np.int32)


def unpack_cols(qzeros: np.ndarray) -> np.ndarray:
    """Zero codes z[g][n] stored as int32 [num_groups][N/8]."""
    w = np.asarray(qzeros).view(np.uint32)
    ng, nw = w.shape
    z = np.empty((ng, nw * 8), dtype=np.int64)
    for j in range(8):
        z[:, j::8] = (w >> np.uint32(4 * j)) & np.uint32(0xF)
    return z


def pack_cols(z: np.ndarray) -> np.ndarray:
    z = np.asarray(z, dtype=np.uint32)
    ng, n = z.shape
    if n % 8:
        raise ValueError("N must be a multiple of 8")
    if z.max(initial=0) > 15:
        raise ValueError("codes must be 0..15")
    w = np.zeros((ng, n // 8), dtype=np.uint32)
    for j in range(8):
        w |= z[:, j::8] << np.uint32(4 * j)
    return w.view(np.int32)


# ----------------------------------------------------------------------------
# Group index arrays (section 1.1, Eq. 1-3) and the reorder (section 2.1, Alg. 1)
# ----------------------------------------------------------------------------


def g_idx_naive(K: int, G: int) -> np.ndarray:
    """Eq. 1: g[i] = floor(i / G) for i = 0..K-1."""
    return np.array([i // G for i in range(K)], dtype=np.int64)


def g_idx_actorder(phi: np.ndarray, G: int) -> np.ndarray:
    """Eq. 3: g[i] = floor(phi(i) / G), phi a permutation of 0..K-1 (Eq. 2)."""
    return np.asarray(phi, dtype=np.int64) // G


class GroupIndexError(ValueError):
    pass


def eq3_group_counts(K: int, G: int) -> np.ndarray:
    """Rows per group that Eq. 3 gives for a permutation phi of 0..K-1: the
    values phi(i) in [g G, (g + 1) G) are exactly those of group g, so every
    group has G rows except the last, which has K - (ng - 1) G (ng =
    ceil(K / G))."""
    ng = -(-K // G)
    counts = np.full(ng, G, dtype=np.int64)
    counts[-1] = K - (ng - 1) * G
    return counts


def check_groups(g_idx: np.ndarray, G: int, num_groups: int | None = None) -> None:
    """G > 0: every g_idx value is a group index and the groups hold the rows
    Eq. 3 gives (eq3_group_counts: G each, a partial last group when G does
    not divide K). G == 0: groups of any size (a checkpoint's own grouping);
    only the range [0, num_groups) is checked."""
    g = np.asarray(g_idx, dtype=np.int64)
    K = g.shape[0]
    if G == 0:
        if num_groups is None:
            raise GroupIndexError("groups of unequal size need num_groups")
    elif num_groups is None:
        num_groups = -(-K // G)
    if g.size and (g.min() < 0 or g.max() >= num_groups):
        raise GroupIndexError("g_idx value out of range")
    if G == 0:
        return
    counts = np.bincount(g, minlength=num_groups)
    if num_groups != -(-K // G) or np.any(counts != eq3_group_counts(K, G)):
        raise GroupIndexError("the groups do not hold the rows Eq. 3 gives")


def reorder(g_idx: np.ndarray):
    """Alg. 1 (Reorder): P = argsort(g_idx), g_opt = g_idx[P].

    The argsort is ascending and stable (equal group indices keep ascending
    row order), so P is unique."""
    g = np.asarray(g_idx, dtype=np.int64)
    P = np.argsort(g, kind="stable")
    return P.astype(np.int64), g[P]


# ----------------------------------------------------------------------------
# Dequantization and the W4A16 GEMM (section 1.1; Fig. 1 and Fig. 2 loads)
# ----------------------------------------------------------------------------


def dequant(qweight, scales, qzeros, g_idx, cols=None, zero_offset=0) -> np.ndarray:
    """W[k][n] = s[g_idx[k]][n] * (q[k][n] - z[g_idx[k]][n]) in float64, with
    z the stored zero code plus zero_offset.

    Row k takes its scale and zero from group g_idx[k] (Eq. 3 for act-order,
    Eq. 1 / the sorted g_idx for ordered weights). `cols` restricts the result
    to a subset of output columns."""
    g = np.asarray(g_idx, dtype=np.int64)
    if cols is None:
        q = unpack_rows(qweight)
        z = unpack_cols(qzeros)
        s = np.asarray(scales).astype(np.float64)
    else:
        # codes are packed along K, so a column of words is a column of codes
        cols = np.asarray(cols, dtype=np.int64)
        q = unpack_rows(np.asarray(qweight)[:, cols])
        z = unpack_cols(qzeros)[:, cols]
        s = np.asarray(scales)[:, cols].astype(np.float64)
    return s[g, :] * (q - (z[g, :] + int(zero_offset))).astype(np.float64)


def matmul(X, W, acc="f64") -> np.ndarray:
    """Y = X @ W accumulated in float64 (default) or float32."""
    dt = np.float64 if acc == "f64" else np.float32
    return np.asarray(X).astype(dt) @ np.asarray(W).astype(dt)


def to_fp16(a) -> np.ndarray:
    return np.asarray(a).astype(np.float16)


def to_bf16(a) -> np.ndarray:
    """Round to bfloat16 (8 significant bits, ties to even), once, from the
    float64 value; returned as float32, which holds every bfloat16 exactly.

    With x = m * 2**e and 1/2 <= |m| < 1, the rounded value is
    round(m * 2**8) * 2**(e - 8), numpy's round sending halves to the even
    integer. Normal range only (|x| >= 2**-126): the values here are far
    from both ends of it."""
    x = np.asarray(a, dtype=np.float64)
    m, e = np.frexp(x)
    return np.ldexp(np.round(m * 256.0), e - 8).astype(np.float32)


def round_to(a, dtype="fp16") -> np.ndarray:
    """Round to the storage type of activations and outputs."""
    if dtype == "fp16":
        return to_fp16(a)
    if dtype == "bf16":
        return to_bf16(a)
    raise ValueError(f"unknown dtype {dtype}")


def w4a16_gemm(X, qweight, scales, qzeros, g_idx, x_perm=None, acc="f64", cols=None,
               round_fp16=True, dtype="fp16", zero_offset=0):
    """Y[m][n] = sum_k X'[m][k] * W[k][n] with X' = X[:, x_perm] when a gather
    is given (the X[:, P1] of Alg. 2 and Alg. 3), rounded to fp16 (or to
    bfloat16 with dtype="bf16"; round_fp16=False keeps the float64 sum)."""
    X = np.asarray(X)
    if x_perm is not None:
        X = X[:, np.asarray(x_perm, dtype=np.int64)]
    Y = matmul(X, dequant(qweight, scales, qzeros, g_idx, cols, zero_offset), acc)
    return round_to(Y, dtype) if round_fp16 else Y


# ----------------------------------------------------------------------------
# TP-aware fold (section 2.2, Alg. 3) and the Megatron shards
# ----------------------------------------------------------------------------


def fold(w1, w2, P1, P2):
    """Offline permutation of Alg. 3's inputs.

    W1' = W1[P1, P2]: rows gathered by P1 and columns by P2; its scales and
    zeros (one per group and column) follow the column gather. W2' = W2[P2]:
    rows gathered by P2; its scales and zeros are unchanged because they are
    indexed by group, not by row. w1/w2 are dicts with qweight, scales,
    qzeros. Returns (w1', w2') as dicts of packed arrays."""
    P1 = np.asarray(P1, dtype=np.int64)
    P2 = np.asarray(P2, dtype=np.int64)
    q1 = unpack_rows(w1["qweight"])[P1][:, P2]
    s1, z1 = fold_meta(w1["scales"], w1["qzeros"], P2)
    out1 = dict(qweight=pack_rows(q1), scales=s1, qzeros=z1)
    out2 = None
    if w2 is not None:
        q2 = unpack_rows(w2["qweight"])[P2]
        out2 = dict(qweight=pack_rows(q2), scales=np.asarray(w2["scales"]).copy(),
                    qzeros=np.asarray(w2["qzeros"]).copy())
    return out1, out2


def fold_meta(scales, qzeros, P2):
    """Metadata of W1[P1, P2]: the scale and zero of each (group, column)
    follow the column gather by P2 (rows are indexed by group, not by row)."""
    P2 = np.asarray(P2, dtype=np.int64)
    return np.asarray(scales)[:, P2].copy(), pack_cols(unpack_cols(qzeros)[:, P2])


def permute_rows(w, P):
    """W[P] alone (Alg. 1 applied to one layer): rows gathered by P."""
    q = unpack_rows(w["qweight"])[np.asarray(P, dtype=np.int64)]
    return dict(qweight=pack_rows(q), scales=np.asarray(w["scales"]).copy(),
                qzeros=np.asarray(w["qzeros"]).copy())


def column_shard(w, rank, tp):
    """Column-parallel shard (Megatron column-TP, section 2.2): columns
    [rank*N/tp, (rank+1)*N/tp) of the weight and of its metadata."""
    N = w["qweight"].shape[1]
    n = N // tp
    c0 = rank * n
    return dict(qweight=w["qweight"][:, c0:c0 + n], scales=w["scales"][:, c0:c0 + n],
                qzeros=w["qzeros"][:, c0 // 8:(c0 + n) // 8])


def row_shard(w, rank, tp, G, keep_all_groups=False):
    """Row-parallel shard (Megatron row-TP): rows [rank*K/tp, (rank+1)*K/tp).

    For sorted rows the shard's groups are the consecutive block
    [rank*K/(tp*G), ...). An act-order shard (keep_all_groups) keeps every
    group's metadata, since its rows may reference any group."""
    K = w["qweight"].shape[0] * 8
    k = K // tp
    r0 = rank * k
    out = dict(qweight=w["qweight"][r0 // 8:(r0 + k) // 8, :])
    if keep_all_groups:
        out.update(scales=w["scales"], qzeros=w["qzeros"])
    else:
        g0, ng = r0 // G, k // G
        out.update(scales=w["scales"][g0:g0 + ng], qzeros=w["qzeros"][g0:g0 + ng])
    return out


# ----------------------------------------------------------------------------
# The MLP (section 2.2; Alg. 2 and Alg. 3 per rank, collectives simulated)
# ----------------------------------------------------------------------------


def _layer(w, g):
    return w["qweight"], w["scales"], w["qzeros"], g


def mlp_reference(X, w1, g1, w2, g2, acc="f64", y1_fp16=True, dtype="fp16"):
    """Unsharded act-order MLP: Y2 = (X @ deq(W1)) @ deq(W2), Y1 in fp16 (or
    the dtype given)."""
    Y1 = w4a16_gemm(X, *_layer(w1, g1), acc=acc, round_fp16=y1_fp16, dtype=dtype)
    return w4a16_gemm(Y1, *_layer(w2, g2), acc=acc, dtype=dtype)


def mlp_tp_aware_rank(X, P1, w1f_shard, w2f_shard, G, acc="f64", y1_fp16=True, round_y2=True,
                      dtype="fp16", g1=None, g2=None):
    """Alg. 3 on one rank, up to its AllReduce:
      Y1_local = X[:, P1] @ W1_local   (W1_local a column shard of W1[P1, P2])
      Y2_local = Y1_local @ W2_local   (W2_local a row shard of W2[P2])
    Both shards hold sorted rows, so their group of local row k is floor(k/G)
    (Eq. 1 applied to the shard). With groups of unequal size (G = 0) the
    sorted group indices of the shards' rows are given instead (g1, g2; a
    row shard of W2 then keeps every group's metadata)."""
    K1 = w1f_shard["qweight"].shape[0] * 8
    K2 = w2f_shard["qweight"].shape[0] * 8
    g1 = g_idx_naive(K1, G) if g1 is None else g1
    g2 = g_idx_naive(K2, G) if g2 is None else g2
    Y1 = w4a16_gemm(X, *_layer(w1f_shard, g1), x_perm=P1, acc=acc, round_fp16=y1_fp16, dtype=dtype,
                    zero_offset=w1f_shard.get("zero_offset", 0))
    Y2 = w4a16_gemm(Y1, *_layer(w2f_shard, g2), acc=acc, round_fp16=round_y2, dtype=dtype,
                    zero_offset=w2f_shard.get("zero_offset", 0))
    return Y1, Y2


def mlp_actorder_rank(X, w1_shard, g1, w2_shard, g2_shard, acc="f64", y1_fp16=True, round_y2=True,
                      dtype="fp16"):
    """The act-order (no reorder) MLP on one rank: column shard of W1 with its
    g_idx, row shard of W2 with the global g_idx values of its rows and the
    full metadata (Eq. 3 loads, Fig. 1)."""
    Y1 = w4a16_gemm(X, *_layer(w1_shard, g1), acc=acc, round_fp16=y1_fp16, dtype=dtype)
    Y2 = w4a16_gemm(Y1, *_layer(w2_shard, g2_shard), acc=acc, round_fp16=round_y2, dtype=dtype)
    return Y1, Y2


def all_reduce_sum(partials, round_fp16=True):
    """Simulated AllReduce(SUM) of the per-rank partials (float64 sum)."""
    total = np.zeros_like(np.asarray(partials[0], dtype=np.float64))
    for p in partials:
        total = total + np.asarray(p, dtype=np.float64)
    return to_fp16(total) if round_fp16 else total


def all_gather_cols(shards):
    """Simulated AllGather along dim 1."""
    return np.concatenate([np.asarray(s) for s in shards], axis=1)


def mlp_naive_algorithm(X, P1, P2, w1o, w2o, G, tp, acc="f64"):
    """Alg. 2 with every rank simulated in one process.

    w1o = W1[P1] (rows sorted, columns untouched), w2o = W2[P2]. Per rank:
    Y1_local = X[:, P1] @ W1_local; then AllGather(Y1), Y1_global[:, P2],
    CHUNK, Y2_local = Y1_local @ W2_local; then AllReduce. Returns Y2 and the
    per-rank partials."""
    K1 = w1o["qweight"].shape[0] * 8
    y1_shards = []
    for r in range(tp):
        w1r = column_shard(w1o, r, tp)
        y1_shards.append(w4a16_gemm(X, *_layer(w1r, g_idx_naive(K1, G)), x_perm=P1, acc=acc))
    Y1g = all_gather_cols(y1_shards)[:, np.asarray(P2, dtype=np.int64)]
    n = Y1g.shape[1] // tp
    partials = []
    for r in range(tp):
        w2r = row_shard(w2o, r, tp, G)
        y1l = Y1g[:, r * n:(r + 1) * n]
        partials.append(w4a16_gemm(y1l, *_layer(w2r, g_idx_naive(n, G)), acc=acc))
    return all_reduce_sum(partials), partials


def mlp_tp_aware(X, P1, w1f, w2f, G, tp, acc="f64"):
    """Alg. 3 with every rank simulated in one process (w1f = W1[P1, P2],
    w2f = W2[P2]). Returns the AllReduced Y2 and the per-rank partials."""
    partials = []
    for r in range(tp):
        _, y2 = mlp_tp_aware_rank(X, P1, column_shard(w1f, r, tp), row_shard(w2f, r, tp, G), G, acc)
        partials.append(y2)
    return all_reduce_sum(partials), partials


# ----------------------------------------------------------------------------
# Gated MLP (the experiments section notes that the method carries over to an
# MLP with a gate projection): Y1 = silu(X W_gate) * (X W_up), Y2 = Y1 W_down.
# Readings: gate and up take the same input, hence the same act-order
# permutation (one g_idx, one P1); P2 (from W_down) is folded into the columns
# of both; both products stay unrounded until Y1, which is rounded once.
# ----------------------------------------------------------------------------


def silu(x) -> np.ndarray:
    """x * sigma(x) = x / (1 + exp(-x)) in float64."""
    x = np.asarray(x, dtype=np.float64)
    return x / (1.0 + np.exp(-x))


def gated_y1(X, gate, up, g_idx, x_perm=None, acc="f64", cols=None, round_fp16=True, dtype="fp16"):
    """Y1 = silu(X' @ deq(W_gate)) * (X' @ deq(W_up)), X' = X[:, x_perm] when
    given; gate and up are (qweight, scales, qzeros) of the same shape sharing
    g_idx. Rounded once to the storage type (round_fp16=False: float64)."""
    yg = w4a16_gemm(X, *gate, g_idx, x_perm=x_perm, acc=acc, cols=cols, round_fp16=False)
    yu = w4a16_gemm(X, *up, g_idx, x_perm=x_perm, acc=acc, cols=cols, round_fp16=False)
    y = silu(yg) * yu
    return round_to(y, dtype) if round_fp16 else y


def _triple(w):
    return w["qweight"], w["scales"], w["qzeros"]


def gated_mlp_reference(X, gate, up, g1, down, g2, acc="f64", y1_fp16=True, dtype="fp16"):
    """Unsharded act-order gated MLP (dicts of packed arrays; g1 shared by
    gate and up)."""
    Y1 = gated_y1(X, _triple(gate), _triple(up), g1, acc=acc, round_fp16=y1_fp16, dtype=dtype)
    return w4a16_gemm(Y1, *_triple(down), g2, acc=acc, dtype=dtype)


def gated_mlp_tp_aware_rank(X, P1, gate_f, up_f, down_f, G, acc="f64", y1_fp16=True, round_y2=True,
                            dtype="fp16"):
    """Alg. 3 for the gated MLP on one rank: gate_f and up_f are column shards
    of W_gate[P1, P2] and W_up[P1, P2], down_f a row shard of W_down[P2]; all
    hold sorted rows, so their local group of row k is floor(k / G)."""
    K1 = gate_f["qweight"].shape[0] * 8
    K2 = down_f["qweight"].shape[0] * 8
    Y1 = gated_y1(X, _triple(gate_f), _triple(up_f), g_idx_naive(K1, G), x_perm=P1, acc=acc,
                  round_fp16=y1_fp16, dtype=dtype)
    Y2 = w4a16_gemm(Y1, *_triple(down_f), g_idx_naive(K2, G), acc=acc, round_fp16=round_y2, dtype=dtype)
    return Y1, Y2


def gated_rank_from_global(X, lg, lu, l2, rank, tp, ordered, P2=None, cols2=None, acc="f64",
                           dtype="fp16", y1_round=True, round_y2=True):
    """One rank's (Y1, Y2 partial[:, cols2]) of the gated MLP from the
    unpermuted global layers lg, lu = (qweight, scales, qzeros, g_idx) with a
    shared g_idx, and l2; column block `rank` of gate and up (original columns
    P2[block] when ordered), as in mlp_rank_from_global. y1_round / round_y2
    False keep Y1 / Y2 in float64."""
    N1 = np.asarray(lg[0]).shape[1]
    n = N1 // tp
    blk = np.arange(rank * n, (rank + 1) * n)
    sel = np.asarray(P2, dtype=np.int64)[blk] if ordered else blk
    yg = matmul(X, dequant(*lg, cols=sel), acc)
    yu = matmul(X, dequant(*lu, cols=sel), acc)
    Y1 = silu(yg) * yu
    if y1_round:
        Y1 = round_to(Y1, dtype)
    W2 = dequant(*l2, cols=cols2)[sel]
    Y2 = matmul(Y1, W2, acc)
    return Y1, (round_to(Y2, dtype) if round_y2 else Y2)


def fold_sample(qweight, P_row, P_col, rows, cols):
    """Codes of W[P_row, P_col] at rows x cols (P_col None: columns in place),
    read from the source words element by element; for layers too large to
    unpack whole. New row j / column c take old row P_row[j] / column P_col[c]."""
    src_rows = np.asarray(P_row, dtype=np.int64)[np.asarray(rows, dtype=np.int64)]
    cols = np.asarray(cols, dtype=np.int64)
    src_cols = cols if P_col is None else np.asarray(P_col, dtype=np.int64)[cols]
    words = np.asarray(qweight).view(np.uint32)[np.ix_(src_rows // 8, src_cols)]
    shift = (4 * (src_rows % 8)).astype(np.uint32)[:, None]
    return ((words >> shift) & np.uint32(0xF)).astype(np.int64)


def _split_layer(l):
    """(qweight, scales, qzeros, g_idx[, zero_offset]) -> the four arrays and the offset."""
    return tuple(l[:4]), (int(l[4]) if len(l) > 4 else 0)


def mlp_rank_from_global(X, l1, l2, rank, tp, ordered, P2=None, cols2=None, acc="f64",
                         dtype="fp16", y1_round=True, round_y2=True):
    """One rank's (Y1, Y2 partial[:, cols2]) computed from the unpermuted
    global layers l1 = (qweight, scales, qzeros, g_idx) and l2.

    Act-order rank (Megatron shards of the original layers): W1 columns and
    W2 rows [rank*n, (rank+1)*n), n = N1/tp.
    TP-aware rank (Alg. 3): its W1[P1, P2] column block holds original columns
    P2[block] with rows relabelled by P1, and its W2[P2] row block holds
    original rows P2[block]; since relabelling the rows of W1 together with
    the columns of X (X[:, P1]) leaves every dot product's terms unchanged, the
    partial is X @ deq(W1)[:, P2[block]] then @ deq(W2)[P2[block], :].
    y1_round / round_y2 False keep Y1 / Y2 in float64."""
    (l1, zo1), (l2, zo2) = _split_layer(l1), _split_layer(l2)
    N1 = np.asarray(l1[0]).shape[1]
    n = N1 // tp
    blk = np.arange(rank * n, (rank + 1) * n)
    sel = np.asarray(P2, dtype=np.int64)[blk] if ordered else blk
    Y1 = matmul(X, dequant(*l1, cols=sel, zero_offset=zo1), acc)
    if y1_round:
        Y1 = round_to(Y1, dtype)
    W2 = dequant(*l2, cols=cols2, zero_offset=zo2)[sel]
    Y2 = matmul(Y1, W2, acc)
    return Y1, (round_to(Y2, dtype) if round_y2 else Y2)


# ----------------------------------------------------------------------------
# Metric helpers used by the tests
# ----------------------------------------------------------------------------


def rel_err(y, ref) -> float:
    """max|y - ref| / max|ref| (the acceptance measure for fp16 outputs)."""
    y = np.asarray(y, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    denom = np.max(np.abs(ref)) if ref.size else 0.0
    if denom == 0.0:
        return float(np.max(np.abs(y - ref), initial=0.0))
    return float(np.max(np.abs(y - ref)) / denom)


def distinct_groups_per_tile(g_idx, T) -> np.ndarray:
    """Distinct metadata rows a tile of T consecutive weight rows touches."""
    g = np.asarray(g_idx, dtype=np.int64)
    return np.array([len(np.unique(g[i:i + T])) for i in range(0, len(g), T)])


def expected_distinct_groups(K, G, T, num_groups=None):
    """Expectation of distinct_groups_per_tile for a uniform permutation:
    ng * (1 - C(K-G, T) / C(K, T)) (each group has G of the K rows)."""
    ng = K // G if num_groups is None else num_groups
    p_miss = 1.0
    for i in range(T):
        p_miss *= (K - G - i) / (K - i)
    return ng * (1.0 - p_miss)
