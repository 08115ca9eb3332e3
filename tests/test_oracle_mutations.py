"""Plant plausible mistakes in the oracle (on the CPU) and check that at least
one pin catches each of them, so the pins are known to bite."""
import numpy as np
import pytest

from oracle import tpdq_oracle as o
from tests import pins

_orig = {name: getattr(o, name) for name in dir(o) if callable(getattr(o, name))}


def _unpack_rows_reversed(qweight):
    w = np.asarray(qweight).view(np.uint32)
    q = np.empty((w.shape[0] * 8, w.shape[1]), dtype=np.int64)
    for j in range(8):
        q[j::8] = (w >> np.uint32(4 * (7 - j))) & np.uint32(0xF)
    return q


def _unpack_cols_reversed(qzeros):
    w = np.asarray(qzeros).view(np.uint32)
    z = np.empty((w.shape[0], w.shape[1] * 8), dtype=np.int64)
    for j in range(8):
        z[:, j::8] = (w >> np.uint32(4 * (7 - j))) & np.uint32(0xF)
    return z


def _dequant_no_zero(qweight, scales, qzeros, g_idx, cols=None):
    q = _orig["unpack_rows"](qweight)
    s = np.asarray(scales).astype(np.float64)
    g = np.asarray(g_idx, dtype=np.int64)
    if cols is not None:
        q, s = q[:, cols], s[:, cols]
    return s[g] * q


def _dequant_sign(qweight, scales, qzeros, g_idx, cols=None):
    return -_orig["dequant"](qweight, scales, qzeros, g_idx, cols)


def _dequant_shifted_group(qweight, scales, qzeros, g_idx, cols=None):
    g = np.roll(np.asarray(g_idx, dtype=np.int64), 1)
    return _orig["dequant"](qweight, scales, qzeros, g, cols)


def _reorder_unstable(g_idx):
    g = np.asarray(g_idx, dtype=np.int64)
    K = len(g)
    P = np.lexsort((-np.arange(K), g))     # ties by descending row
    return P, g[P]


def _reorder_descending(g_idx):
    g = np.asarray(g_idx, dtype=np.int64)
    P = np.argsort(-g, kind="stable")
    return P, g[P]


def _reorder_inverse(g_idx):
    P, gs = _orig["reorder"](g_idx)
    inv = np.empty_like(P)
    inv[P] = np.arange(len(P))
    return inv, gs


def _fold_no_scale_perm(w1, w2, P1, P2):
    a, b = _orig["fold"](w1, w2, P1, P2)
    a["scales"] = np.asarray(w1["scales"]).copy()
    return a, b


def _fold_no_zero_perm(w1, w2, P1, P2):
    a, b = _orig["fold"](w1, w2, P1, P2)
    a["qzeros"] = np.asarray(w1["qzeros"]).copy()
    return a, b


def _fold_rows_only(w1, w2, P1, P2):
    a, b = _orig["fold"](w1, w2, P1, np.arange(len(P2)))
    a2, b2 = _orig["fold"](w1, w2, P1, P2)
    return a, b2


def _row_shard_no_offset(w, rank, tp, G, keep_all_groups=False):
    out = _orig["row_shard"](w, rank, tp, G, keep_all_groups)
    if not keep_all_groups:
        K = w["qweight"].shape[0] * 8
        ng = K // tp // G
        out["scales"] = w["scales"][:ng]
        out["qzeros"] = w["qzeros"][:ng]
    return out


def _gemm_ignores_perm(X, qweight, scales, qzeros, g_idx, x_perm=None, acc="f64", cols=None,
                       round_fp16=True, dtype="fp16"):
    return _orig["w4a16_gemm"](X, qweight, scales, qzeros, g_idx, None, acc, cols, round_fp16, dtype)


def _eq3_ceil(phi, G):
    return -(-np.asarray(phi, dtype=np.int64) // G)


def _bf16_truncate(a):
    x = np.asarray(a, dtype=np.float64)
    m, e = np.frexp(x)
    return np.ldexp(np.trunc(m * 256.0), e - 8).astype(np.float32)


def _round_to_fp16_always(a, dtype="fp16"):
    return np.asarray(a).astype(np.float16)


def _silu_is_sigmoid(x):
    x = np.asarray(x, dtype=np.float64)
    return 1.0 / (1.0 + np.exp(-x))


def _gated_silu_on_up(X, gate, up, g_idx, x_perm=None, acc="f64", cols=None, round_fp16=True,
                      dtype="fp16"):
    return _orig["gated_y1"](X, up, gate, g_idx, x_perm, acc, cols, round_fp16, dtype)


def _rank_mutant(kind, gated):
    """mlp_rank_from_global / gated_rank_from_global with one planted mistake:
    'blk' the unpermuted column block on the ordered path, 'inv' P2's inverse
    in place of P2, 'w2cols' the selection applied to W2's columns instead of
    its rows (W2's rows then taken in block order)."""
    def f(X, l1, *rest, **kw):
        if gated:
            lu, l2, rank, tp, ordered = rest[0], rest[1], rest[2], rest[3], rest[4]
        else:
            l2, rank, tp, ordered = rest[0], rest[1], rest[2], rest[3]
        P2 = kw.get("P2")
        cols2 = kw.get("cols2")
        acc = kw.get("acc", "f64")
        dtype = kw.get("dtype", "fp16")
        y1_round = kw.get("y1_round", True)
        round_y2 = kw.get("round_y2", True)
        N1 = np.asarray(l1[0]).shape[1]
        n = N1 // tp
        blk = np.arange(rank * n, (rank + 1) * n)
        P2 = np.asarray(P2, dtype=np.int64)
        if kind == "inv":
            inv = np.empty_like(P2)
            inv[P2] = np.arange(len(P2))
            P2 = inv
        sel = P2[blk] if (ordered and kind != "blk") else blk
        if gated:
            Y1 = o.silu(o.matmul(X, o.dequant(*l1, cols=sel), acc)) * o.matmul(X, o.dequant(*lu, cols=sel), acc)
        else:
            Y1 = o.matmul(X, o.dequant(*l1, cols=sel), acc)
        if y1_round:
            Y1 = o.round_to(Y1, dtype)
        if kind == "w2cols":
            W2 = o.dequant(*l2, cols=cols2)[blk]  # W2's rows in block order
        else:
            W2 = o.dequant(*l2, cols=cols2)[sel]
        Y2 = o.matmul(Y1, W2, acc)
        return Y1, (o.round_to(Y2, dtype) if round_y2 else Y2)
    return f


def _fold_sample_unpermuted_rows(qweight, P_row, P_col, rows, cols):
    return _orig["fold_sample"](qweight, np.arange(len(P_row)), P_col, rows, cols)


def _fold_sample_shift(qweight, P_row, P_col, rows, cols):
    src_rows = np.asarray(P_row, dtype=np.int64)[np.asarray(rows, dtype=np.int64)]
    cols = np.asarray(cols, dtype=np.int64)
    src_cols = cols if P_col is None else np.asarray(P_col, dtype=np.int64)[cols]
    words = np.asarray(qweight).view(np.uint32)[np.ix_(src_rows // 8, src_cols)]
    shift = (4 * (7 - src_rows % 8)).astype(np.uint32)[:, None]
    return ((words >> shift) & np.uint32(0xF)).astype(np.int64)


def _fold_sample_inverse_cols(qweight, P_row, P_col, rows, cols):
    if P_col is not None:
        P_col = np.asarray(P_col, dtype=np.int64)
        inv = np.empty_like(P_col)
        inv[P_col] = np.arange(len(P_col))
        P_col = inv
    return _orig["fold_sample"](qweight, P_row, P_col, rows, cols)


def _dequant_offset_ignored(qweight, scales, qzeros, g_idx, cols=None, zero_offset=0):
    return _orig["dequant"](qweight, scales, qzeros, g_idx, cols, 0)


def _dequant_offset_sign(qweight, scales, qzeros, g_idx, cols=None, zero_offset=0):
    return _orig["dequant"](qweight, scales, qzeros, g_idx, cols, -zero_offset)


def _check_groups_strict(g_idx, G, num_groups=None):
    g = np.asarray(g_idx, dtype=np.int64)
    if G == 0:
        return _orig["check_groups"](g_idx, G, num_groups)
    if len(g) % G:
        raise o.GroupIndexError("K must be a multiple of G")
    return _orig["check_groups"](g_idx, G, num_groups)


def _eq3_counts_full(K, G):
    ng = -(-K // G)
    return np.full(ng, G, dtype=np.int64)


MUTANTS = {
    "unpack_rows": _unpack_rows_reversed,
    "unpack_cols": _unpack_cols_reversed,
    "dequant:no_zero": _dequant_no_zero,
    "dequant:sign": _dequant_sign,
    "dequant:group_shift": _dequant_shifted_group,
    "reorder:unstable": _reorder_unstable,
    "reorder:descending": _reorder_descending,
    "reorder:inverse": _reorder_inverse,
    "fold:scales": _fold_no_scale_perm,
    "fold:zeros": _fold_no_zero_perm,
    "fold:columns": _fold_rows_only,
    "row_shard:offset": _row_shard_no_offset,
    "w4a16_gemm:perm": _gemm_ignores_perm,
    "g_idx_actorder:ceil": _eq3_ceil,
    "to_bf16:truncate": _bf16_truncate,
    "round_to:fp16": _round_to_fp16_always,
    "silu:sigmoid": _silu_is_sigmoid,
    "gated_y1:swapped": _gated_silu_on_up,
    "mlp_rank_from_global:blk": _rank_mutant("blk", False),
    "mlp_rank_from_global:inverse_P2": _rank_mutant("inv", False),
    "mlp_rank_from_global:w2_columns": _rank_mutant("w2cols", False),
    "gated_rank_from_global:blk": _rank_mutant("blk", True),
    "gated_rank_from_global:inverse_P2": _rank_mutant("inv", True),
    "gated_rank_from_global:w2_columns": _rank_mutant("w2cols", True),
    "fold_sample:rows": _fold_sample_unpermuted_rows,
    "fold_sample:shift": _fold_sample_shift,
    "fold_sample:inverse_cols": _fold_sample_inverse_cols,
    "dequant:zero_offset_ignored": _dequant_offset_ignored,
    "dequant:zero_offset_sign": _dequant_offset_sign,
    "check_groups:no_partial_group": _check_groups_strict,
    "eq3_group_counts:full_last_group": _eq3_counts_full,
}


@pytest.mark.parametrize("key", sorted(MUTANTS))
def test_mutant_is_caught(key, monkeypatch):
    name = key.split(":")[0]
    monkeypatch.setattr(o, name, MUTANTS[key])
    caught = []
    for pin in pins.ALL_PINS:
        try:
            pin(o)
        except Exception:  # an assertion, or a shape error the mistake causes
            caught.append(pin.__name__)
    assert caught, f"no pin catches the planted mistake {key}"
