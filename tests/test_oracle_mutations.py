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
