"""Pins of the CPU oracle: checks against what the paper and the mathematics fix.

Each pin is a plain function taking the oracle module, so that the mutation
tests can run the same pin against an oracle with a planted mistake and see it
fail. None of these re-types the oracle's own formula: they use hand-worked
values, closed forms, invariants, and brute force by other means.
"""
from __future__ import annotations

import os

import numpy as np

from paper_2402_04925_amd import inputs

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load_golden(name):
    out = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            k, v = line.split(":", 1)
            out[k.strip()] = v.split()
    return out


def hex_words(vals):
    return np.array([int(v, 16) for v in vals], dtype=np.uint32).view(np.int32)


def nibble_by_hex(word: int, j: int) -> int:
    """Nibble j of a 32-bit word read off its hexadecimal spelling (digit 7-j),
    a route independent of shifts and masks."""
    return int(format(word & 0xFFFFFFFF, "08x")[7 - j], 16)


# ---------------------------------------------------------------- storage ---

def pin_unpack_bruteforce(o, seed=1):
    """P1: every code of a random tiny weight and zero array, read one element
    at a time off the hex spelling of its word."""
    w1, _ = inputs.make_custom(64, 24, 0, 16, seed)
    q = o.unpack_rows(w1.qweight)
    z = o.unpack_cols(w1.qzeros)
    words = w1.qweight.view(np.uint32)
    for k in range(64):
        for n in range(24):
            assert q[k, n] == nibble_by_hex(int(words[k // 8, n]), k % 8), (k, n)
    zw = w1.qzeros.view(np.uint32)
    for g in range(4):
        for n in range(24):
            assert z[g, n] == nibble_by_hex(int(zw[g, n // 8]), n % 8), (g, n)


def pin_pack_roundtrip(o, seed=2):
    """P2: pack(unpack(words)) == words and unpack(pack(codes)) == codes."""
    w1, _ = inputs.make_custom(128, 40, 0, 32, seed)
    assert np.array_equal(o.pack_rows(o.unpack_rows(w1.qweight)), w1.qweight)
    assert np.array_equal(o.pack_cols(o.unpack_cols(w1.qzeros)), w1.qzeros)
    rng = np.random.default_rng(seed)
    codes = rng.integers(0, 16, size=(48, 16))
    assert np.array_equal(o.unpack_rows(o.pack_rows(codes)), codes)
    assert np.array_equal(o.unpack_cols(o.pack_cols(codes)), codes)


def pin_golden_gemm_codes(o):
    """Hand-worked codes: word 0x76543210 holds code k in row k."""
    gd = load_golden("gemm_worked_example.txt")
    qw = hex_words(gd["qweight_hex"]).reshape(1, 8)
    q = o.unpack_rows(qw)
    for n in range(8):
        expect = np.arange(8) + (8 if n % 2 else 0)
        assert np.array_equal(q[:, n], expect)
    z = o.unpack_cols(hex_words(gd["qzeros_hex"]).reshape(2, 1))
    assert np.array_equal(z[0], np.ones(8)) and np.array_equal(z[1], 2 * np.ones(8))


# ---------------------------------------------------------------- reorder ---

def pin_worked_reorder(o):
    """P10: the hand-worked Eq. 3 / Alg. 1 example."""
    gd = load_golden("reorder_worked_example.txt")
    G = int(gd["G"][0])
    phi = np.array(gd["phi"], dtype=np.int64)
    g = o.g_idx_actorder(phi, G)
    assert np.array_equal(g, np.array(gd["g_idx"], dtype=np.int64))
    P, gs = o.reorder(g)
    assert np.array_equal(P, np.array(gd["P"], dtype=np.int64))
    assert np.array_equal(gs, np.array(gd["g_sorted"], dtype=np.int64))


def pin_reorder_closed_form(o, K=512, G=32, seed=3):
    """P3: for a permutation phi and G | K the sorted g_idx is exactly Eq. 1,
    P is a bijection, and g_idx[P[j]] == g_sorted[j]; within a group the
    original rows keep ascending order (the stable reading)."""
    phi = np.random.default_rng(seed).permutation(K)
    g = o.g_idx_actorder(phi, G)
    P, gs = o.reorder(g)
    assert np.array_equal(gs, np.arange(K) // G)          # Eq. 1
    assert np.array_equal(np.sort(P), np.arange(K))      # bijection
    assert np.array_equal(g[P], gs)
    assert np.all(np.diff(gs) >= 0)                      # monotone
    for grp in range(K // G):
        rows = P[grp * G:(grp + 1) * G]
        assert np.all(np.diff(rows) > 0)                 # ascending inside a group
        assert set(rows.tolist()) == set(np.flatnonzero(g == grp).tolist())


def pin_identity_phi(o, K=256, G=32):
    """P4: phi = identity -> Eq. 3 = Eq. 1 -> P = identity."""
    g = o.g_idx_actorder(np.arange(K), G)
    assert np.array_equal(g, o.g_idx_naive(K, G))
    assert np.array_equal(g, np.arange(K) // G)
    P, gs = o.reorder(g)
    assert np.array_equal(P, np.arange(K))


def pin_check_groups(o):
    """Group validation accepts Eq. 3 output and rejects malformed g_idx."""
    g = o.g_idx_actorder(np.random.default_rng(4).permutation(64), 8)
    o.check_groups(g, 8)
    for bad in (np.where(g == 0, 1, g),                   # group 0 empty
                np.concatenate([g[:-1], [8]]),             # out of range
                np.concatenate([[-1], g[1:]])):            # negative
        try:
            o.check_groups(bad, 8)
        except o.GroupIndexError:
            continue
        raise AssertionError("malformed g_idx accepted")


# ------------------------------------------------------------ dequant+GEMM ---

def pin_golden_gemm(o):
    """Hand-worked dequant + GEMM (act-order) and the same through Alg. 1."""
    gd = load_golden("gemm_worked_example.txt")
    qw = hex_words(gd["qweight_hex"]).reshape(1, 8)
    qz = hex_words(gd["qzeros_hex"]).reshape(2, 1)
    s = np.array([[float(gd["scales_group0"][0])] * 8, [float(gd["scales_group1"][0])] * 8],
                 dtype=np.float16)
    g = np.array(gd["g_idx"], dtype=np.int64)
    X = np.array([gd["X0"], gd["X1"]], dtype=np.float64).astype(np.float16)
    Y = o.w4a16_gemm(X, qw, s, qz, g)
    expect = np.array([gd["Y0"], gd["Y1"]], dtype=np.float64)
    assert np.array_equal(Y.astype(np.float64), expect), Y
    P, gs = o.reorder(g)
    assert np.array_equal(P, np.array(gd["P"], dtype=np.int64))
    assert np.array_equal(gs, np.array(gd["g_sorted"], dtype=np.int64))
    ws = o.permute_rows(dict(qweight=qw, scales=s, qzeros=qz), P)
    assert np.array_equal(ws["qweight"], hex_words(gd["qweight_sorted_hex"]).reshape(1, 8))
    Y2 = o.w4a16_gemm(X, ws["qweight"], s, qz, gs, x_perm=P)
    assert np.array_equal(Y2.astype(np.float64), expect)


def pin_gemm_bruteforce(o, seed=5):
    """P6: the oracle's GEMM against a pure-Python triple loop on tiny inputs,
    codes read off hex spellings, products summed as Python floats."""
    K, N, G, M = 32, 16, 8, 3
    w1, _ = inputs.make_custom(K, N, 0, G, seed)
    X = inputs.random_activations(M, K, np.random.default_rng(seed))
    qw = w1.qweight.view(np.uint32)
    zw = w1.qzeros.view(np.uint32)
    ref = np.zeros((M, N))
    for m in range(M):
        for n in range(N):
            acc = 0.0
            for k in range(K):
                g = int(w1.g_idx[k])
                q = nibble_by_hex(int(qw[k // 8, n]), k % 8)
                z = nibble_by_hex(int(zw[g, n // 8]), n % 8)
                acc += float(X[m, k]) * float(w1.scales[g, n]) * (q - z)
            ref[m, n] = acc
    Y = o.w4a16_gemm(X, w1.qweight, w1.scales, w1.qzeros, w1.g_idx, round_fp16=False)
    assert np.max(np.abs(Y - ref)) <= 1e-12 * max(1.0, np.max(np.abs(ref)))
    Y16 = o.w4a16_gemm(X, w1.qweight, w1.scales, w1.qzeros, w1.g_idx)
    assert np.array_equal(Y16, ref.astype(np.float16))


def pin_one_hot_rows(o, seed=6):
    """Closed form: X = identity rows picks out rows of the dequantized weight,
    and the dequantized row k of column n is s*(q-z) of its own group."""
    K, N, G = 64, 16, 16
    w1, _ = inputs.make_custom(K, N, 0, G, seed)
    X = np.eye(K, dtype=np.float16)
    Y = o.w4a16_gemm(X, w1.qweight, w1.scales, w1.qzeros, w1.g_idx, round_fp16=False)
    qw = w1.qweight.view(np.uint32)
    zw = w1.qzeros.view(np.uint32)
    for k in range(0, K, 7):
        g = int(w1.g_idx[k])
        for n in range(N):
            q = nibble_by_hex(int(qw[k // 8, n]), k % 8)
            z = nibble_by_hex(int(zw[g, n // 8]), n % 8)
            assert Y[k, n] == float(w1.scales[g, n]) * (q - z)


def pin_special_cases(o, seed=7):
    """P5: one group (G = K) and q == z everywhere -> Y == 0; G = K with every
    code = zero + 1 -> Y[m][n] = s[n] * sum_k X[m][k]."""
    K, N = 64, 16
    rng = np.random.default_rng(seed)
    zc = rng.integers(0, 15, size=(1, N))
    qz = o.pack_cols(zc)
    X = inputs.random_activations(3, K, rng)
    s = inputs.random_scales((1, N), rng)
    g = np.zeros(K, dtype=np.int64)
    q_eq = np.repeat(zc, K, axis=0)
    Y = o.w4a16_gemm(X, o.pack_rows(q_eq), s, qz, g, round_fp16=False)
    assert np.all(Y == 0.0)
    Y1 = o.w4a16_gemm(X, o.pack_rows(q_eq + 1), s, qz, g, round_fp16=False)
    expect = np.outer(X.astype(np.float64).sum(axis=1), s[0].astype(np.float64))
    assert np.max(np.abs(Y1 - expect)) <= 1e-12 * np.max(np.abs(expect))


def pin_ordered_equals_actorder(o, seed=8):
    """P7: X[:, P] @ deq(W[P], g[P]) == X @ deq(W, g) (the reorder only
    relabels the terms of each dot product)."""
    K, N, G, M = 256, 48, 32, 4
    w1, _ = inputs.make_custom(K, N, 0, G, seed)
    X = inputs.random_activations(M, K, np.random.default_rng(seed))
    ref = o.w4a16_gemm(X, w1.qweight, w1.scales, w1.qzeros, w1.g_idx, round_fp16=False)
    P, gs = o.reorder(w1.g_idx)
    ws = o.permute_rows(dict(qweight=w1.qweight, scales=w1.scales, qzeros=w1.qzeros), P)
    Y = o.w4a16_gemm(X, ws["qweight"], ws["scales"], ws["qzeros"], gs, x_perm=P, round_fp16=False)
    assert np.max(np.abs(Y - ref)) <= 1e-12 * np.max(np.abs(ref))
    # the ordered weight's group of row j is Eq. 1, so the g_idx need not be read
    Y_eq1 = o.w4a16_gemm(X, ws["qweight"], ws["scales"], ws["qzeros"], o.g_idx_naive(K, G),
                         x_perm=P, round_fp16=False)
    assert np.array_equal(Y_eq1, Y)
    Y32 = o.w4a16_gemm(X, ws["qweight"], ws["scales"], ws["qzeros"], gs, x_perm=P, acc="f32",
                       round_fp16=False)
    assert np.max(np.abs(Y32 - ref)) <= 1e-5 * np.max(np.abs(ref))


# -------------------------------------------------------------------- MLP ---

def _mlp_case(K1, N1, N2, G, seed):
    w1, w2 = inputs.make_custom(K1, N1, N2, G, seed)
    X = inputs.random_activations(3, K1, np.random.default_rng(seed))
    d1 = dict(qweight=w1.qweight, scales=w1.scales, qzeros=w1.qzeros)
    d2 = dict(qweight=w2.qweight, scales=w2.scales, qzeros=w2.qzeros)
    return w1, w2, d1, d2, X


def pin_tp_aware_mlp(o, seed=9, tps=(1, 2, 4, 8)):
    """P8: the sum over ranks of Alg. 3's partials equals the unsharded
    act-order MLP, for every TP degree (the paper's section 2.2 claim)."""
    K1, N1, N2, G = 256, 512, 128, 32
    w1, w2, d1, d2, X = _mlp_case(K1, N1, N2, G, seed)
    ref64 = o.w4a16_gemm(o.w4a16_gemm(X, *_l(d1, w1.g_idx), round_fp16=False),
                         *_l(d2, w2.g_idx), round_fp16=False)
    P1, _ = o.reorder(w1.g_idx)
    P2, _ = o.reorder(w2.g_idx)
    w1f, w2f = o.fold(d1, d2, P1, P2)
    for tp in tps:
        parts = []
        for r in range(tp):
            _, y2 = o.mlp_tp_aware_rank(X, P1, o.column_shard(w1f, r, tp),
                                        o.row_shard(w2f, r, tp, G), G, y1_fp16=False,
                                        round_y2=False)
            parts.append(y2)
        tot = o.all_reduce_sum(parts, round_fp16=False)
        assert np.max(np.abs(tot - ref64)) <= 1e-12 * np.max(np.abs(ref64)), tp
        # with the paper's fp16 activations
        y2_16, _ = o.mlp_tp_aware(X, P1, w1f, w2f, G, tp)
        ref16 = o.mlp_reference(X, d1, w1.g_idx, d2, w2.g_idx)
        assert o.rel_err(y2_16, ref16) <= 2e-3, tp


def _l(d, g):
    return d["qweight"], d["scales"], d["qzeros"], g


def pin_actorder_shard_mlp(o, seed=10, tps=(2, 4)):
    """The act-order (no reorder) rank: a row shard keeps its rows' global
    g_idx values and the full metadata; the ranks' partials sum to the
    unsharded MLP."""
    K1, N1, N2, G = 128, 256, 64, 32
    w1, w2, d1, d2, X = _mlp_case(K1, N1, N2, G, seed)
    ref = o.w4a16_gemm(o.w4a16_gemm(X, *_l(d1, w1.g_idx), round_fp16=False),
                       *_l(d2, w2.g_idx), round_fp16=False)
    for tp in tps:
        n = N1 // tp
        parts = []
        for r in range(tp):
            _, y2 = o.mlp_actorder_rank(X, o.column_shard(d1, r, tp), w1.g_idx,
                                        o.row_shard(d2, r, tp, G, keep_all_groups=True),
                                        w2.g_idx[r * n:(r + 1) * n], y1_fp16=False, round_y2=False)
            parts.append(y2)
        tot = o.all_reduce_sum(parts, round_fp16=False)
        assert np.max(np.abs(tot - ref)) <= 1e-12 * np.max(np.abs(ref)), tp


def pin_alg2_equals_alg3(o, seed=11):
    """P9: Alg. 2 (AllGather, Y1[:, P2], CHUNK) and Alg. 3 (P2 folded into
    W1's columns) compute the same per-column dot products; in the oracle the
    fp16 results agree bit for bit at every TP degree."""
    K1, N1, N2, G = 128, 256, 64, 32
    w1, w2, d1, d2, X = _mlp_case(K1, N1, N2, G, seed)
    P1, _ = o.reorder(w1.g_idx)
    P2, _ = o.reorder(w2.g_idx)
    w1o = o.permute_rows(d1, P1)
    w2o = o.permute_rows(d2, P2)
    w1f, w2f = o.fold(d1, d2, P1, P2)
    assert np.array_equal(w2f["qweight"], w2o["qweight"])
    for tp in (1, 2, 4):
        y_naive, parts_naive = o.mlp_naive_algorithm(X, P1, P2, w1o, w2o, G, tp)
        y_aware, parts_aware = o.mlp_tp_aware(X, P1, w1f, w2f, G, tp)
        for a, b in zip(parts_naive, parts_aware):
            assert np.array_equal(a, b), tp
        assert np.array_equal(y_naive, y_aware)


def pin_fold_elementwise(o, seed=12):
    """W1[P1, P2] element by element against the codes of W1, and the
    metadata columns against P2 (brute force over a tiny layer)."""
    K1, N1, N2, G = 32, 16, 8, 8
    w1, w2, d1, d2, X = _mlp_case(K1, N1, N2, G, seed)
    P1 = np.random.default_rng(seed).permutation(K1)
    P2 = np.random.default_rng(seed + 1).permutation(N1)
    w1f, w2f = o.fold(d1, d2, P1, P2)
    qa = w1.qweight.view(np.uint32)
    qb = w1f["qweight"].view(np.uint32)
    for j in range(K1):
        for c in range(N1):
            assert nibble_by_hex(int(qb[j // 8, c]), j % 8) == \
                nibble_by_hex(int(qa[P1[j] // 8, P2[c]]), P1[j] % 8)
    za = w1.qzeros.view(np.uint32)
    zb = w1f["qzeros"].view(np.uint32)
    for g in range(K1 // G):
        for c in range(N1):
            assert w1f["scales"][g, c] == w1.scales[g, P2[c]]
            assert nibble_by_hex(int(zb[g, c // 8]), c % 8) == nibble_by_hex(int(za[g, P2[c] // 8]), P2[c] % 8)
    q2a = w2.qweight.view(np.uint32)
    q2b = w2f["qweight"].view(np.uint32)
    for j in range(N1):
        for n in range(N2):
            assert nibble_by_hex(int(q2b[j // 8, n]), j % 8) == nibble_by_hex(int(q2a[P2[j] // 8, n]), P2[j] % 8)
    assert np.array_equal(w2f["scales"], w2.scales) and np.array_equal(w2f["qzeros"], w2.qzeros)


def pin_distinct_groups(o, seed=13):
    """P11: per 128-row tile, act-order rows touch about
    ng*(1 - C(K-G,T)/C(K,T)) distinct metadata rows; sorted rows touch one."""
    K, G, T = 8192, 128, 128
    rng = np.random.default_rng(seed)
    g = o.g_idx_actorder(rng.permutation(K), G)
    d = o.distinct_groups_per_tile(g, T)
    e = o.expected_distinct_groups(K, G, T)
    assert abs(d.mean() - e) < 1.0, (d.mean(), e)
    assert 55.0 < e < 56.5
    _, gs = o.reorder(g)
    assert np.all(o.distinct_groups_per_tile(gs, T) == 1)



# ------------------------------------------------ full-size checkers ---
# The GPU tests at full size cannot build W1[P1, P2] on the host in reasonable
# time, so their expected values come from helpers that read the unpermuted
# global layers (mlp_rank_from_global, gated_rank_from_global, fold_sample).
# These pins tie each helper to the step-by-step construction it shortcuts.

def _close(a, b, tol=1e-12):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    assert a.shape == b.shape, (a.shape, b.shape)
    assert np.max(np.abs(a - b)) <= tol * max(1e-300, np.max(np.abs(b))), np.max(np.abs(a - b))


def _glob(L):
    return L.qweight, L.scales, L.qzeros, L.g_idx


def pin_rank_from_global(o, seed=27, tps=(1, 2, 4, 8)):
    """mlp_rank_from_global against the step-by-step Alg. 3 rank (fold, then
    the column shard of W1[P1, P2] and the row shard of W2[P2], X[:, P1]) and
    against the act-order rank (Megatron shards of the unpermuted layers, W2's
    shard with its rows' global g_idx and all the metadata), for every rank
    and TP degree, in float64 to 1e-12; a subset of Y2's columns equals those
    columns of the full result; the ranks sum to the unsharded MLP; with the
    fp16 roundings on, within 2e-3 of the step-by-step rank."""
    K1, N1, N2, G = 256, 512, 128, 32
    w1, w2, d1, d2, X = _mlp_case(K1, N1, N2, G, seed)
    l1, l2 = _glob(w1), _glob(w2)
    P1, _ = o.reorder(w1.g_idx)
    P2, _ = o.reorder(w2.g_idx)
    w1f, w2f = o.fold(d1, d2, P1, P2)
    ref = o.w4a16_gemm(o.w4a16_gemm(X, *_l(d1, w1.g_idx), round_fp16=False),
                       *_l(d2, w2.g_idx), round_fp16=False)
    cols = np.array([0, 5, 77, N2 - 1])
    f64 = dict(y1_round=False, round_y2=False)
    for tp in tps:
        n = N1 // tp
        tot_o = np.zeros_like(ref)
        tot_a = np.zeros_like(ref)
        for r in range(tp):
            y1, y2 = o.mlp_rank_from_global(X, l1, l2, r, tp, True, P2=P2, **f64)
            e1, e2 = o.mlp_tp_aware_rank(X, P1, o.column_shard(w1f, r, tp), o.row_shard(w2f, r, tp, G),
                                         G, y1_fp16=False, round_y2=False)
            _close(y1, e1)
            _close(y2, e2)
            a1, a2 = o.mlp_rank_from_global(X, l1, l2, r, tp, False, P2=P2, **f64)
            f1, f2 = o.mlp_actorder_rank(X, o.column_shard(d1, r, tp), w1.g_idx,
                                         o.row_shard(d2, r, tp, G, keep_all_groups=True),
                                         w2.g_idx[r * n:(r + 1) * n], y1_fp16=False, round_y2=False)
            _close(a1, f1)
            _close(a2, f2)
            _, c2 = o.mlp_rank_from_global(X, l1, l2, r, tp, True, P2=P2, cols2=cols, **f64)
            _close(c2, y2[:, cols])
            h1, h2 = o.mlp_rank_from_global(X, l1, l2, r, tp, True, P2=P2)
            g1, g2 = o.mlp_tp_aware_rank(X, P1, o.column_shard(w1f, r, tp), o.row_shard(w2f, r, tp, G), G)
            assert h1.dtype == np.float16 and h2.dtype == np.float16
            assert o.rel_err(h1, g1) <= 2e-3 and o.rel_err(h2, g2) <= 2e-3, (tp, r)
            tot_o += y2
            tot_a += a2
        _close(tot_o, ref)
        _close(tot_a, ref)


def pin_gated_rank_from_global(o, seed=28, tps=(1, 2, 4)):
    """gated_rank_from_global against the step-by-step gated Alg. 3 rank
    (gate and up folded with W[P1, P2], down with W[P2], column and row
    shards) and against the act-order gated rank built from the pinned
    gated_y1 and GEMM on Megatron shards of the unpermuted layers, every rank,
    float64 to 1e-12; the ranks sum to the unsharded gated MLP."""
    gate, up, down, dg, du, dd, X, G = _gated_case(seed)
    lg, lu, l2 = _glob(gate), _glob(up), _glob(down)
    P1, _ = o.reorder(gate.g_idx)
    P2, _ = o.reorder(down.g_idx)
    gf, df = o.fold(dg, dd, P1, P2)
    uf, _ = o.fold(du, None, P1, P2)
    ref = o.w4a16_gemm(o.gated_y1(X, o._triple(dg), o._triple(du), gate.g_idx, round_fp16=False),
                       *o._triple(dd), down.g_idx, round_fp16=False)
    f64 = dict(y1_round=False, round_y2=False)
    N1 = gate.N
    for tp in tps:
        n = N1 // tp
        tot = np.zeros_like(ref)
        for r in range(tp):
            y1, y2 = o.gated_rank_from_global(X, lg, lu, l2, r, tp, True, P2=P2, **f64)
            e1, e2 = o.gated_mlp_tp_aware_rank(X, P1, o.column_shard(gf, r, tp), o.column_shard(uf, r, tp),
                                               o.row_shard(df, r, tp, G), G, y1_fp16=False,
                                               round_y2=False)
            _close(y1, e1)
            _close(y2, e2)
            a1, a2 = o.gated_rank_from_global(X, lg, lu, l2, r, tp, False, P2=P2, **f64)
            f1 = o.gated_y1(X, o._triple(o.column_shard(dg, r, tp)), o._triple(o.column_shard(du, r, tp)),
                            gate.g_idx, round_fp16=False)
            f2 = o.w4a16_gemm(f1, *o._triple(o.row_shard(dd, r, tp, G, keep_all_groups=True)),
                              down.g_idx[r * n:(r + 1) * n], round_fp16=False)
            _close(a1, f1)
            _close(a2, f2)
            tot += y2
        _close(tot, ref)


def pin_fold_sample(o, seed=29):
    """fold_sample (codes of W[P_row, P_col] read from the source words one
    by one) against the codes of the folded and the row-permuted layer, on
    every row and column of a tiny layer, and against the hex spelling of the
    source words on a few elements."""
    K, N, G = 64, 24, 16
    w1, _ = inputs.make_custom(K, N, 0, G, seed)
    d = dict(qweight=w1.qweight, scales=w1.scales, qzeros=w1.qzeros)
    rng = np.random.default_rng(seed)
    Pr, Pc = rng.permutation(K), rng.permutation(N)
    rows, cols = np.arange(K), np.arange(N)
    full = o.unpack_rows(o.fold(d, None, Pr, Pc)[0]["qweight"])
    assert np.array_equal(o.fold_sample(w1.qweight, Pr, Pc, rows, cols), full)
    perm_only = o.unpack_rows(o.permute_rows(d, Pr)["qweight"])
    assert np.array_equal(o.fold_sample(w1.qweight, Pr, None, rows, cols), perm_only)
    sr, sc = np.array([3, 17, 40, 63]), np.array([0, 9, 23])
    got = o.fold_sample(w1.qweight, Pr, Pc, sr, sc)
    words = w1.qweight.view(np.uint32)
    for a, r in enumerate(sr):
        for b, c in enumerate(sc):
            src_r, src_c = int(Pr[r]), int(Pc[c])
            assert got[a, b] == nibble_by_hex(int(words[src_r // 8, src_c]), src_r % 8)


# -------------------------------------------- checkpoint conventions ---

def pin_zero_offset(o, seed=30):
    """A layer whose packer stores z - 1 (zero_offset = 1): dequantizing stored
    zeros z' with the offset equals dequantizing stored zeros z' + 1 without
    it (zeros of at most 14 stored); a hand value where the offset reaches the
    zero 16 that four bits cannot store: q = 5, stored z' = 15 gives
    s (5 - 16) = -11 s; and the GEMM with the offset against a triple loop
    over hex spellings."""
    K, N, G = 32, 16, 8
    w1, _ = inputs.make_custom(K, N, 0, G, seed)
    z = o.unpack_cols(w1.qzeros)
    z14 = np.minimum(z, 14)
    a = o.dequant(w1.qweight, w1.scales, o.pack_cols(z14), w1.g_idx, zero_offset=1)
    b = o.dequant(w1.qweight, w1.scales, o.pack_cols(z14 + 1), w1.g_idx)
    assert np.array_equal(a, b)
    qw = np.zeros((1, 8), dtype=np.uint32)
    qw[0, 0] = 0x5                                # row 0, column 0: code 5
    qz = np.array([[0xF]], dtype=np.uint32)       # column 0: stored zero 15
    sc = np.full((1, 8), 0.25, dtype=np.float16)
    W = o.dequant(qw.view(np.int32), sc, qz.view(np.int32), np.zeros(8, np.int64), zero_offset=1)
    assert W[0, 0] == 0.25 * (5 - 16) and W[1, 0] == 0.25 * (0 - 16)
    M = 2
    X = inputs.random_activations(M, K, np.random.default_rng(seed))
    words, zw = w1.qweight.view(np.uint32), w1.qzeros.view(np.uint32)
    Y = o.w4a16_gemm(X, w1.qweight, w1.scales, w1.qzeros, w1.g_idx, round_fp16=False, zero_offset=1)
    for m in range(M):
        for n in range(N):
            acc = 0.0
            for k in range(K):
                g = int(w1.g_idx[k])
                q = nibble_by_hex(int(words[k // 8, n]), k % 8)
                zz = nibble_by_hex(int(zw[g, n // 8]), n % 8) + 1
                acc += float(X[m, k]) * float(w1.scales[g, n]) * (q - zz)
            assert abs(Y[m, n] - acc) <= 1e-12 * max(1.0, abs(acc)), (m, n)


def pin_partial_last_group(o, seed=31):
    """G not dividing K (K = 72, G = 32): Eq. 3 gives groups of 32, 32 and 8
    rows, which check_groups accepts (and a last group of 9 rows it rejects);
    Alg. 1 still yields Eq. 1, g_sorted[j] = floor(j / G); the ordered product
    equals the act-order product; a triple loop over hex spellings fixes the
    GEMM; the TP-aware MLP with a partial last group in both layers equals the
    unsharded act-order MLP (TP = 1), and the act-order rank sum does at
    TP = 2."""
    K1, N1, N2, G = 72, 80, 16, 32
    w1, w2 = inputs.make_custom(K1, N1, N2, G, seed)
    assert w1.scales.shape[0] == 3 and w2.scales.shape[0] == 3
    assert np.array_equal(np.bincount(w1.g_idx), [32, 32, 8])
    assert np.array_equal(np.bincount(w2.g_idx), [32, 32, 16])
    o.check_groups(w1.g_idx, G)
    bad = w1.g_idx.copy()
    bad[np.flatnonzero(bad == 1)[0]] = 2          # groups of 31, 32, 9 rows
    try:
        o.check_groups(bad, G)
        raise AssertionError("a wrong partial group accepted")
    except o.GroupIndexError:
        pass
    P, gs = o.reorder(w1.g_idx)
    assert np.array_equal(gs, np.arange(K1) // G)
    X = inputs.random_activations(3, K1, np.random.default_rng(seed))
    ref = o.w4a16_gemm(X, w1.qweight, w1.scales, w1.qzeros, w1.g_idx, round_fp16=False)
    ws = o.permute_rows(dict(qweight=w1.qweight, scales=w1.scales, qzeros=w1.qzeros), P)
    Yo = o.w4a16_gemm(X, ws["qweight"], ws["scales"], ws["qzeros"], o.g_idx_naive(K1, G), x_perm=P,
                      round_fp16=False)
    _close(Yo, ref)
    words, zw = w1.qweight.view(np.uint32), w1.qzeros.view(np.uint32)
    for m in range(3):
        for n in (0, 7, 41, 79):
            acc = 0.0
            for k in range(K1):
                g = int(w1.g_idx[k])
                q = nibble_by_hex(int(words[k // 8, n]), k % 8)
                zz = nibble_by_hex(int(zw[g, n // 8]), n % 8)
                acc += float(X[m, k]) * float(w1.scales[g, n]) * (q - zz)
            assert abs(ref[m, n] - acc) <= 1e-12 * max(1.0, abs(acc))
    d1 = dict(qweight=w1.qweight, scales=w1.scales, qzeros=w1.qzeros)
    d2 = dict(qweight=w2.qweight, scales=w2.scales, qzeros=w2.qzeros)
    mref = o.w4a16_gemm(ref, *_l(d2, w2.g_idx), round_fp16=False)
    P2, _ = o.reorder(w2.g_idx)
    w1f, w2f = o.fold(d1, d2, P, P2)
    _, y2 = o.mlp_tp_aware_rank(X, P, w1f, w2f, G, y1_fp16=False, round_y2=False)
    _close(y2, mref)
    tot = np.zeros_like(mref)
    for r in range(2):
        n = N1 // 2
        _, a2 = o.mlp_actorder_rank(X, o.column_shard(d1, r, 2), w1.g_idx,
                                    o.row_shard(d2, r, 2, G, keep_all_groups=True),
                                    w2.g_idx[r * n:(r + 1) * n], y1_fp16=False, round_y2=False)
        tot += a2
    _close(tot, mref)


def pin_unequal_groups(o, seed=32):
    """Groups of unequal size (G = 0: the grouping is g_idx alone): the
    generator's group sizes are the bincount of g_idx; check_groups accepts
    them only in the unequal mode; Alg. 1's sorted g_idx is the runs of those
    sizes in group order (closed form); the ordered product through the
    sorted g_idx equals the act-order product; the TP-aware MLP (W2's row
    shards keep every group's metadata and their rows' sorted group indices)
    sums over ranks to the unsharded MLP at TP = 1, 2 and 4."""
    K1, N1, N2, ng1, ng2 = 96, 128, 24, 7, 9
    w1 = inputs.make_unequal_layer(K1, N1, ng1, seed, layer=0)
    w2 = inputs.make_unequal_layer(N1, N2, ng2, seed, layer=1)
    sizes1 = np.bincount(w1.g_idx, minlength=ng1)
    assert sizes1.sum() == K1 and len(set(sizes1.tolist())) > 1
    o.check_groups(w1.g_idx, 0, num_groups=ng1)
    try:
        o.check_groups(w1.g_idx, K1 // ng1 // 8 * 8 or 8)
        raise AssertionError("unequal groups accepted as equal ones")
    except o.GroupIndexError:
        pass
    P1, g1s = o.reorder(w1.g_idx)
    assert np.array_equal(g1s, np.repeat(np.arange(ng1), sizes1))
    P2, g2s = o.reorder(w2.g_idx)
    X = inputs.random_activations(4, K1, np.random.default_rng(seed))
    d1 = dict(qweight=w1.qweight, scales=w1.scales, qzeros=w1.qzeros)
    d2 = dict(qweight=w2.qweight, scales=w2.scales, qzeros=w2.qzeros)
    ref1 = o.w4a16_gemm(X, *_l(d1, w1.g_idx), round_fp16=False)
    ws = o.permute_rows(d1, P1)
    _close(o.w4a16_gemm(X, *_l(ws, g1s), x_perm=P1, round_fp16=False), ref1)
    mref = o.w4a16_gemm(ref1, *_l(d2, w2.g_idx), round_fp16=False)
    w1f, w2f = o.fold(d1, d2, P1, P2)
    for tp in (1, 2, 4):
        n = N1 // tp
        tot = np.zeros_like(mref)
        for r in range(tp):
            sh2 = o.row_shard(w2f, r, tp, 0, keep_all_groups=True)
            _, y2 = o.mlp_tp_aware_rank(X, P1, o.column_shard(w1f, r, tp), sh2, 0, y1_fp16=False,
                                        round_y2=False, g1=g1s, g2=g2s[r * n:(r + 1) * n])
            tot += y2
        _close(tot, mref)

# ------------------------------------------------------------- bfloat16 ---

def pin_bf16_rounding(o, seed=21):
    """to_bf16 against torch's CPU float32 -> bfloat16 cast (a library
    routine) over a wide exponent range, and against hand-worked values:
    ties go to the even significand, and a float64 value just above a tie
    rounds up although its float32 rounding sits on the tie (one rounding,
    not two)."""
    import torch
    rng = np.random.default_rng(seed)
    x = (rng.standard_normal(4096) * np.exp2(rng.integers(-60, 60, 4096))).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(o.to_bf16(x).view(np.uint32), ref.view(np.uint32))
    cases = [
        (1.0 + 2.0 ** -8, 1.0),                        # tie -> even significand 1.0000000
        (1.0 + 3 * 2.0 ** -8, 1.0 + 2.0 ** -6),        # tie -> even 1.0000010
        (-(1.0 + 3 * 2.0 ** -8), -(1.0 + 2.0 ** -6)),
        (255.5, 256.0),                                # 9 significant bits, tie -> 2^8
        (1.0 + 2.0 ** -8 + 2.0 ** -30, 1.0 + 2.0 ** -7),  # just above the tie
        (3.0, 3.0), (0.0, 0.0), (2.0 ** -100, 2.0 ** -100),
    ]
    for v, want in cases:
        assert float(o.to_bf16(np.array([v]))[0]) == want, (v, want)


def pin_bf16_gemm(o, seed=22):
    """The bfloat16 GEMM's output is the exact product rounded once to
    bfloat16: every value is a bfloat16 (low 16 bits of its float32 zero) and
    lies within half a unit in the last place (2^-8 relative) of the float64
    sum; an fp16 rounding would leave values bfloat16 cannot hold."""
    w1, _ = inputs.make_custom(256, 64, 0, 32, seed, scale_dtype=inputs.BF16)
    X = inputs.random_activations(5, 256, np.random.default_rng(seed), dtype=inputs.BF16)
    args = (X, w1.qweight, w1.scales, w1.qzeros, w1.g_idx)
    Y = o.w4a16_gemm(*args, dtype="bf16")
    Y64 = o.w4a16_gemm(*args, round_fp16=False)
    y = np.asarray(Y, dtype=np.float32)
    assert np.all(y.view(np.uint32) & 0xFFFF == 0)
    assert np.all(np.abs(y.astype(np.float64) - Y64) <= np.exp2(-8) * np.abs(Y64))
    assert np.max(np.abs(Y64)) > 1.0  # a non-trivial product



# ------------------------------------------------------------- gated MLP ---

def pin_silu(o, seed=23):
    """silu against scipy's logistic function (a library routine), the
    identity silu(x) - silu(-x) = x, and hand values: silu(0) = 0,
    silu(1) = 1 / (1 + e^-1), silu(x) -> x for large x and -> 0 for very
    negative x."""
    from scipy.special import expit
    x = np.random.default_rng(seed).standard_normal(1000) * 8
    assert np.allclose(o.silu(x), x * expit(x), rtol=1e-14, atol=0)
    assert np.allclose(o.silu(x) - o.silu(-x), x, rtol=1e-13, atol=1e-13)
    assert o.silu(np.array([0.0]))[0] == 0.0
    assert abs(o.silu(np.array([1.0]))[0] - 0.7310585786300049) < 1e-15
    assert abs(o.silu(np.array([40.0]))[0] - 40.0) < 1e-12
    assert abs(o.silu(np.array([-40.0]))[0]) < 1e-15


def _gated_case(seed):
    K1, N1, N2, G = 256, 512, 128, 32
    gate, down = inputs.make_custom(K1, N1, N2, G, seed)
    up, _ = inputs.make_custom(K1, N1, 0, G, seed + 1000)
    up.g_idx = gate.g_idx          # one input, one act-order permutation
    X = inputs.random_activations(6, K1, np.random.default_rng(seed))
    d = lambda w: dict(qweight=w.qweight, scales=w.scales, qzeros=w.qzeros)
    return gate, up, down, d(gate), d(up), d(down), X, G


def pin_gated_tp_aware_mlp(o, seed=24, tps=(1, 2, 4)):
    """The gated MLP under the TP-aware fold: P2 folded into the columns of
    both gate and up (W[P1, P2]) and into the rows of down; the sum over ranks
    equals the unsharded act-order gated MLP (float64), for each TP degree;
    with fp16 activations within 2e-3. The elementwise silu(gate) * up
    commutes with the column permutation, which is why the fold carries over."""
    gate, up, down, dg, du, dd, X, G = _gated_case(seed)
    ref64 = o.w4a16_gemm(o.gated_y1(X, o._triple(dg), o._triple(du), gate.g_idx, round_fp16=False),
                         *o._triple(dd), down.g_idx, round_fp16=False)
    P1, _ = o.reorder(gate.g_idx)
    P2, _ = o.reorder(down.g_idx)
    gf, df = o.fold(dg, dd, P1, P2)
    uf, _ = o.fold(du, None, P1, P2)
    for tp in tps:
        parts, parts16 = [], []
        for r in range(tp):
            sg, su = o.column_shard(gf, r, tp), o.column_shard(uf, r, tp)
            sd = o.row_shard(df, r, tp, G)
            _, y2 = o.gated_mlp_tp_aware_rank(X, P1, sg, su, sd, G, y1_fp16=False, round_y2=False)
            parts.append(y2)
            parts16.append(o.gated_mlp_tp_aware_rank(X, P1, sg, su, sd, G)[1])
        tot = o.all_reduce_sum(parts, round_fp16=False)
        assert np.max(np.abs(tot - ref64)) <= 1e-12 * np.max(np.abs(ref64)), tp
        ref16 = o.gated_mlp_reference(X, dg, du, gate.g_idx, dd, down.g_idx)
        assert o.rel_err(o.all_reduce_sum(parts16), ref16) <= 2e-3, tp


def pin_gated_special_cases(o, seed=25):
    """q == z in W_up (up = 0) gives Y1 = 0 whatever the gate; q == z in
    W_gate (gate = 0, silu(0) = 0) gives Y1 = 0 whatever up."""
    gate, up, down, dg, du, dd, X, G = _gated_case(seed)
    for which in ("up", "gate"):
        dz = dict(dg if which == "gate" else du)
        z = o.unpack_cols(dz["qzeros"])
        dz["qweight"] = o.pack_rows(z[gate.g_idx])   # every code equals its zero
        a, b = (dz, du) if which == "gate" else (dg, dz)
        y1 = o.gated_y1(X, o._triple(a), o._triple(b), gate.g_idx, round_fp16=False)
        assert np.all(y1 == 0), which



def pin_gated_bruteforce(o, seed=26):
    """gated_y1 against scalar loops on a tiny layer pair: every weight read
    off the hex spelling of its word, both dot products summed term by term,
    silu from math.exp, so a swap of gate and up, or a dropped zero, shows."""
    import math
    K, N, G, M = 16, 8, 8, 2
    gate, _ = inputs.make_custom(K, N, 0, G, seed)
    up, _ = inputs.make_custom(K, N, 0, G, seed + 7)
    up.g_idx = gate.g_idx
    X = inputs.random_activations(M, K, np.random.default_rng(seed))

    def w(layer, k, n):
        q = nibble_by_hex(int(layer.qweight.view(np.uint32)[k // 8, n]), k % 8)
        g = int(gate.g_idx[k])
        z = nibble_by_hex(int(layer.qzeros.view(np.uint32)[g, n // 8]), n % 8)
        return float(layer.scales[g, n]) * (q - z)

    d = lambda L: (L.qweight, L.scales, L.qzeros)
    y = o.gated_y1(X, d(gate), d(up), gate.g_idx, round_fp16=False)
    for m in range(M):
        for n in range(N):
            yg = sum(float(X[m, k]) * w(gate, k, n) for k in range(K))
            yu = sum(float(X[m, k]) * w(up, k, n) for k in range(K))
            want = yg / (1.0 + math.exp(-yg)) * yu
            assert abs(y[m, n] - want) <= 1e-12 * max(1.0, abs(want)), (m, n)


ALL_PINS = [
    pin_unpack_bruteforce, pin_pack_roundtrip, pin_golden_gemm_codes, pin_worked_reorder,
    pin_reorder_closed_form, pin_identity_phi, pin_check_groups, pin_golden_gemm,
    pin_gemm_bruteforce, pin_one_hot_rows, pin_special_cases, pin_ordered_equals_actorder,
    pin_tp_aware_mlp, pin_actorder_shard_mlp, pin_alg2_equals_alg3, pin_fold_elementwise,
    pin_distinct_groups, pin_bf16_rounding, pin_bf16_gemm, pin_silu,
    pin_gated_tp_aware_mlp, pin_gated_special_cases, pin_gated_bruteforce,
    pin_rank_from_global, pin_gated_rank_from_global, pin_fold_sample,
    pin_zero_offset, pin_partial_last_group, pin_unequal_groups,
]
