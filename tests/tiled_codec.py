"""Decoder and encoder of the library's tiled qweight layout, for the tests.

The tiled layout is a storage order private to the library's decode kernels
(documented in include/tpdq.h under TPDQ_LAYOUT_TILED), not part of the
paper's arithmetic, so it lives with the tests and not in the oracle. It is
written from the header's description alone and shares no code with the HIP
sources. GPU tests use it to turn the words the library wrote back into GPTQ
words (untile) or to state the words the library must write (tile).
"""
from __future__ import annotations

import numpy as np


def tiled_ld(K: int) -> int:
    """Words per 16-column tile: 256 per 128-row block."""
    return (K + 127) // 128 * 256


def _nibble_shifts():
    """Bit position, in a tiled word, of the code of row 8 r + i: even rows in
    the low half-word, odd rows in the high one (i // 2 nibbles up)."""
    return [4 * (i // 2) + 16 * (i % 2) for i in range(8)]


def interleave_word(w: np.ndarray) -> np.ndarray:
    """GPTQ words (row 8 r + i at bits 4 i) -> the tiled nibble order."""
    w = np.asarray(w).view(np.uint32)
    out = np.zeros_like(w)
    for i, sh in enumerate(_nibble_shifts()):
        out |= ((w >> np.uint32(4 * i)) & np.uint32(0xF)) << np.uint32(sh)
    return out


def deinterleave_word(w: np.ndarray) -> np.ndarray:
    """Inverse of interleave_word."""
    w = np.asarray(w).view(np.uint32)
    out = np.zeros_like(w)
    for i, sh in enumerate(_nibble_shifts()):
        out |= ((w >> np.uint32(sh)) & np.uint32(0xF)) << np.uint32(4 * i)
    return out


def _index(K: int, N: int):
    r = np.arange(K // 8)[:, None]
    c = np.arange(N)[None, :]
    s, kq = r // 4, r % 4
    b, u = s // 4, s % 4
    t, jj = c // 16, c % 16
    return t, 256 * b + 4 * (16 * kq + jj) + u


def untile(qt: np.ndarray, K: int, N: int) -> np.ndarray:
    """GPTQ words [K/8][N] of a qweight stored in the tiled order: for tile t
    (16 columns), block b (128 rows), lane l = 16 kq + j and step u,
    tiled[t][256 b + 4 l + u] is GPTQ word [4 (4 b + u) + kq][16 t + j] with
    its codes interleaved (interleave_word)."""
    qt = np.asarray(qt).view(np.uint32)
    t, w = _index(K, N)
    return deinterleave_word(qt[t, w]).view(np.int32)


def tile(qw: np.ndarray) -> np.ndarray:
    """Inverse of untile, with zero padding past K and N."""
    qw = np.asarray(qw).view(np.uint32)
    kw, N = qw.shape
    K = kw * 8
    out = np.zeros(((N + 15) // 16, tiled_ld(K)), dtype=np.uint32)
    t, w = _index(K, N)
    out[t, w] = interleave_word(qw)
    return out.view(np.int32)
