"""The tests' decoder of the tiled qweight layout (tests/tiled_codec.py)
against the layout as include/tpdq.h states it, walked lane by lane."""
import numpy as np

from oracle import tpdq_oracle as o
from paper_2402_04925_amd import inputs
from tests import tiled_codec as tc


def test_tiled_layout_lane_walk():
    """For K = 256, N = 32 and random codes q[k][n], the word a lane finds at
    tiled[t][256 b + 4 l + u] covers rows 8 (4 (4 b + u) + l // 16) .. +7 of
    column 16 t + l % 16, and the code of row 8 r + i sits at bits
    4 (i // 2) + 16 (i % 2); so the 16-bit masks the unpack uses
    (0x000F000F and 0x00F000F0, on the word and on the word >> 8) pick two
    consecutive rows each, low half first."""
    K, N = 256, 32
    q = np.random.default_rng(5).integers(0, 16, size=(K, N))
    qt = tc.tile(o.pack_rows(q)).view(np.uint32)
    assert qt.shape == (2, 512)
    for t in range(2):
        for b in range(2):
            for lane in range(64):
                for u in range(4):
                    r = 4 * (4 * b + u) + lane // 16
                    col = 16 * t + lane % 16
                    w = int(qt[t, 256 * b + 4 * lane + u])
                    for i in range(8):
                        assert (w >> (4 * (i // 2) + 16 * (i % 2))) & 0xF == q[8 * r + i, col]
                    pairs = [(w & 0x000F000F), (w & 0x00F000F0) >> 4,
                             ((w >> 8) & 0x000F000F), ((w >> 8) & 0x00F000F0) >> 4]
                    for p_, v in enumerate(pairs):
                        assert v & 0xF == q[8 * r + 2 * p_, col]
                        assert (v >> 16) & 0xF == q[8 * r + 2 * p_ + 1, col]
    assert np.array_equal(tc.untile(qt, K, N), o.pack_rows(q))


def test_tiled_ragged_roundtrip():
    """K % 128 != 0 and N % 16 != 0: the round trip is the identity and every
    word the layout does not use is zero."""
    w1, _ = inputs.make_custom(160, 24, 0, 32, 14)
    qt2 = tc.tile(w1.qweight)
    assert qt2.shape == (2, 512)
    assert np.array_equal(tc.untile(qt2, 160, 24), w1.qweight)
    used = np.zeros(qt2.shape, bool)
    r = np.arange(20)[:, None]
    c = np.arange(24)[None, :]
    used[c // 16, 256 * ((r // 4) // 4) + 4 * (16 * (r % 4) + c % 16) + (r // 4) % 4] = True
    assert np.all(qt2.view(np.uint32)[~used] == 0)
    assert tc.tiled_ld(160) == 512 and tc.tiled_ld(128) == 256
