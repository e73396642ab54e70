"""CPU checks of the test-side device-layout construction against the
header's worked definition (so the GPU repack test compares with something
pinned)."""

import numpy as np

from oracle import qmatmul_oracle as O
from tests.helpers import device_layout


def test_q4_device_chunk_by_hand():
    q = np.zeros((1, 32), np.int8)
    q[0, :8] = [1, -2, 3, -4, 5, -6, 7, -8]          # k = 0..7 of dword 0
    s16 = np.array([[0x3C00]], np.uint16)
    b, s = device_layout(q, s16, O.Q4)
    d0 = int.from_bytes(b[:4].tobytes(), "little")
    # slots t=0..3 hold k=0,2,4,6 -> u = 9,11,13,15; t=4..7 hold k=1,3,5,7 -> u = 6,4,2,0
    want = 0
    for t, u in enumerate([9, 11, 13, 15, 6, 4, 2, 0]):
        want |= u << (4 * t)
    assert d0 == want
    # rows 1..63 of the panel are padding: zero bytes
    assert not b[16:].any() and b.size == 64 * 16
    assert s[0] == 0x3C00 and not s[1:].any()


def test_q8_device_halves_by_hand():
    q = np.zeros((2, 64), np.int8)
    q[1, 16] = -127            # row 1, group 0, half 1, byte 0
    q[1, 32 + 15] = 5          # row 1, group 1, half 0, byte 15
    s16 = np.ones((2, 2), np.uint16)
    b, s = device_layout(q, s16, O.Q8)
    G = 2
    def off(n, g, h, byte):
        return ((0 * G + g) * 2 + h) * 1024 + n * 16 + byte
    assert b[off(1, 0, 1, 0)] == 1
    assert b[off(1, 1, 0, 15)] == 133
    assert b[off(0, 0, 0, 0)] == 128
    assert b[off(5, 0, 0, 0)] == 0          # padding row
    assert s[(0 * G + 1) * 64 + 1] == 1
