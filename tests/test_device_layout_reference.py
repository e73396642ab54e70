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


def _dword(b, off):
    return int.from_bytes(b[off:off + 4].tobytes(), "little")


def test_q5_planes_by_hand():
    q = np.zeros((1, 32), np.int8)          # zero codes: u = 16 (nibble 0, bit 1)
    q[0, 0], q[0, 1], q[0, 2], q[0, 17] = 15, -16, 1, -1
    b, s = device_layout(q, np.array([[0x3C00]], np.uint16), O.Q5)
    assert b.size == 1280
    assert _dword(b, 0) == 0x1F             # k0 nibble 15 (slot 0), k2 nibble 1 (slot 1)
    assert _dword(b, 8) == 0x000F0000       # k17 nibble 15: dword 2, slot 4
    assert _dword(b, 1024) == 0xFEFEFFFF    # bit plane: k1 (bit 16) and k17 (bit 24) clear
    assert not b[16:1024].any() and not b[1028:].any()     # padding rows


def test_q3_planes_by_hand():
    q = np.zeros((1, 32), np.int8)          # zero codes: u = 4 (crumb 0, bit 1)
    q[0, 0], q[0, 1], q[0, 16] = 3, -4, -1
    b, _ = device_layout(q, np.array([[0x3C00]], np.uint16), O.Q3)
    assert b.size == 768
    assert _dword(b, 0) == 0x3 and _dword(b, 4) == 0x3   # crumbs of k0 and k16
    assert _dword(b, 512) == 0xFFFEFEFF     # bits: k16 (bit 8) and k1 (bit 16) clear


def test_q6_planes_by_hand():
    q = np.zeros((1, 32), np.int8)          # zero codes: u = 32 (nibble 0, crumb 2)
    q[0, 0], q[0, 1] = 31, -32
    b, _ = device_layout(q, np.array([[0x3C00]], np.uint16), O.Q6)
    assert b.size == 1536
    assert _dword(b, 0) == 0xF and not b[4:16].any()
    assert _dword(b, 1024) == 0xAAA8AAAB and _dword(b, 1028) == 0xAAAAAAAA


def test_q2_crumbs_by_hand():
    q = np.zeros((1, 32), np.int8)          # zero codes: u = 2
    q[0, 0], q[0, 1], q[0, 31] = 1, -2, -1
    b, _ = device_layout(q, np.array([[0x3C00]], np.uint16), O.Q2)
    assert b.size == 512
    assert _dword(b, 0) == 0xAAA8AAAB and _dword(b, 4) == 0x6AAAAAAA


def test_f16_quarters_by_hand():
    v = np.zeros((2, 64), np.uint16)
    v[1, 9] = 0x1234                        # row 1, group 0, quarter 1, position 1
    v[0, 32 + 31] = 0xABCD                  # row 0, group 1, quarter 3, position 7
    b, s = device_layout(v, None, O.F16)
    assert s is None and b.size == 2 * 4096
    assert int.from_bytes(b[1024 + 16 + 2:1024 + 16 + 4].tobytes(), "little") == 0x1234
    assert int.from_bytes(b[4096 + 3 * 1024 + 14:4096 + 3 * 1024 + 16].tobytes(), "little") == 0xABCD
    assert int(b.view(np.uint16).astype(np.int64).sum()) == 0x1234 + 0xABCD
