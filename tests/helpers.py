"""Shared test helpers: the comparison metric and a test-side construction of
the device layout written from its definition in include/qmatmul.h."""

import numpy as np

from oracle import qmatmul_oracle as O


def rel_err(y, ref) -> float:
    """Normwise max error relative to the largest reference entry."""
    y = np.asarray(y, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert y.shape == ref.shape, (y.shape, ref.shape)
    assert np.all(np.isfinite(y)), "non-finite output"
    scale = np.abs(ref).max()
    if scale == 0:
        return float(np.abs(y).max())
    return float(np.abs(y - ref).max() / scale)


GEMV_TOL = 2e-3    # fp32 accumulation
MFMA_TOL = 1e-2    # fp16 MFMA inputs


def _nibble_plane(u):
    """u [p, g, 64, 32] (values < 16) -> bytes [p, g, 64*16]: dword j of a
    row covers k = 8j..8j+7, nibble t holds k-offset 2t (t < 4) or
    2(t-4)+1."""
    chunks = u.reshape(*u.shape[:3], 4, 8).astype(np.uint32)              # (p, g, r, j, koff)
    slot_of_koff = [0, 4, 1, 5, 2, 6, 3, 7]
    d = np.zeros(chunks.shape[:-1], np.uint32)
    for koff in range(8):
        d |= chunks[..., koff] << np.uint32(4 * slot_of_koff[koff])
    return d.reshape(*u.shape[:2], -1).view(np.uint8)


def _crumb_plane(u):
    """u (values < 4) -> 8 bytes a row: dword j, bits 2t..2t+1 hold
    k = 16j + 2t and bits 16+2t.. hold k = 16j + 2t + 1."""
    halves = u.reshape(*u.shape[:3], 2, 16).astype(np.uint32)             # (p, g, r, j, 16)
    d = np.zeros(halves.shape[:-1], np.uint32)
    for t in range(8):
        d |= halves[..., 2 * t] << np.uint32(2 * t)
        d |= halves[..., 2 * t + 1] << np.uint32(16 + 2 * t)
    return d.reshape(*u.shape[:2], -1).view(np.uint8)


def _bit_plane(u):
    """u (values < 2) -> 4 bytes a row: bit t holds k = 2t, bit 16+t holds
    k = 2t + 1."""
    uu = u.astype(np.uint32)
    d = np.zeros(u.shape[:3], np.uint32)
    for t in range(16):
        d |= uu[..., 2 * t] << np.uint32(t)
        d |= uu[..., 2 * t + 1] << np.uint32(16 + t)
    return d.reshape(*u.shape[:2], -1).view(np.uint8)


def device_layout(q: np.ndarray, s16, fmt: int):
    """Expected DEVICE-layout bytes (uint8) and scales (uint16; None for
    F16/BF16) of one [N][K] matrix of codes q (int8; uint16 patterns for
    F16/BF16) and scale bits s16, per the header's text."""
    n, k = q.shape
    g = k // 32
    npad = (n + 63) // 64 * 64
    p = npad // 64
    if fmt in O.FLOATS:
        vv = np.zeros((npad, k), np.uint16)
        vv[:n] = q
        quarters = vv.reshape(p, 64, g, 4, 8).transpose(0, 2, 3, 1, 4)     # (p, g, j, r, 8)
        return quarters.reshape(-1).view(np.uint8).copy(), None
    qq = np.zeros((npad, k), np.int16)
    qq[:n] = q
    ss = np.zeros((npad, g), np.uint16)
    ss[:n] = s16
    scales = ss.reshape(p, 64, g).transpose(0, 2, 1).reshape(-1)          # (p, g, r)
    if fmt in (O.Q2, O.Q3, O.Q5, O.Q6):
        b = O.BITS[fmt]
        u = (qq + (1 << (b - 1))).astype(np.uint32)
        u[n:] = 0
        u = u.reshape(p, 64, g, 32).transpose(0, 2, 1, 3)                 # (p, g, r, k)
        if fmt == O.Q2:
            planes = [_crumb_plane(u)]
        elif fmt == O.Q3:
            planes = [_crumb_plane(u & 3), _bit_plane(u >> 2)]
        elif fmt == O.Q5:
            planes = [_nibble_plane(u & 15), _bit_plane(u >> 4)]
        else:
            planes = [_nibble_plane(u & 15), _crumb_plane(u >> 4)]
        return np.concatenate(planes, axis=2).reshape(-1).copy(), scales
    if fmt == O.Q4:
        u = (qq + 8).astype(np.uint32)                                       # offset binary
        if n < npad:
            u[n:] = 0
        chunks = u.reshape(p, 64, g, 4, 8).transpose(0, 2, 1, 3, 4)          # (p, g, r, j, koff)
        slot_of_koff = [0, 4, 1, 5, 2, 6, 3, 7]                              # nibble slot per k offset
        d = np.zeros(chunks.shape[:-1], np.uint32)
        for koff in range(8):
            d |= chunks[..., koff] << np.uint32(4 * slot_of_koff[koff])
        return d.reshape(-1).view(np.uint8).copy(), scales
    u = (qq + 128).astype(np.uint8)
    if n < npad:
        u[n:] = 0
    chunks = u.reshape(p, 64, g, 2, 16).transpose(0, 2, 3, 1, 4)             # (p, g, h, r, b)
    return chunks.reshape(-1).copy(), scales
