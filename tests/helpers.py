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


def device_layout(q: np.ndarray, s16: np.ndarray, fmt: int):
    """Expected DEVICE-layout bytes (uint8) and scales (uint16) of one [N][K]
    matrix of codes q (int8) and scale bits s16, per the header's text."""
    n, k = q.shape
    g = k // 32
    npad = (n + 63) // 64 * 64
    p = npad // 64
    qq = np.zeros((npad, k), np.int16)
    qq[:n] = q
    ss = np.zeros((npad, g), np.uint16)
    ss[:n] = s16
    scales = ss.reshape(p, 64, g).transpose(0, 2, 1).reshape(-1)          # (p, g, r)
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
