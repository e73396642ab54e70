"""MI355X (gfx950) weight-only-quantised matmul: Q4/Q8 group-32 fused
dequantise+GEMV, Q4 MFMA GEMM and a top-k-routed MoE expert layer, behind
the C ABI in include/qmatmul.h (libqmatmul.so).  ``binding`` holds the thin
ctypes layer; ``inputs`` the seeded synthetic input generators; ``workloads``
the layer shapes of the benchmark workloads."""

from . import binding, inputs, workloads  # noqa: F401
from .binding import (LAYOUT_CANONICAL, LAYOUT_DEVICE, Q4_G32, Q8_G32, QmError, QWeight,  # noqa: F401
                      Routing, empty_qweight, qm_dequantise, qm_device_config, qm_last_error,
                      qm_quantise, qm_repack, qm_weight_bytes, qmatmul_gemm, qmatmul_gemv,
                      qmoe_grouped_gemm, qmoe_route, qmoe_workspace_bytes)
