"""CPU oracle (test infrastructure only; the product package never imports it)."""
from .qmatmul_oracle import *  # noqa: F401,F403
from .qmatmul_oracle import GROUP, Q4, Q8, QMAX, QLO, QHI  # noqa: F401
