"""Float64 CPU oracle of the DendSN layer (test infrastructure only).

Only the test-suite, the smoke check and the benchmark's CPU-baseline leg may
import this package; the product path never does.
"""
from .dendsn_oracle import (  # noqa: F401
    PSI_IDENTITY, PSI_MEXHAT, SG_ATAN, SG_SIGMOID,
    psi, dpsi, surrogate_grad, forward, backward,
)
