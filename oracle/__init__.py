"""CPU oracle for the Matryoshka multi-head LM loss (test infrastructure only).

This package is the plain, slow, obviously-correct statement of what the GPU
path computes. It exists to check the GPU path, and nothing in the product
path may import it: only the test suite, the smoke check and the CPU leg of
the benchmark use it.

Modules
-------
``mls_oracle``  vectorised float64 numpy implementation (forward losses,
                per-row statistics, the exact gradient, loss coefficients).
``junction``    the inter-model junction of eq. (1), forward and backward.
``bruteforce``  the same definitions written as pure-Python loops with
                ``math.fsum``; only usable on tiny shapes. It shares no code
                with ``mls_oracle`` and exists to pin it.
"""

from .mls_oracle import (  # noqa: F401
    IGNORE_INDEX,
    coeffs,
    forward,
    backward,
    objective,
    per_row,
    grad_h_rows,
    grad_W_rows,
    n_valid,
    teacher_logq,
    diagnostics,
)
from . import junction  # noqa: F401,E402
