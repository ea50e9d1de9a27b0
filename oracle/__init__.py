"""fp64 CPU oracle for packed variable-length attention (forward and gradient).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the library.  It computes the plain
definition of Eq. (2) (section 3) and its calculus gradient; see
oracle/attention.py for the readings taken where the paper is silent.
"""
from .attention import (forward, backward, rows_forward_backward, cols_backward,  # noqa: F401
                        head_rows, key_window_backward, segments)
