"""CPU oracle of the sparse basis convolution.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU-baseline
leg of the benchmark import this package; the product library and its Python
binding never do, and this package imports nothing of theirs.  It is written
from the paper's definitions (Section 3: the finite convolution sum, the
basis-function kernel, ball and backwards-in-time neighbourhoods) and is
deliberately plain: float64 arithmetic, exhaustive enumeration, library
primitives (numpy matmul, sorting) only as whole steps.

Pins: every function here is checked, in the CPU test suite, against results
fixed by the paper or by mathematics (hand-computed cases, a KD-tree library
search, invariants, the dense-matrix form, the textbook 2D convolution, the
deployment recursion of the event convolution, adjoint identities and finite
differences).  No function is left unpinned.
"""
from . import basis, conv, sampling
from ._native import (block_order, build, csr_transpose, events_csc, events_csr, max_threads,
                      points_csr, points_d2)

__all__ = ["basis", "conv", "sampling", "block_order", "build", "csr_transpose", "events_csc",
           "events_csr", "max_threads",
           "points_csr", "points_d2"]
