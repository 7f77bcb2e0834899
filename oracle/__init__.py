"""Scalar CPU oracle for HOBFLOPS arithmetic (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg use this
package; the GPU library never imports, links or calls it.
"""
from .oracle import *  # noqa: F401,F403
