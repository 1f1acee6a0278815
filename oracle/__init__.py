"""CPU oracle for the streaming action-decode step (test infrastructure only).

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The HIP library and its Python binding never do.
"""
from .flashvla import *  # noqa: F401,F403
from . import flashvla  # noqa: F401
