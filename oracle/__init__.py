"""Plain CPU oracle for the RNS-CKKS projection path.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg import this package.  It shares no code with the HIP library
and never imports it.  See ``oracle/ckks.py`` for the scheme and
``oracle/ckks_oracle.c`` for the inner loops.
"""
from .ckks import *  # noqa: F401,F403
