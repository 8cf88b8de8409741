"""Serial CPU oracle for the WFST decoder -- TEST INFRASTRUCTURE ONLY.

Only the test suite, the smoke check and the CPU-baseline leg of the
benchmark may import this package.  It shares no code with the GPU decoder.
"""
from .oracle import build, decode, validate_graph, OracleResult, ORACLE_OK, ORACLE_EINVAL, \
    ORACLE_ENOPATH  # noqa: F401
