"""CPU oracle of the QCFuse fusion step (test infrastructure only).

Only the tests, the graft entry point's smoke check and the benchmark's
CPU-baseline leg may import this package.  See ``oracle.qcfuse``.
"""
from .qcfuse import *  # noqa: F401,F403
from .qcfuse import __all__  # noqa: F401
