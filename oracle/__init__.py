"""CPU oracle (float64 numpy) of the BK clipping path -- test infrastructure only.

Imported by tests/, by the smoke check and by the benchmark's CPU-baseline leg;
never by the library.
"""
from .bk_oracle import *  # noqa: F401,F403
from .bk_oracle import __all__  # noqa: F401
