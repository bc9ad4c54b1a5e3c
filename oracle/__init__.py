"""CPU oracle (fp64) for the swap engine.  Test infrastructure only: used by
the tests, the package smoke check and the bench's CPU-baseline leg."""
from .forward import *  # noqa: F401,F403
