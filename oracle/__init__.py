"""fp64 CPU oracle for the Sketch&Walk hot path.

Test infrastructure only: the tests, the smoke check and the benchmark's CPU
baseline leg may import it; the product path (the HIP library and its Python
binding) never does.
"""
from .sketchwalk_oracle import *  # noqa: F401,F403
from .sketchwalk_oracle import FORCE_BOTH, FORCE_FIRST, FORCE_LAST  # noqa: F401
