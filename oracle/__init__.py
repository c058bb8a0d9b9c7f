"""CPU oracle for the INT4 HQ-MM / LSS-MM linear operator.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this package: only the tests, the smoke check and the CPU-baseline leg
of the benchmark use it.  It shares no code with the GPU library.
"""
from .hqlss_ref import *  # noqa: F401,F403
from .philox_ref import philox4x32_10, uniforms16  # noqa: F401
