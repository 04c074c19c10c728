"""The oracle: a plain fp64 CPU evaluation of composed modules.

TEST INFRASTRUCTURE ONLY.  Only tests, the package smoke check and the
benchmark's CPU-baseline leg may import it.  It shares no code with the HIP
library and imports nothing from the product package: modules arrive as the
plain dicts described in mko.py and inputs as raw storage arrays.
"""
from .mko import build, library, plan, run, round_bf16, round_f32, gelu_erf, gelu_tanh  # noqa: F401
