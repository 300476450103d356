"""CPU oracle for the OmniCache cached attention layer.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this package: only the tests, the smoke check of the graft entry
point and the benchmark's CPU-baseline leg use it.  It shares no code with
the HIP library and does not import it.
"""
from .oc_oracle import *  # noqa: F401,F403
