"""CPU oracle of the ResBM boundary module (test infrastructure only).

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this package; the product path never does.
"""
from .resbm_oracle import *  # noqa: F401,F403
from . import muon_oracle  # noqa: F401
from . import two_linear_oracle  # noqa: F401
from . import fusion_oracle  # noqa: F401
