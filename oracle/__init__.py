"""Plain fp64 CPU oracle of the RoLA attention module.

TEST INFRASTRUCTURE ONLY. The test-suite, the smoke check and the benchmark's CPU-baseline leg are the
only code allowed to import it. The GPU library never imports, links or calls anything in here, and
nothing in here imports the GPU library: the oracle is an independent restatement of the paper.
"""

from .rola_oracle import *  # noqa: F401,F403
from . import rola_grad  # noqa: E402,F401  gradients for fine-tuning (torch fp64 autograd)
