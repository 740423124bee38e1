"""CPU oracle for the UAD action-expert hot path.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call, link
or execute anything in this package; only the tests, the smoke check and the
CPU-baseline leg of the benchmark use it.  It shares no code with the HIP
library (``paper_2609_37772_amd``) and never imports it.
"""
from .uad_oracle import *  # noqa: F401,F403
from .uad_oracle import __all__  # noqa: F401
