"""CPU oracle of the ASP linear layer: test infrastructure only.

Only the tests, the smoke check and the benchmark's CPU-baseline leg import
this package.  It never imports the GPU library and shares no code with it.
"""
from .qwam_oracle import *  # noqa: F401,F403
from . import qwam_oracle  # noqa: F401
