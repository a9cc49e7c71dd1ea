"""CPU oracle of the GBA push-step: test infrastructure, never the product
path.  Only the tests, the smoke check and the benchmark's CPU-baseline leg
import it."""
from .gba_oracle import *  # noqa: F401,F403
from . import gba_oracle  # noqa: F401
