"""CPU oracle (test infrastructure only; never imported by the product path)."""
from .backbone import *  # noqa: F401,F403
