"""CPU float64 oracle (test infrastructure only; see oracle.naive)."""
from .naive import *  # noqa: F401,F403
from .naive import __all__  # noqa: F401
from . import decode  # noqa: F401,E402  (decode step; test infrastructure only)
