"""CPU oracle (test infrastructure only; see luffy_oracle)."""
from .luffy_oracle import *  # noqa: F401,F403
from . import luffy_oracle  # noqa: F401
