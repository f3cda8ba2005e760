"""CPU oracle for BF1 attention: test infrastructure only (see bf1_oracle)."""

from .bf1_oracle import *  # noqa: F401,F403
from .bf1_oracle import __all__  # noqa: F401
