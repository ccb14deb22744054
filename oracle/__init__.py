"""CPU oracle of ReSA decoding (test infrastructure only; see resa_oracle)."""
from .resa_oracle import *  # noqa: F401,F403
from . import resa_oracle  # noqa: F401
