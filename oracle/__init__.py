"""CPU oracle of the denoise loop (test infrastructure; see vla_oracle)."""
from .vla_oracle import *  # noqa: F401,F403
