"""CPU oracle of the BRISK-DLM decoding hot path (test infrastructure only)."""
from .brisk_oracle import *  # noqa: F401,F403
from .brisk_oracle import __all__  # noqa: F401
