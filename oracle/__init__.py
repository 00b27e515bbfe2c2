"""CPU oracle (test infrastructure only; see erase_oracle.py)."""
from .erase_oracle import *  # noqa: F401,F403
from .erase_oracle import total_loss  # noqa: F401
