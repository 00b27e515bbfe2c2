"""CPU oracle (test infrastructure only; see erase_oracle.py, embed_oracle.py and transformer_oracle.py)."""
from .erase_oracle import *  # noqa: F401,F403
from .erase_oracle import total_loss  # noqa: F401
from . import transformer_oracle  # noqa: F401
from .embed_oracle import embed_bags, embed_bags_backward  # noqa: F401
