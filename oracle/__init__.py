"""CPU oracle (test infrastructure only; never part of the product path)."""
from .sllm_oracle import *  # noqa: F401,F403
