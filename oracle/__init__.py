"""fp64 CPU oracle (test infrastructure only; see comfuse_oracle)."""
from .comfuse_oracle import *  # noqa: F401,F403
