"""CPU oracle for the SSC / SC layers (test infrastructure only)."""
from .sscn_oracle import *  # noqa: F401,F403
