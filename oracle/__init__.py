"""CPU oracle for the ternary x int8 mpGEMM (test infrastructure only; never on the product path)."""
from .bitnet_oracle import *  # noqa: F401,F403
