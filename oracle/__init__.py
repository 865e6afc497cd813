"""CPU fp64 oracle of the MCA forward pass (test infrastructure; see mca_oracle)."""
from .mca_oracle import *  # noqa: F401,F403
