"""CPU oracle for the DeLS-Spec drafting path (test infrastructure only; see dels_oracle)."""
from .dels_oracle import *  # noqa: F401,F403
