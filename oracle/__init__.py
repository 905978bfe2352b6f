"""CPU oracle for the PASK decode hot path (test infrastructure only; see
pask_oracle's module docstring)."""

from .pask_oracle import *  # noqa: F401,F403
