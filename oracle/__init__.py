"""fp64 CPU oracle for the Gaunt Tensor Product (test infrastructure only)."""
from .gtp_oracle import *  # noqa: F401,F403
