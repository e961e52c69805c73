"""CPU oracle for SWAN (test infrastructure only; see swan_oracle.py)."""
from .swan_oracle import *  # noqa: F401,F403
