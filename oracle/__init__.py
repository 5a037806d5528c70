"""CPU oracle package (test infrastructure only; see pqhsa_ref)."""
from .pqhsa_ref import *  # noqa: F401,F403
