"""CPU oracle for the CIS token loss (test infrastructure only; see ``oracle.cis``)."""
from .cis import *  # noqa: F401,F403
