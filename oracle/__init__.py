"""CPU oracle for the CIS token loss, its operator family, the decoupled PPO-clip path and the
LM-head form (test infrastructure only; see ``oracle.cis``, ``oracle.ops``, ``oracle.lmhead``)."""
from .cis import *  # noqa: F401,F403
from .ops import *  # noqa: F401,F403
from .lmhead import *  # noqa: F401,F403
