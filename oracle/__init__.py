"""CPU oracle for the CIS token loss, its operator family and the decoupled PPO-clip path
(test infrastructure only; see ``oracle.cis`` and ``oracle.ops``)."""
from .cis import *  # noqa: F401,F403
from .ops import *  # noqa: F401,F403
