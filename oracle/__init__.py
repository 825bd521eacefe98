"""CPU oracle (test infrastructure only): see ``gsc_oracle``."""
from .gsc_oracle import *  # noqa: F401,F403
