"""CPU oracle (test infrastructure only): see ``catekv_oracle``."""
from .catekv_oracle import *  # noqa: F401,F403
