"""CPU oracle (test infrastructure; see ``cardan_oracle``)."""
from .cardan_oracle import *  # noqa: F401,F403
from .cardan_oracle import LAYER_KEYS  # noqa: F401
