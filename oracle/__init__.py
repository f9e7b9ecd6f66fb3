"""CPU oracle of the ArborKV hot path: test infrastructure only (see arbor_oracle)."""
from .arbor_oracle import *  # noqa: F401,F403
from . import arbor_oracle  # noqa: F401
