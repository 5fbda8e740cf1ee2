"""Float64 CPU oracle (test infrastructure only; never part of the library path)."""
from .dppo_oracle import *  # noqa: F401,F403
from .dppo_oracle import (  # noqa: F401
    FLAG_BAD_ID, FLAG_BAND, FLAG_PPO, FLAG_VALID, Params, RD_MODES, SCALE_MODES,
    STAT_N_ACTIVE, STAT_N_BAD, STAT_N_BAND, STAT_N_PPO, STAT_N_VALID,
)
