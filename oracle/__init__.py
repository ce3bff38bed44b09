"""Float64 CPU oracle (test infrastructure; see timebill_oracle)."""
from .timebill_oracle import *  # noqa: F401,F403
