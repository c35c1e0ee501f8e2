"""CPU oracle of the AGN hot path: test infrastructure only (see agn_oracle)."""
from .agn_oracle import *  # noqa: F401,F403
from .efficiency import *  # noqa: F401,F403
