"""Float64 CPU oracle (test infrastructure only; see lapsum_oracle)."""
from .lapsum_oracle import *  # noqa: F401,F403
from .lapsum_oracle import __all__  # noqa: F401
