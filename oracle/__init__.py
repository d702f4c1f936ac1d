"""Float64 CPU oracle (test infrastructure only; see taylor.py)."""
from .taylor import *  # noqa: F401,F403
from .metrics import *  # noqa: F401,F403
