"""fp64 CPU oracle (test infrastructure only; never on the product path)."""

from . import acache_oracle
from .acache_oracle import *  # noqa: F401,F403
