"""fp64 CPU oracle (test infrastructure only; see patchkv_oracle's header)."""
from .patchkv_oracle import *  # noqa: F401,F403
from .patchkv_oracle import __all__  # noqa: F401
