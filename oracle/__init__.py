"""fp64 CPU oracle (test infrastructure only; never imported by the product path)."""
from .aal_oracle import *  # noqa: F401,F403
from .aal_oracle import __all__  # noqa: F401
