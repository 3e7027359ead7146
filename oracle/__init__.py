"""CPU oracle (test infrastructure only; see ``cmsd_oracle``)."""
from .cmsd_oracle import *  # noqa: F401,F403
from .cmsd_oracle import __all__  # noqa: F401
