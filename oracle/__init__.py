"""CPU oracle (test infrastructure only; see ``fsdp_oracle``)."""

from .fsdp_oracle import *  # noqa: F401,F403
from .fsdp_oracle import __all__  # noqa: F401
