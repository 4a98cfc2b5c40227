"""CPU oracle for the TRACE hot path: test infrastructure only (see trace_oracle)."""
from .trace_oracle import *  # noqa: F401,F403
from .trace_oracle import Config, Controller, Adam  # noqa: F401
