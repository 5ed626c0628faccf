"""fp64 CPU oracle (test infrastructure only: tests, smoke check, bench CPU baseline)."""
from .psattn_oracle import *  # noqa: F401,F403
