"""CPU oracle (test infrastructure only; see fusion_oracle's docstring)."""
from .fusion_oracle import *  # noqa: F401,F403
from .fusion_oracle import bf16_round, run, run_sample, plain_forward  # noqa: F401
