"""CPU oracle of the EAT MoE-layer forward.  Test infrastructure only: the
product path never imports it."""
from .eat_oracle import *  # noqa: F401,F403
