"""CPU oracle of the EC2MoE hot path (test infrastructure only; see ec2moe_oracle)."""
from .ec2moe_oracle import *  # noqa: F401,F403
