"""Workload definitions and seeded synthetic inputs for the FarSkip MoE block.

This package holds none of the method's arithmetic.  It defines the five
workload shapes (a tiny fp32 block pair and four bf16 layers shaped like
DeepSeek-V2-Lite, Llama-4-Scout and DeepSeek-V3 prefill/decode) and draws
their inputs from seeded generators.  Both the CPU oracle and the HIP path
consume exactly the tensors produced here.
"""

from .configs import CONFIGS, MoEConfig, get_config  # noqa: F401
from .generate import Workload, make_workload, bf16_round  # noqa: F401
