"""CPU oracle (test infrastructure only): see polyq_oracle.py."""
from .polyq_oracle import *  # noqa: F401,F403
from .polyq_oracle import (block_table, num_groups, group_size, average_bits, code_bits, dequantize,  # noqa
                           permute_activations, linear, linear_scalar, check_tolerance,
                           effective_weight_bytes)
