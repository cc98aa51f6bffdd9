"""Benchmark of the fused W-way aggregation + AdamW step (work in progress)."""

# Section III-D, step 5 of the backward stage (and Table III): per element
# the parameter server's Adam reads a 2-byte gradient and 12 bytes of model
# state (fp32 master weight, m, v) and writes the 12 bytes back plus a
# 2-byte parameter copy, doing 17 floating-point operations.
ADAM_CORE_BYTES = {"grad_in": 2, "states_in": 12, "states_out": 12,
                   "param_copy_out": 2}
ADAM_FLOPS_PER_ELEMENT = 17
