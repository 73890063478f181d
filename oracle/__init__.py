"""CPU oracle for SparseTem's Diff Computation -- TEST INFRASTRUCTURE ONLY.

This package is a plain, slow, obviously-correct numpy implementation of
what the diff-computation hot path computes.  It exists to check the HIP
path: only the test suite, the smoke check and the benchmark's CPU-baseline
leg may import it.  The product path never calls it and shares no code with
it; the two meet only on identical seeded inputs from ``workloads``.
"""

from .sparsetem_oracle import (ACT_NONE, ACT_RELU, ACT_SILU, OracleNet,
                               activation, conv2d_nhwc, dense_forward,
                               maxpool_nhwc, round_storage, rulebook,
                               se_apply, se_gates, window_targets)

__all__ = [
    "ACT_NONE", "ACT_RELU", "ACT_SILU", "OracleNet", "activation",
    "conv2d_nhwc", "dense_forward", "maxpool_nhwc", "round_storage",
    "rulebook", "se_apply", "se_gates", "window_targets",
]
