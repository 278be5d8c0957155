"""Shapes that take every launch plan of the grouped FFN path (batch >= 2).

A plan is (16-token tiles per pass, K splits of the gate/up projection, K splits of the
down projection), as apex_moe_ffn_plan reports it.  The GPU parity test runs each shape
against the oracle; a CPU test checks that each shape still takes its plan, so a change
of the planning rule cannot drop a path from the parity tests unnoticed.
"""

# Every launch plan of the grouped path in every weight format: (token tiles per pass,
# gate/up K splits, down K splits), with ragged d (partial row tiles) and ragged I (a
# partial last K block).  Each case first checks that the shape still takes its plan.
PLAN_CASES = [
    # (weights, B, d, I, E, plan)
    ("bf16", 5, 72, 536, 3, (1, 1, 1)), ("bf16", 5, 72, 2072, 3, (1, 1, 2)),
    ("bf16", 5, 648, 536, 3, (1, 2, 1)), ("bf16", 5, 648, 2072, 3, (1, 2, 2)),
    ("bf16", 26, 72, 536, 3, (2, 1, 1)), ("bf16", 26, 72, 2072, 3, (2, 1, 2)),
    ("bf16", 26, 648, 536, 3, (2, 2, 1)), ("bf16", 26, 648, 2072, 3, (2, 2, 2)),
    ("bf16", 50, 72, 536, 3, (4, 1, 1)), ("bf16", 50, 72, 2072, 3, (4, 1, 2)),
    ("bf16", 50, 648, 536, 3, (4, 2, 1)), ("bf16", 50, 648, 2072, 3, (4, 2, 2)),
    ("fp8", 5, 144, 560, 3, (1, 1, 1)), ("fp8", 5, 144, 3888, 3, (1, 1, 2)),
    ("fp8", 5, 1296, 560, 3, (1, 2, 1)), ("fp8", 5, 1296, 3888, 3, (1, 2, 2)),
    ("fp8", 26, 144, 560, 3, (2, 1, 1)), ("fp8", 26, 144, 2096, 3, (2, 1, 2)),
    ("fp8", 26, 656, 560, 3, (2, 2, 1)), ("fp8", 26, 656, 2096, 3, (2, 2, 2)),
    ("fp8", 50, 144, 560, 3, (4, 1, 1)), ("fp8", 50, 144, 2096, 3, (4, 1, 2)),
    ("fp8", 50, 656, 560, 3, (4, 2, 1)), ("fp8", 50, 656, 2096, 3, (4, 2, 2)),
    ("mxfp4", 5, 288, 608, 3, (1, 1, 1)), ("mxfp4", 5, 288, 7776, 3, (1, 1, 2)),
    ("mxfp4", 5, 2592, 608, 3, (1, 2, 1)), ("mxfp4", 5, 2592, 7776, 2, (1, 2, 2)),
    ("mxfp4", 26, 288, 608, 3, (2, 1, 1)), ("mxfp4", 26, 288, 3936, 3, (2, 1, 2)),
    ("mxfp4", 26, 1312, 608, 3, (2, 2, 1)), ("mxfp4", 26, 1312, 3936, 3, (2, 2, 2)),
    ("mxfp4", 50, 288, 608, 3, (4, 1, 1)), ("mxfp4", 50, 288, 3936, 3, (4, 1, 2)),
    ("mxfp4", 50, 1312, 608, 3, (4, 2, 1)), ("mxfp4", 50, 1312, 3936, 3, (4, 2, 2)),
]
