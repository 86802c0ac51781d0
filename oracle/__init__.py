"""Reference oracle for the learner-update hot path: plain, slow, obviously correct numpy.

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import, call or execute this
package; only the test suite, the smoke check and the benchmark's CPU-baseline leg do. It
shares no code with the HIP library (no kernels, headers, layouts or helpers): the two meet
only through the seeded inputs of the ``synth`` package.

Every function follows the paper's definition in the paper's order and cites the passage it
follows (sections, equations, Algorithm 1 and the Appendix B tables of Huang et al., "Cleanba:
A Reproducible and Efficient Distributed Reinforcement Learning Platform"). Where the paper
only names a method (IMPALA's ResNet, GAE, V-trace, Adam), the standard published definition
is written out and the reading is recorded in the design notes.

Arithmetic is float64 by default. ``prec="fp32"`` runs in float32 and ``prec="bf16"`` emulates
a bf16 matrix-core path: every GEMM operand and every stored activation is rounded to bf16
(round to nearest even) while sums stay in float32.

Parity status: every function here is pinned by a CPU test against an independent fact
(finite differences, closed forms, brute force, the paper's worked example); the bf16
emulation mode is "parity unpinned" against the paper, which fixes no precision.
"""
from . import net, targets, losses, optim, learner, cfg  # noqa: F401
