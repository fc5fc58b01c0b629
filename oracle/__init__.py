"""Plain float64 CPU oracle for the Ball Sparse Attention (BSA) layer.

TEST INFRASTRUCTURE ONLY. Nothing on the product path imports, links or calls this
package: only the tests, the package smoke check and the benchmark's CPU-baseline leg do.
It shares no code with the HIP library (no kernels, headers, helpers, constants or table
generators); the only thing both sides consume is the seeded input generator in
``workloads``, which holds none of the method's arithmetic.

The oracle follows the paper (arXiv 2506.12541, "Ball Sparse Attention") step by step:
ball tree ordering (Section 2.1, Ball Tree Attention, after Erwin), ball attention (Eq. 3),
MLP block compression and compressed attention (Eq. 5), group-pooled importance scores and
shared top-k block selection (Eq. 6, 7, 10-12), selection attention (Eq. 8), and the
sigmoid-gated sum of the three branches (Eq. 9), plus the analytic backward pass.
Readings where the paper is silent are listed in the module docstrings of ``tree`` and
``bsa``.
"""
from .tree import build_ball_tree, permute_rows  # noqa: F401
from .bsa import Params, forward, backward  # noqa: F401
