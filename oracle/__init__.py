"""CPU oracle for modality-aware permutation sparse attention (MMInference).

TEST INFRASTRUCTURE ONLY. This package is a plain, slow, obviously-correct
numpy (fp64) implementation of what the sparse prefill path computes, written
step by step from the paper: estimation of the attention map from the last
queries (Algorithm 1; Appendix C.3), the Grid stride/phase search
(Algorithm 1), the Grid and modality permutations (Section 3.1-3.2,
Appendix C.4), A-shape and Vertical-Slash selections (Appendix C.3),
Q-Boundary and 2D-Boundary heads (Algorithms 2 and 3, Grid modalities
included), the static baseline patterns (Section 4.1), neighborhood
attention through a tile permutation (Appendix F), the block-sparse lift
("sparse loading, dense computation", Figure "dynamic_sparse_pipelines"),
masked softmax attention (Algorithms 5-7) and the modality-aware pattern
search (Algorithm 4).

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may
import it. It shares no code with the HIP library and never imports it.

Parity status of each function is stated in its module docstring; every
function is pinned by tests under tests/test_oracle_*.py against closed
forms, invariants, brute force or library routines, except the statement
"the sparse output approximates dense attention on real VLM activations",
which needs model weights and datasets that are not available: parity
unpinned for that claim (it is not something this package computes).
"""
from . import numerics, layout, estimate, grid, vslash, natten, plan, attention, search  # noqa: F401
