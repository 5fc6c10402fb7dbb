"""Plain float64 CPU oracle for progressive approximate-LSTM inference.

TEST INFRASTRUCTURE ONLY.  Nothing in the product package may import, call,
link or execute this package: only ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the
HIP path (no kernels, headers, helpers or constant tables); the only module
both sides use is the seeded input generator, which holds none of the method's
arithmetic.

What it computes follows "Approximate LSTMs for Time-Constrained Inference"
(Rizakis et al., arXiv 1905.00689):

* ``lstm``        -- the exact LSTM cell and recurrence (Sec. II, Fig. 1), and
                     the dense baseline cut after a number of rows per gate
                     (the row-tile anytime baseline of Sec. VI-B).
* ``factorise``   -- the hybrid residual rank-1 SVD + magnitude pruning that
                     turns each augmented gate matrix into an ordered list of
                     refinement terms (Sec. III, Eq. (1) and the residual
                     definition that follows it).
* ``progressive`` -- the progressive gate evaluation under a refinement budget
                     K (Eq. (1)) followed by the cell update, per requested
                     level or per-timestep schedule.
* ``opcount``     -- the per-gate operation counts of Sec. III and Sec. VI-B
                     and the Table I efficiency arithmetic.

Every function is pinned by ``tests/test_oracle_pins.py`` against library
routines, closed forms, invariants, brute force and the paper's printed
numbers (no function here is "parity unpinned").
"""

from .lstm import sigmoid, cell_update, exact_lstm, row_tile_lstm
from .factorise import Factors, nz_from_ratio, top_triplet, magnitude_mask, prepare, round_bf16
from .progressive import run, run_schedule, reconstruct, dense_pruned_v
from .opcount import gate_ops_progressive, gate_ops_dense, table1_efficiency

__all__ = [
    "sigmoid", "cell_update", "exact_lstm", "row_tile_lstm",
    "Factors", "nz_from_ratio", "top_triplet", "magnitude_mask", "prepare", "round_bf16",
    "run", "run_schedule", "reconstruct", "dense_pruned_v",
    "gate_ops_progressive", "gate_ops_dense", "table1_efficiency",
]
