"""Plain, slow CPU oracle for the AllReduce plans of GenModel / GenTree
(arXiv 2409.04202, "Revisiting the Time Cost Model of AllReduce").

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute anything in this package: only ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the
HIP library (``paper_2409_04202_amd``) and imports nothing from it.

What it computes
----------------
An AllReduce leaves every processor with the element-wise sum of all
processors' data (Section 1; Section 2.1 defines a *plan* as an ordering of
data-movement and reduce steps).  For int32 that result is unique.  For
floating point every association order is a correct AllReduce, and a plan
fixes one order; the oracle therefore expands each plan from the paper's text
(``plans``), independently of the library, and executes its steps phase by
phase in that fixed order (``execute``).

Precision: the paper computes on ``float`` (Section 3, experimental
settings), so the fp32 path folds in IEEE fp32 (numpy float32 adds, round to
nearest even).  bf16 buffers are widened to fp32, folded in fp32 and rounded
once per step (``bf16``).  ``model`` counts the memory operations, transfers
and rounds of a plan, i.e. the coefficients of GenModel (Section 3.3, Table 2).

Modules
-------
plans    -- Ring, RHD, co-located PS, hierarchical CPS / GenTree tree plans
gentree  -- the block placement of Algorithm 1 and the basic plan it gives
            on arbitrary (also asymmetric) trees
execute  -- phase-by-phase executor (full and sampled-index forms)
bf16     -- fp32 <-> bf16 conversion (round to nearest even)
model    -- per-plan step, byte and round counts (GenModel coefficients)
"""

from .plans import (Step, Plan, block_bounds, ring, rhd, cps, tree,
                    reduce_broadcast, make_plan)
from .execute import execute, execute_sampled, fold
from .bf16 import bf16_to_f32, f32_to_bf16
from .gentree import (server, switch, symmetric_tree, basic_placement,
                      gentree_plan, from_preorder, preorder_children)
from . import model

__all__ = [
    "Step", "Plan", "block_bounds", "ring", "rhd", "cps", "tree",
    "reduce_broadcast", "make_plan", "execute", "execute_sampled", "fold",
    "bf16_to_f32", "f32_to_bf16", "server", "switch", "symmetric_tree",
    "basic_placement", "gentree_plan", "from_preorder", "preorder_children",
    "model",
]
