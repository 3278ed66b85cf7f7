"""CPU oracle for SparDL's per-worker sparse synchronisation (d = 1).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, calls or links
this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may use it.  It shares no code with the
HIP library (no common helpers, tables or constants); the two meet only at the
seeded input generator, which holds none of the method's arithmetic.

The oracle is plain numpy in fp32, because the method's values are fp32
gradients and every arithmetic step on them is a single fp32 addition.
"""

from .spardl_oracle import (  # noqa: F401
    block_bounds,
    srs_partition_bags,
    srs_schedule,
    magnitude_key,
    top_k,
    index_sum,
    merge_and_resparsify,
    residual_add,
    local_sparsify,
    spar_reduce_scatter,
    allgather_densify,
    global_residual_collect,
    spardl_step,
    SparDLStepResult,
)
