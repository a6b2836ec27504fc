"""One GPU's share of a block join-agg (Einsummable's "every kernel is a join")
on AMD MI355X.  The compute path is libea.so (hand-written HIP for gfx950,
C ABI in include/ea.h); this package is its Python binding."""
from .ea import (AGG_LSE, AGG_MAX, AGG_NONE, AGG_SUM, BF16, F16, F32, JOIN_ADD, JOIN_MUL, OP_ATTENTION,
                 OP_RMSNORM, OP_SOFTMAX, OP_SWIGLU, EAError, Relation, from_dense, join_tuples, joinagg,
                 joinagg_workspace, layout_nbytes, lib, new_workspace, overlay, plan_cache_clear, plan_cache_size,
                 repartition, repartition_plan, to_dense, version)
