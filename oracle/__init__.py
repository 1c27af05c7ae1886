"""CPU fp64 oracle for the per-GPU hot path of Nested Sequence Parallelism.

TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and the
cpu_baseline leg of bench.py may import or run anything in this package.
The product path (the paper_2609_22755_amd package and its HIP library)
never imports it and shares no code, header, table or helper with it; the
only thing both sides consume is the seeded input generator
(paper_2609_22755_amd.workloads), which holds none of the method's
arithmetic.

What the oracle computes, and from which passage of the paper:

* attention.py -- per-sequence causal softmax attention over a packed,
  variable-length batch (Background, Sequence Packing: sequences in a pack do
  not attend to each other), computed per query head on the heads this GPU
  holds after the Ulysses exchange (Background, Sequence Parallelism: each GPU
  holds the full sequence for a subset of heads and attention is computed
  locally over complete sequences), with grouped-query KV heads.  Forward and
  backward, in float64, by the plain definition; the method's FlashAttention
  kernels (Implementation) compute exactly this, only faster.
* ulysses.py -- the local halves of the Ulysses prologue/epilogue
  (Background, Sequence Parallelism; Implementation, backend interface):
  sequence-sharded <-> head-sharded re-layout, as pure index maps.
* planner.py -- SP-tree routing, the NSP Planner (Design, NSP Planner: SP
  Tree Topology, Routing Objective and Cost Model, Routing Algorithm): the
  token loads, the hierarchical cost model with its profiled coefficients as
  parameters, and Algorithm 1 (beam search over the longest samples, greedy
  completion of the tail), in plain Python.
* recompute.py -- the tree-level recomputation plan (Design, NSP Executor,
  Tree-Level Recomputation): SAVE / RECOMPUTE marks from an activation
  budget, walking the SP tree root first, in plain Python.

Every function is pinned by tests/test_oracle_*.py against brute force,
torch's fp64 SDPA + autograd, finite differences, closed forms and
invariants; see those files for which pin catches which mistake.
"""

from . import attention, planner, recompute, ulysses  # noqa: F401
