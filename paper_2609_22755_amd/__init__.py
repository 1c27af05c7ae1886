"""MI355X-native per-GPU hot path of Nested Sequence Parallelism (NSP).

Variable-length causal grouped-query attention, forward and backward, over
one GPU's share of an SP tree, plus the local Ulysses re-layout around it,
as hand-written HIP kernels for gfx950 behind the C-ABI library libnsp.so
(include/nsp.h).  ``paper_2609_22755_amd.nsp`` is the thin ctypes binding;
``paper_2609_22755_amd.workloads`` draws seeded synthetic work lists.
"""
