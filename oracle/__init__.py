"""CPU oracle for pipelined model swap-in and execution.

TEST INFRASTRUCTURE ONLY. Nothing on the product path imports this package: only the
test suite, the smoke check and the benchmark's CPU-baseline leg call it. It shares no
code with the HIP library; its sole input from elsewhere is the seeded synthetic data
(weights, layouts and request inputs) produced by ``synth``.

Swapping changes where and when weights arrive, never the arithmetic: the redirected
execution keeps the order of operations and hence the inference result (paper Sec. 4.2),
the host copy of a model is always kept (Sec. 4.3, "Model eviction"), and swapping only
relocates memory blocks whose internal offsets are unchanged (Sec. 4.4, "Memory address
management"). So the oracle is the plain forward pass of each model from the same weight
bytes (``forward``), plus the byte-level placement and eviction rules (``arena_sim``) and
the transfer grouping rule (``chunks``) and the modelled time of a pipelined request
under a grouping (``pipeline``), and the SLO-aware queueing rules (``slo_queue``).

Precision: float64 by default (the paper fixes none); ``dt=np.float32`` gives the fp32
variant. bf16 weights and inputs are widened exactly.
"""
from . import ops, forward, arena_sim, partition_sim, chunks, pipeline, slo_queue  # noqa: F401
