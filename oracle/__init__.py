"""Plain CPU oracle for Hybrid-SWA paged attention.

TEST INFRASTRUCTURE ONLY. Nothing in the product path (the HIP library and its
Python binding) may import, call or execute anything in this package; only the
tests, the smoke check and the CPU-baseline leg of the benchmark use it.

The oracle is written from the paper ("Full-Pipeline Inference Optimization for
MiMo-V2.5 Series", sections "Compute Analysis", "KVCache Storage Analysis",
"KVCache Dual-Pool Design" and "SWA-Aware Prefix Cache Tree") and shares no code,
table or constant with the GPU path. It imports numpy only.

* ``attention``: fp64 masked softmax attention over a contiguous, unpaged KV
  history with an explicit causal / sliding-window mask.
* ``layout``: the integer rules of the dual-pool paged layout (ring size, block
  tables, slot mapping, post-append pool content, storage accounting).

Every function is pinned by the CPU tests (brute force, closed forms,
invariants, a library routine); none is "parity unpinned".
"""

from . import attention, layout  # noqa: F401
