"""CPU oracle for the layer-wise prefix-KV reload and prefill attention path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product library imports, links or
calls this package: only the test-suite, the smoke check and the CPU-baseline
leg of the benchmark do.  It shares no code with the HIP path (no kernels,
headers, helpers or constant tables); both sides only consume the same seeded
inputs.

Contents
--------
``kvcache``   block-major donor pool addressing, the per-layer gather of a
              conversation's prefix blocks into an active-layer buffer, the
              append of the new turn, and the write-back (store) of the new
              turn into pool blocks (paper §3.2 "Layer Stream Cache", §3.3
              "KV Store"/"KV Load", §3.4 "Block-Major Layout", Eq. 1).
``attention`` exact causal GQA prefill attention over prefix + new tokens in
              float64, a row-sampled variant for large shapes, and the
              log-sum-exp merge of attention over disjoint key sets
              (paper §2.1-§2.2: causal attention over every earlier position and itself;
              §5 "Model": GQA).
``capacity``  the master's layer stream cache and regular cache sizes and
              the longest supported context (§3.2, Eq. 1-5).
``elastic``   the worker's elastic cache: layer-major vs block-major resize
              moves, the minimum elastic unit (Eq. 6-9) and the scale-up /
              scale-down decisions of Algorithm 1 (§3.4-§3.5).

Precision: bf16 inputs are upcast exactly to float64 and everything is
computed in float64 (the paper fixes half precision for storage only).

Every function here is pinned by the ``-m "not gpu"`` tests against brute
force, closed forms, invariants and library routines; see the module
docstrings for which pin covers which function.  No function is "parity
unpinned".
"""

from . import attention, capacity, elastic, kvcache  # noqa: F401
