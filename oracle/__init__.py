"""CPU oracle for FlashCP's rank-shard attention path.

TEST INFRASTRUCTURE ONLY. Nothing on the product path may import, call or
link anything in this package: only the test suite, the smoke check in
``__graft_entry__`` and the CPU-baseline leg of ``bench.py`` use it. It shares
no code with the HIP library (``paper_2606_08476_amd``) and imports nothing
from it; the two are handed the same seeded inputs and compared.

Modules
-------
planner    shard plans: Per-Doc, Whole-Doc LPT, the hybrid heuristic
           (Algorithm 1), validation against Eq. 1/Eq. 2, and statistics
           (per-rank workload W, Eq. 4 and Eq. 5 volumes, imbalance).
view       a rank's view of a plan (its query tokens, the received KV set,
           document segments, pieces) and the tile maps derived from it.
attention  document-masked causal attention forward/backward in fp64, its
           partial passes over a subset of keys, and the log-sum-exp merge.

Parity status of each function is stated in its module header.
"""
