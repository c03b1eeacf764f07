"""CPU oracle for the ECASQ hot path.

TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and the
cpu_baseline leg of bench.py may import, call, link or execute anything under
oracle/.  It shares no code with the GPU library (paper_2608_18147_amd).

Modules:
  plain      per-entry definitions, brute force, ASQ DP, optimal DP
  pipeline   histogram, exact prefix sums, search/recovery/refinement via C,
             stochastic rounding
  native     ctypes loader for ecasq_oracle.c (canonical-arithmetic DP)
  philox     Philox4x32-10 in numpy
  log2_table correctly rounded table of the canonical log2 (mpmath)

Every function is pinned to something other than itself (closed forms, brute
force, the paper's worked examples, per-entry definitions in plain.py);
tests/test_oracle_*.py hold the pins.  The refinement is the paper's
heuristic procedure: what it computes is pinned step by step against the
per-entry objective (tests/test_oracle_refine_pins.py).
"""
