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

Parity status per function is recorded in the header of each module; the
refinement heuristic is "parity unpinned" beyond the invariants its tests
check (objective never increases; the three colour classes are separable).
"""
