"""CPU oracle of the FOCUS hot path (arXiv 2511.14694) -- TEST INFRASTRUCTURE.

A plain, slow, obviously correct implementation of what the hot path computes,
written from the paper in float64 NumPy and pure Python.  It exists to check the
HIP path; it is not part of it.  Only `tests/`, `__graft_entry__.smoke()` and the
`cpu_baseline` leg of `bench.py` may import or run anything in this package.
It shares no code with `paper_2511_14694_amd/`: neither imports the other, and
the only module both sides use is `focus_workloads` (seeded random inputs,
which holds none of the method's arithmetic).

Modules
  layout     summary-token insertion and window/cache bookkeeping
             (Section 3.2 "Setup and tokens"; Appendix A window and B_w definitions)
  attention  window attention over [retained summary KV ; window KV] under the
             visibility set C(t) (Appendix A eq. focus-attn, A.1 "Objective and
             visibility" and "Cross-window consistency"), the retained-KV
             compaction (Appendix A "KV compression and budget") and the
             textbook dense causal attention it must reduce to with no summaries
  decode     streaming one token at a time over the same state
             (Appendix A.2 "Streaming with controlled memory")

Parity pins (each function is checked against facts the paper or mathematics
fix, never against itself) live in tests/test_oracle_*.py.  No function here is
"parity unpinned".
"""
