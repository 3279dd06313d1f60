"""CPU oracle of the ABFT-protected attention layer (EEC-ABFT, ATTNChecker).

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import, call or
execute this package: only tests/, __graft_entry__.smoke() and bench.py's
cpu_baseline leg use it. It shares no code with the HIP path; the only
common module is `workloads`, which draws seeded inputs and holds none of
the method's arithmetic.

All arithmetic is float64. Every tensor the GPU stores is rounded here to
the storage dtype (round-to-nearest-even) at the same point, and injected
faults are written after that rounding. Propagated checksums stay float64.

Modules:
  numerics  - storage rounding and extreme-value classification (Sec. 2.2)
  eec       - checksum encoding (Sec. 2.3) and per-vector EEC-ABFT (Sec. 4.2),
              column/row passes for 1-D propagation (Sec. 4.3)
  layer     - the protected layer forward (Sec. 4.4 protection sections) and
              the protected backward chain (an extension; the paper is silent)
  freq      - adaptive detection frequencies (Sec. 4.5, Algorithm 1)
  fused     - the score/softmax/context core in an online-softmax form that
              stores neither AS nor AP (an extension), row-side checks

Parity pins are listed in the test files that check each function.
"""
from .numerics import round_to, stored_threshold, classify, KINDS
from .eec import (col_checksums, row_checksums, eec_locate, fix_by_checksum,
                  EECResult, Verifier)
from .layer import OracleParams, forward, backward, pattern_of_events

__all__ = [
    "round_to", "stored_threshold", "classify", "KINDS",
    "col_checksums", "row_checksums", "eec_locate", "fix_by_checksum",
    "EECResult", "Verifier", "OracleParams", "forward", "backward",
    "pattern_of_events",
]
