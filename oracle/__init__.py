"""CPU oracle for the ChronoStitch KV-composition hot path.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, obviously correct
reference written from the paper (ChronoStitch, Section 2, Eqs. 1-3 and 5 and
the top-rho repair procedure that follows Eq. 5).  It computes in float64 with
numpy and rounds to the storage dtype only where the stored cache itself is
rounded.  It shares no code with the HIP library and imports nothing from it.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import or call anything in this package.  The product path
(the C-ABI library and its Python binding) never does.

Modules
  bf16       exact bfloat16 codec (decode to fp64, fp64 -> bf16 round-to-nearest-even)
  rope       three-axis mRoPE primitives (Eq. 2)
  rebase     three-axis delta rotation of stored post-rotary keys (Eq. 3)
  score      per-token key deviation (Eq. 5)
  select     top-rho selection over later-chunk tokens (Section 2, after Eq. 5)
  attention  scatter of fresh K/V rows, then causal GQA softmax attention (Eq. 1)
  compose    the stages chained in the paper's order

Every function here is pinned by ``tests/test_oracle_*.py`` against closed
forms, invariants, library routines or brute force; none is "parity unpinned".
"""
from . import bf16, rope, rebase, score, select, attention, compose, inputs, policies  # noqa: F401
