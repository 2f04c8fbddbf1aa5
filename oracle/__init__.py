"""CPU oracle for the CAI-dLLM denoising step -- TEST INFRASTRUCTURE ONLY.

This package is a plain, slow, deliberately unoptimised restatement of what
the paper computes, used to check the HIP path.  It is not part of the
product: only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg
of ``bench.py`` may import it, and the product path never calls it.  It shares
no code with the HIP library and imports nothing from the product package;
it receives weights, prompts and traces as plain numpy arrays.

Modules
  forward    -- the bidirectional transformer forward (Section 2, Section 4.1)
  vocab      -- token confidence and greedy prediction (Box 1, Eq. first_conf)
  controller -- thresholds, budgets and Algorithm 1 (Boxes 2-7, Section 4.7)
  kvcache    -- cross-step key/value reuse (Section 5's cached decoder)

Parity status: every function is pinned by ``tests/test_oracle_*.py``
against library routines, closed forms, hand-derived traces and invariants;
the absolute decoding trajectory of a random-weight model has no printed
counterpart in the paper and is pinned only through those pieces.
"""
from . import controller, forward, kvcache, vocab  # noqa: F401
