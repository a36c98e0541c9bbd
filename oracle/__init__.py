"""Plain fp64 CPU oracle for CoWindow Attention (CoWA).

TEST INFRASTRUCTURE ONLY.  This package is the parity reference that the
GPU library is checked against.  Only the test suite, the smoke check in
``__graft_entry__`` and the ``cpu_baseline`` leg of ``bench.py`` may import
it.  The product path (the HIP library and its Python binding) never
imports, links or calls anything here, and nothing here imports the product.

Everything is written from the paper's definitions, one step at a time, in
float64 NumPy (and pure Python for the tiny brute-force cases):

* ``windows``   -- the window rule: causal distance (Eq. fwa_distance), GQA
                   head map (Sec. 2.1), long-range span and breakpoints
                   (Eq. fwa_long_range_span), the three windows and their
                   union (Eq. fwa_support), global KV-head indexing
                   (Eq. fwa_global_head).
* ``schedule``  -- the KV-block sets J(i) and their inverse I(j) (Sec. 2.3,
                   forward and backward execution), built two independent
                   ways.
* ``attention`` -- masked softmax attention forward (Alg. 1 computes exactly
                   this), its exact gradient (Alg. 2), and decoding
                   (Sec. 2.3, decoding execution).
* ``counts``    -- support sizes, legal-pair counts and FLOP accounting
                   (Eq. fwa_support_counts; App. A.2 and A.3).

Every function is pinned by tests that check it against what the paper or
plain mathematics fixes (printed budgets and mean supports, collective
coverage, closed-form counts, reductions to dense causal attention, library
routines, finite differences, brute force).
"""

from . import windows, schedule, attention, counts  # noqa: F401
