"""CPU oracle for Prof-K top-k selection -- TEST INFRASTRUCTURE ONLY.

This package is a plain, slow, obviously-correct CPU statement of what the
Prof-K method computes.  It exists to check the HIP implementation, never to
serve as one: only the test suite, the smoke check and the benchmark's CPU
baseline leg may import it.  It shares no code with the HIP library (no
headers, no helpers, no tables) and never imports it.

Modules
  keys   -- the order-preserving integer key that defines the total order
            (value descending, then index ascending) used for every result.
  philox -- Philox4x64-10 counter-based generator (Salmon et al., SC'11) and
            the map from a 64-bit word to a sample index in [0, N).
  plan   -- Algorithm 1 (adaptive parameter selection) and the exact
            binomial-tail choice of the threshold rank t and capacity M.
  exact  -- O1: exact top-k by a full stable sort (Sec. 3 problem statement).
  profk  -- O2: the four stages of Prof-K (Sec. 3) step by step on the CPU,
            for the flat, per-row and flattened-BatchTopK forms.

Floating point is fp64 throughout the planner; every other step is integer
or bit-copy work and therefore exact.
"""

from . import keys, philox, plan, exact, profk  # noqa: F401
