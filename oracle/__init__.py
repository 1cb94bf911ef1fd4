"""Plain, slow, fp64 CPU oracle of the DraftExpert MoE draft/verify hot path.

TEST INFRASTRUCTURE ONLY.  It exists to check the HIP path, never to serve
it: only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg
of ``bench.py`` may import it.  It shares no code with the HIP library and
imports nothing from it.

Modules
    moe     one MoE layer: routing (Eq. 1), union and token lists (Eq. 2-3),
            target output (Eq. 4), draft output (Eq. 5), RMSNorm, greedy accept
    decode  the stacked model, the exact draft/verify step and greedy AR
            decoding (Algorithm 1)
    cache_sim  the expert cache bookkeeping with draft-router prefetch
               (Section 3.5, Algorithm 1)
    truncation confidence-expansion truncation of the draft loop
               (Section 3.4, Eqs. 12-14, Algorithm 1)
    q4      dequantisation of Q4_0 expert weights (Section 4.1's 4.5-bit format)
    distill the self-distillation signals of Eqs. 6-10 from teacher-forced passes

Pins (tests/test_oracle_*.py) tie every function to the paper or to
mathematics independent of this code; functions without such a pin say
"parity unpinned" in their docstring.
"""
from . import cache_sim, decode, distill, moe, q4, truncation  # noqa: F401
