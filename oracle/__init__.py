"""CPU oracle for the rolling denoise step -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously correct numpy definition of what the GPU library
computes, written from the paper (Sec. 3.1 Eq. 1/3, Sec. 3.2 Eq. 4, App. A.1)
plus the readings listed in each module's header.  It shares no code with the
HIP path: only the tests, ``__graft_entry__.smoke()`` and the bench's
CPU-baseline leg may import it.  Product code never does.

Modules:
  philox   -- Philox4x32-10 + Box-Muller ring noise (pinned by published
              known-answer vectors).
  expert   -- the action expert v_theta (conditioning, adaptive RMSNorm,
              grouped-query attention over [prefix ; buffer], FOP adapters,
              gated-GeLU MLP, output head) and the FOP stand-in encoder.
  rolling  -- the rolling buffer: Euler update, release, noise append,
              context publication and temporal offset.
  full     -- the full-horizon synchronous baseline (all slots share one flow
              time, S Euler steps per chunk).
  training -- the streaming-aligned training objective (buffer at the rolling
              profile, offset p / K, flow-matching loss).

Pins: every function here is checked in tests/test_oracle_*.py against
something other than itself (library routines, closed forms, special cases,
invariants, known-answer vectors, planted mistakes that must fail).  The paper
prints no numeric example of the expert's output (no trained weights exist), so
values at random weights rest on those pins.
"""

from .expert import Expert, fop_encode  # noqa: F401
from .philox import philox4x32_10, ring_noise  # noqa: F401
from .rolling import OracleRavel  # noqa: F401
from .full import expert_velocity, full_denoise  # noqa: F401
from .training import training_buffer, training_loss  # noqa: F401
