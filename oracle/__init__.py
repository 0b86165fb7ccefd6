"""Oracle for the two-party publisher/subscriber split-learning training step.

TEST INFRASTRUCTURE ONLY.  A plain, slow, float64 CPU implementation written
from the paper (PubSub-VFL, arXiv 2510.12494: Section 3 "Problem Formulation",
Eqs. (1)-(2); Section 4.1 "System Design"; Appendix "Differential Privacy
Protocol"; Assumption 4 and the Theorem's delayed update rule; Algorithm 1).
Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import it.  It shares no code with the GPU path: the two meet
only in the seeded input generators of ``vfl_synth``.

Modules:
  philox    Philox4x32-10 (published definition) + Box-Muller Gaussians
  rounding  storage rounding for the bf16 / f32 emulation modes
  layers    dense layer, ReLU, BCE (Eq. 1), per-row clip, embedding lookup
  schedule  closed-form integer schedule (slots, versions, delays)
  pubsub    the tick loop: publish, subscribe + top step, delayed backward,
            parameter-server averaging, SGD (Eq. 2)

Parity status: every function here is pinned by a CPU test in ``tests/``
(test_oracle_*.py) except the privacy accounting that would relate the
noise multiplier to a privacy budget, which the paper gives only up to an
unspecified constant (Eq. 25): parity unpinned, and not implemented.
"""
from .pubsub import PubSubOracle, ROUNDING_POINTS  # noqa: F401
from . import layers, philox, rounding, schedule  # noqa: F401
