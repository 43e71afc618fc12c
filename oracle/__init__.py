"""CPU oracle for the WAMachine denoising hot path — TEST INFRASTRUCTURE ONLY.

A plain, slow, float64 NumPy implementation of what the device path computes:
the synthetic DiT denoiser (``dit``), the flow solver, and the paper's three
state-adaptation operators together with the joint replan runtime
(``method``), plus the paper's timing and reuse statistics (``metrics``).

Only the test-suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  It shares no code with the HIP library and does not
import it; both consume the seeded inputs of the ``synth`` package.

Parity status per function is stated in each module header.  The DiT itself
is not defined by the paper (it only cites DiT), so its absolute outputs are
pinned by library cross-checks of each piece rather than by printed values.
"""
from . import dit, method, metrics  # noqa: F401
