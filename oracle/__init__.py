"""fp64 CPU oracle for Turbo-Muon orthogonalization.

TEST INFRASTRUCTURE ONLY.  Only the tests, the package's smoke check and the
benchmark's CPU-baseline leg may import this package.  The HIP library never
calls it and shares no code with it.
"""
from .turbomuon import (  # noqa: F401
    CONSTANT_TRIPLE, aol_vector, aol, frobenius_scale, schatten4_scale, first_iterate,
    quintic_step, newton_schulz, schedule_last,
    orthogonalize, polar_factor, eps_ortho, eps_polar, eps_bias, eps_approx,
    rel_frobenius, preconditioned, round_bf16, muon_step,
)
