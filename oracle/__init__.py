"""CPU oracle for the WorldDynCache denoising rollout (test infrastructure).

Plain, slow, float64 NumPy written from the paper. Only the test suite, the
``__graft_entry__.smoke()`` self-check and the benchmark's CPU-baseline leg may
import it; the GPU product path never does and shares no code with it (the
only common module is ``synth``, which generates seeded inputs and holds none
of the method's arithmetic).

Modules
  dit        the denoiser F_theta of Eq. (1) (a synthetic video DiT; the paper
             does not specify its architecture) -- parity pinned by the tests
             in tests/test_oracle_dit.py
  scheduler  the scheduler transition Psi_t of Eq. (1) (flow-matching Euler)
  surrogate  the latent dynamics surrogate G_t: Eq. (2)-(5)
  risk       the transition risk controller: Eq. (6)-(10)
  rollout    the inference loop of Sec. 4.4 (exact anchors and surrogate steps),
             with the periodic placement and surrogate variants of Sec. 5.4
  diagnostics  the injection sweep of Observation 1 (Sec. 3) and the
             correlation / false-safe statistics of Sec. 4.3

Where the paper defers details to its supplementary material, the reading
used is recorded in ``params.DEFAULTS`` and in the module docstrings.

Pins: every operation, block and the composed ``dit.dit_forward`` is pinned
(library routines, closed forms, brute force, an independent torch
composition, and invariants the architecture fixes: head relabelling,
text-token order, zero residual gates). A random-init model has no output
value the paper prints, and the paper's correlations and false-safe rates come
from trained models, so the values the diagnostics produce here are not
compared with the paper's; the diagnostics' arithmetic is pinned.
"""
from . import params, dit, scheduler, surrogate, risk, rollout  # noqa: F401
