"""Constants of the method that the paper leaves to its supplementary material.

Each entry is a reading; the paper fixes only the anchor-age limit (six, in the
reliability decision of Sec. 4.3) and the cap of 2 on the future-sensitivity
weight (Eq. (9)).
"""
from dataclasses import dataclass, replace


@dataclass(frozen=True)
class Params:
    # memory (Sec. 4.2 "Local Lifted Evolution": capacity is unspecified)
    bank_capacity: int = 4
    # compatibility thresholds defining the supported set N_t (Eq. (3) text)
    theta_sim: float = 0.25
    theta_q: float = 0.43          # chosen off the 1/8, 1/20, 1/50 time grids
    # temperatures and the phase penalty (Eq. (3), Eq. (5))
    tau_in: float = 0.05
    tau_obs: float = 0.02
    gamma_q: float = 10.0
    # scheduler scaling clip (Eq. (4))
    alpha_min: float = 0.5
    alpha_max: float = 2.0
    eps: float = 1e-8
    # RMS normalisation nu in the lifted state (Eq. (2))
    eps_nu: float = 1e-6
    # proxy weights (Eq. (6))
    w_z: float = 1.0
    w_age: float = 0.05
    w_phase: float = 0.5
    w_cam: float = 0.5
    w_depth: float = 0.5
    # online calibration (Eq. (8))
    eta0: float = 1.0
    beta_d: float = 0.8
    eta_min: float = 0.05
    eta_max: float = 20.0
    # future sensitivity (Eq. (9))
    a_cam: float = 0.5
    a_depth: float = 0.5
    a_phase: float = 0.5
    lam: float = 0.8
    r0: float = 0.0
    # availability (Eq. (10) text)
    age_max: int = 6               # pre-decision anchor age at most six (given by the paper)
    n_min: int = 1                 # adequate retrieval support
    k_init: int = 1                # mandatory-exact initialisation steps
    k_ref: int = 0                 # mandatory-exact refinement steps at the end
    tau_risk: float = 0.5
    # Variants compared in the ablation study (Sec. 5.4, matched-budget tables).
    # Controller "periodic": exact when k mod period == 0, otherwise the
    # surrogate whenever it is available (periodic placement).
    period: int = 4
    # Surrogate construction: "lifted" (Eq. (2)-(5)) or "secant" (native latent
    # secant: extrapolate the latest exact transition in latent space).
    surrogate: str = "lifted"
    # Observation: "kernel" (Eq. (5)) or "linear" (undo the RMS normalisation of
    # the evolved latent block of the lifted state).
    observation: str = "kernel"
    lift_condition: bool = True      # False: no condition / phase information in the lift
    impact_weight: bool = True       # False: w_t = 1 (no future-impact weighting, Eq. (9))
    calibrate: bool = True           # False: eta_d stays at eta0 (no counterfactual calibration)
    support_constraint: bool = True  # False: availability ignores retrieval support


DEFAULTS = Params()


def with_(p: Params = DEFAULTS, **kw) -> Params:
    return replace(p, **kw)
