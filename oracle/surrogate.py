"""Latent Dynamics Surrogate G_t (Sec. 4.2, Eq. (2)-(5)), float64.

Lifted state, Eq. (2):
    phi = [nu(z), nu(z - z_a), cam, depth, q, h]
with nu(x) = x / sqrt(mean(x^2) + eps_nu) over all of x (RMS normalisation),
z_a the anchor (input latent of the latest exact step; nu(z - z_a) = 0 before
the first one), cam and depth 16-d normalised descriptors (zero when absent),
q the scheduler phase (normalised timestep) and h a 32-d summary of the latest
exact transition: h = P_2(nu(z_out - z_in)) (zero before the first one).

Summary s, "a fixed 256-dimensional summary" (Sec. 4.2): the reading is a
linear chunk pooling,
    s(phi) = [P_8(phi.z) (128), P_4(phi.dz) (64), h (32), cam (16), depth (16)]
with P_G(x)[c, g] = n_{c,g}^{-1/2} * sum over flat spatial index j of
channel c with floor(j*G/T) = g, T = F*H*W. q is not part of s.

Transition retrieval, Eq. (3); scheduler scaling and lifted evolution, Eq. (4);
kernelized observation, Eq. (5). The lifted evolution is carried out on the
full-size lifted state and only then summarised.

Variants of the ablation study (Sec. 5.4, matched-budget tables), as read here:

* linear observation: the evolved lifted state is read back linearly, by
  undoing the RMS normalisation of its latent block:
  z_hat = rho(z_t) * phi_hat.z, rho(x) = sqrt(mean(x^2) + eps_nu);
* lift without condition: the camera/depth blocks are zero and retrieval
  ignores the scheduler phase (no phase penalty, no phase compatibility test);
* native latent secant: no lift at all; the latest exact transition
  (z_a -> z_out, phases q_a -> q_{a-1}) is extrapolated in latent space,
  z_hat = z_t + (q_{t-1} - q_t) / (q_{a-1} - q_a) * (z_out - z_a).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

S_DIM = 256
G_Z, G_DZ, G_H, G_CAM = 8, 4, 2, 16


def f64(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64)


def nu(x: np.ndarray, eps: float) -> np.ndarray:
    x = f64(x)
    return x / np.sqrt(np.mean(x * x) + eps)


def pool(x: np.ndarray, groups: int) -> np.ndarray:
    """P_G over the flattened spatial index of each channel; x: [C, ...] -> [C*G]."""
    x = f64(x)
    c = x.shape[0]
    flat = x.reshape(c, -1)
    t = flat.shape[1]
    g = (np.arange(t) * groups) // t
    out = np.zeros((c, groups))
    for gi in range(groups):
        m = g == gi
        out[:, gi] = flat[:, m].sum(axis=1) / np.sqrt(m.sum())
    return out.reshape(-1)


def cam_descriptor(cam: Optional[np.ndarray], eps: float) -> np.ndarray:
    """16-d normalised camera/motion descriptor P_16(nu(cam)); zero when absent."""
    if cam is None:
        return np.zeros(G_CAM)
    return pool(nu(cam, eps)[None, :], G_CAM)


@dataclass
class Lifted:
    """phi = Phi(z, H) of Eq. (2), kept block by block at full size."""
    z: np.ndarray        # nu(z), latent shape
    dz: np.ndarray       # nu(z - z_a), latent shape
    cam: np.ndarray      # [16]
    depth: np.ndarray    # [16]
    q: float
    h: np.ndarray        # [32]

    def __sub__(self, o: "Lifted") -> "Lifted":
        return Lifted(self.z - o.z, self.dz - o.dz, self.cam - o.cam, self.depth - o.depth,
                      self.q - o.q, self.h - o.h)

    def axpy(self, a: float, o: "Lifted") -> "Lifted":
        """self + a * o."""
        return Lifted(self.z + a * o.z, self.dz + a * o.dz, self.cam + a * o.cam,
                      self.depth + a * o.depth, self.q + a * o.q, self.h + a * o.h)


def lift(z, z_anchor, h, q: float, cam_desc, p) -> Lifted:
    """Eq. (2). ``h``: current history summary (None -> zero); ``z_anchor`` None -> no anchor."""
    z = f64(z)
    dz = np.zeros_like(z) if z_anchor is None else nu(z - f64(z_anchor), p.eps_nu)
    c = z.shape[0]
    cam = f64(cam_desc) if p.lift_condition else np.zeros(G_CAM)
    return Lifted(nu(z, p.eps_nu), dz, cam, np.zeros(G_CAM), float(q),
                  np.zeros(c * G_H) if h is None else f64(h))


def summary(phi: Lifted) -> np.ndarray:
    s = np.concatenate([pool(phi.z, G_Z), pool(phi.dz, G_DZ), phi.h, phi.cam, phi.depth])
    assert s.shape == (S_DIM,), "the 256-d summary assumes 16 latent channels"
    return s


def history_summary(z_in, z_out, p) -> np.ndarray:
    """h(H) = P_2(nu(z_out - z_in)) of the latest exact transition."""
    return pool(nu(f64(z_out) - f64(z_in), p.eps_nu), G_H)


def sim(a: np.ndarray, b: np.ndarray) -> float:
    """Cosine similarity; 0 when either vector is (numerically) zero."""
    den = np.linalg.norm(a) * np.linalg.norm(b)
    return float(a @ b / den) if den >= 1e-30 else 0.0


def softmax(x: np.ndarray) -> np.ndarray:
    e = np.exp(x - x.max())
    return e / e.sum()


@dataclass
class Record:
    """One exact transition in the bank B_t (Sec. 4.2): lifted input/output,
    their summaries, phases and the exact output latent."""
    phi_in: Lifted
    phi_out: Lifted
    s_in: np.ndarray
    s_out: np.ndarray
    q_in: float
    q_out: float
    z_out: np.ndarray


@dataclass
class Bank:
    """FIFO of capacity M; slot = (number of inserts) mod M. Only exact
    transitions are ever inserted."""
    capacity: int
    slots: List[Optional[Record]] = field(default_factory=list)
    inserts: int = 0

    def __post_init__(self):
        if not self.slots:
            self.slots = [None] * self.capacity

    def records(self):
        """(slot, record) in slot order."""
        return [(i, r) for i, r in enumerate(self.slots) if r is not None]

    def __len__(self):
        return sum(r is not None for r in self.slots)

    def insert(self, rec: Record) -> int:
        slot = self.inserts % self.capacity
        self.slots[slot] = rec
        self.inserts += 1
        return slot


@dataclass
class Candidate:
    support: List[int]          # slots in N_t
    sims_in: np.ndarray         # sim(s(phi_t), s(phi_i^in)) per record (slot order)
    logits: np.ndarray          # l_i per record
    pi: np.ndarray              # retrieval weights per record (0 outside N_t)
    alpha: float
    s_hat: np.ndarray           # s(phi_hat)
    kappa: np.ndarray           # observation weights per record
    z_hat: np.ndarray
    finite: bool
    slots: List[int]


def scheduler_scale(t_cur: float, t_next: float, q_a: float, q_am1: float, p) -> float:
    """alpha_t of Eq. (4): clip(|q_{t-1} - q_t| / (|q_{a-1} - q_a| + eps), alpha_min, alpha_max)."""
    return float(np.clip(abs(t_next - t_cur) / (abs(q_am1 - q_a) + p.eps), p.alpha_min, p.alpha_max))


def candidate(phi: Lifted, bank: Bank, t_next: float, q_a: float, q_am1: float, p,
              z=None) -> Optional[Candidate]:
    """G_t(z_t, H_t): retrieval (Eq. (3)), lifted evolution (Eq. (4)) and
    kernelized observation (Eq. (5)). None when the bank is empty. ``z`` (the
    current latent) is needed only by the linear observation."""
    recs = bank.records()
    if not recs:
        return None
    s_t = summary(phi)
    slots = [i for i, _ in recs]
    sims_in = np.array([sim(s_t, r.s_in) for _, r in recs])
    dq = np.array([phi.q - r.q_in for _, r in recs])
    if p.lift_condition:
        logits = sims_in - p.gamma_q * dq ** 2
        supp = [j for j in range(len(recs)) if sims_in[j] >= p.theta_sim and abs(dq[j]) <= p.theta_q]
    else:
        logits = sims_in.copy()
        supp = [j for j in range(len(recs)) if sims_in[j] >= p.theta_sim]
    pi = np.zeros(len(recs))
    if supp:
        pi[supp] = softmax(logits[supp] / p.tau_in)
    alpha = scheduler_scale(phi.q, t_next, q_a, q_am1, p)
    phi_hat = phi
    for j in supp:
        phi_hat = phi_hat.axpy(alpha * pi[j], recs[j][1].phi_out - recs[j][1].phi_in)
    s_hat = summary(phi_hat)
    if p.observation == "linear":
        zc = f64(z)
        kappa = np.zeros(len(recs))
        z_hat = np.sqrt(np.mean(zc * zc) + p.eps_nu) * phi_hat.z
    else:
        kappa = softmax(np.array([sim(s_hat, r.s_out) for _, r in recs]) / p.tau_obs)
        z_hat = np.zeros_like(recs[0][1].z_out, dtype=np.float64)
        for j, (_, r) in enumerate(recs):
            z_hat = z_hat + kappa[j] * f64(r.z_out)
    return Candidate([slots[j] for j in supp], sims_in, logits, pi, alpha, s_hat, kappa, z_hat,
                     bool(np.all(np.isfinite(z_hat))), slots)


def secant_candidate(z, z_anchor, bank: Bank, t_cur: float, t_next: float, q_a: float, q_am1: float,
                     p) -> Optional[Candidate]:
    """Native latent secant: the latest exact transition z_a -> z_out, taken over
    the phase interval q_a -> q_{a-1}, extrapolated from z_t over q_t -> q_{t-1}.
    None when no exact transition has been recorded."""
    recs = bank.records()
    if not recs or z_anchor is None:
        return None
    latest = (bank.inserts - 1) % bank.capacity
    slots = [i for i, _ in recs]
    j = slots.index(latest)
    ratio = (t_next - t_cur) / (q_am1 - q_a)
    z_hat = f64(z) + ratio * (f64(bank.slots[latest].z_out) - f64(z_anchor))
    n = len(recs)
    pi = np.zeros(n)
    pi[j] = 1.0
    return Candidate([latest], np.zeros(n), np.zeros(n), pi, ratio, np.zeros(S_DIM), np.zeros(n), z_hat,
                     bool(np.all(np.isfinite(z_hat))), slots)
