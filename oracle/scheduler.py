"""Scheduler transition Psi_t of Eq. (1) and the time grid.

The paper leaves Psi_t unspecified (Sec. 4.1). The reading used is the
flow-matching Euler step on the uniform grid t_k = (S-k)/S, k = 0..S: the
paper's step t -> t-1 is step k -> k+1 here, and the scheduler phase q_k is
the normalised timestep t_k (Sec. 4.2, "normalized timestep replaces
unavailable scheduler phase").
"""
import numpy as np


def t_at(k: int, steps: int) -> float:
    """t_k = (S - k) / S, k = 0..S (1 at the start, 0 at the end)."""
    return (steps - k) / steps


def time_grid(steps: int) -> np.ndarray:
    return np.array([t_at(k, steps) for k in range(steps + 1)], dtype=np.float64)


def psi(z: np.ndarray, v: np.ndarray, t_cur: float, t_next: float) -> np.ndarray:
    """z_{k+1} = z_k + (t_{k+1} - t_k) * v_k."""
    return np.asarray(z, dtype=np.float64) + (t_next - t_cur) * np.asarray(v, dtype=np.float64)
