"""Constrained Kernel-SHAP weighted least squares (eq. 2-3, Alg. 1 step 5,
Sec. 3.5).

The surrogate g(m) = phi_0 + sum_i phi_i m_i (eq. 2) is fitted to the sampled
coalition values by minimising sum_b w_b (f(S_b) - g(m_b))^2 (eq. 3).  The
kernel weight is infinite for the empty and the full coalition; that is read
as two exact constraints: phi_0 = f(empty) and sum_i phi_i = f(full) - f(empty)
(efficiency).  The oracle eliminates the last player with the efficiency
constraint and solves the unconstrained problem with numpy's SVD-based lstsq.
"""
import numpy as np


def kernel_shap(masks, weights, y, f_empty, f_full):
    m = np.asarray(masks, dtype=np.float64)
    w = np.asarray(weights, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    delta = float(f_full) - float(f_empty)
    M = m.shape[1]
    if M == 1:
        return np.array([delta])
    X = m[:, :-1] - m[:, -1:]
    t = y - float(f_empty) - m[:, -1] * delta
    sw = np.sqrt(w)
    head, *_ = np.linalg.lstsq(sw[:, None] * X, sw * t, rcond=None)
    return np.concatenate([head, [delta - head.sum()]])
