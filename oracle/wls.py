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


def kernel_shap_normal(masks, weights, y, f_empty, f_full, chunk=2048):
    """The same constrained least squares as kernel_shap (the last player
    eliminated with the efficiency constraint), solved through its normal
    equations: (X'^T W X') head = X'^T W t, with X'^T W X' accumulated over
    blocks of rows in fp64 and factored by Cholesky (LAPACK).  For systems
    whose rows are too many for lstsq's SVD; pinned against kernel_shap."""
    import scipy.linalg as sla
    masks = np.asarray(masks, dtype=bool)
    w = np.asarray(weights, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    delta = float(f_full) - float(f_empty)
    k, M = masks.shape
    if M == 1:
        return np.array([delta])
    G = np.zeros((M - 1, M - 1), dtype=np.float64)
    rhs = np.zeros(M - 1, dtype=np.float64)
    for b0 in range(0, k, chunk):
        m = masks[b0:b0 + chunk].astype(np.float64)
        X = m[:, :-1] - m[:, -1:]
        t = y[b0:b0 + chunk] - float(f_empty) - m[:, -1] * delta
        sw = np.sqrt(w[b0:b0 + chunk])
        A = sw[:, None] * X
        G = sla.blas.dsyrk(1.0, A, beta=1.0, c=G, trans=1, lower=0, overwrite_c=1)
        rhs += A.T @ (sw * t)
    head = sla.cho_solve(sla.cho_factor(G, lower=False, overwrite_a=True, check_finite=False), rhs,
                         check_finite=False)
    return np.concatenate([head, [delta - head.sum()]])
