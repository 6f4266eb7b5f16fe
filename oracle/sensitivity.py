"""Stage-1 sensitivity and the host refinements of the allocation inputs
(oracle).

Sensitivity (Alg. 1 Stage 1; Sec. 3.3 "Sensitivity Estimation"; Appendix
"Temporal aggregation"): the weight of component i (one kv-head's keys or
values) is the squared gradient norm of the loss with respect to that
head's cache, averaged over the T positions and over the calibration
sequences:
    w_i = (1/S) sum_s (1/T) sum_t || dL / dK_{s,i,t} ||^2 .
The gradients are inputs here (the paper takes them from a backward pass in
fp32); the sums are taken exactly enough in fp64.

Refinements:
  * weight cap (Appendix "Failure modes", mitigation of extreme outliers):
    w_i <- min(w_i, c * mean(w)) with c = 5, the mean taken over the
    uncapped weights, summed in index order;
  * fit fallback (Appendix "Distortion Model Parameters", outlier heads):
    a component whose fit has R^2 below 0.96 takes beta_i <- min(beta_i,
    mean(beta)), the mean over all components' fitted beta, summed in index
    order.
"""
import numpy as np


def sensitivity(grads):
    """grads: float array [S][n_comp][T][d] -> w float64[n_comp]."""
    g = np.asarray(grads, dtype=np.float64)
    S, _, T, _ = g.shape
    per_seq = np.sum(g * g, axis=(2, 3)) / T        # [S][n_comp]
    return np.sum(per_seq, axis=0) / S


def _mean_in_order(x):
    s = 0.0
    for v in x:
        s += float(v)
    return s / len(x)


def cap_weights(w, factor=5.0):
    """w_i <- min(w_i, factor * mean(w))."""
    w = np.asarray(w, dtype=np.float64)
    c = factor * _mean_in_order(w)
    return np.minimum(w, c)


def fallback_beta(beta, r2, r2_min=0.96):
    """beta_i <- min(beta_i, mean(beta)) where r2_i < r2_min."""
    beta = np.asarray(beta, dtype=np.float64)
    r2 = np.asarray(r2, dtype=np.float64)
    m = _mean_in_order(beta)
    return np.where(r2 < r2_min, np.minimum(beta, m), beta)
