"""The GDN gate transform applied to the fused a/b gate projection (paper,
Eq. 1): per token t and head h,

    g = -exp(A_log[h]) * softplus(a[t, h] + dt_bias[h]),  alpha = exp(g),
    beta = sigmoid(b[t, h]).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Reading: the paper serves in_proj_b and in_proj_a as one fused GEMM in that
order (section 6), so the fused output has the H b-columns first and the H
a-columns after them; the transform replaces each by beta and alpha.  Both are
evaluated in float64 with the numerically stable forms
softplus(x) = log(1 + e^x) = logaddexp(0, x) and sigmoid(x) = 1 / (1 + e^-x).
"""

import numpy as np


def softplus(x):
    return np.logaddexp(0.0, np.asarray(x, dtype=np.float64))


def sigmoid(x):
    x = np.asarray(x, dtype=np.float64)
    e = np.exp(-np.abs(x))
    return np.where(x >= 0, 1.0 / (1.0 + e), e / (1.0 + e))


def gdn_gates(y_ba, a_log, dt_bias):
    """(M, 2H) fused b|a projection output -> (M, 2H) beta|alpha."""
    y = np.asarray(y_ba, dtype=np.float64)
    h = y.shape[1] // 2
    beta = sigmoid(y[:, :h])
    g = -np.exp(np.asarray(a_log, dtype=np.float64))[None, :] * softplus(y[:, h:] + np.asarray(dt_bias, np.float64)[None, :])
    return np.concatenate([beta, np.exp(g)], axis=1)
