"""Local update (Eq. (6)) and the on-device AdamW of Sec. III-C.

SGD: theta <- theta - lr * g (Eq. (6), with the derivative of the local
loss; the printed derivative of f_k is read as that of L_k).
AdamW with bias correction and decoupled weight decay on the pre-update
value: m <- b1 m + (1-b1) g; v <- b2 v + (1-b2) g^2;
theta <- theta - lr * (m/(1-b1^t) / (sqrt(v/(1-b2^t)) + eps) + wd * theta),
t counting from 1.
"""
import numpy as np


def adamw_step_ref(theta, g, m, v, t, lr, b1, b2, eps, wd):
    theta = np.asarray(theta, np.float64)
    g = np.asarray(g, np.float64)
    m = b1 * np.asarray(m, np.float64) + (1.0 - b1) * g
    v = b2 * np.asarray(v, np.float64) + (1.0 - b2) * g * g
    mhat = m / (1.0 - b1 ** t)
    vhat = v / (1.0 - b2 ** t)
    new = theta - lr * (mhat / (np.sqrt(vhat) + eps) + wd * theta)
    return new, m, v


def sgd_step_ref(theta, g, lr):
    return np.asarray(theta, np.float64) - lr * np.asarray(g, np.float64)
