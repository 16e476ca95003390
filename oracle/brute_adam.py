"""Independent binary64 Adam in the paper's form (Equation 2) -- TEST ONLY.

Written directly from Equation 2 with no reference to the binary32 oracle:
no bias correction, epsilon inside the square root, the variance of the
previous step in the denominator.  The momentum in the model update is the
freshly updated one (the reading the oracle takes for the model and buffer
lines of Algorithm 1), so that 0/1 Adam with synchronisation and variance
updates at every step, one worker and no compression must reproduce it:

    m_{t+1} = b1 m_t + (1 - b1) g_t
    x_{t+1} = x_t - gamma_t m_{t+1} / sqrt(v_t + eps)
    v_{t+1} = b2 v_t + (1 - b2) g_t^2

The hyper-parameters are taken as the binary32 numbers the optimizer
receives, then used in binary64.
"""
import numpy as np


def adam_fp64(x0, grads, gammas, beta1=0.9, beta2=0.999, eps=1e-8):
    """Run len(grads) steps; returns the list of (x, m, v) after every step."""
    b1 = float(np.float32(beta1))
    b2 = float(np.float32(beta2))
    e = float(np.float32(eps))
    x = np.asarray(x0, dtype=np.float64).copy()
    m = np.zeros_like(x)
    v = np.zeros_like(x)
    out = []
    for g, gamma in zip(grads, gammas):
        g = np.asarray(g, dtype=np.float64)
        m = b1 * m + (1.0 - b1) * g
        x = x - float(np.float32(gamma)) * m / np.sqrt(v + e)
        v = b2 * v + (1.0 - b2) * g * g
        out.append((x.copy(), m.copy(), v.copy()))
    return out


def adam_eq2_fp64(x0, grads, gammas, beta1=0.9, beta2=0.999, eps=1e-8, update_v=None):
    """Equation 2 exactly as printed, in binary64: the model update uses the
    momentum and variance of the previous step,

        m_{t+1} = b1 m_t + (1 - b1) g_t
        v_{t+1} = b2 v_t + (1 - b2) g_t^2      (only where update_v(t); else v_{t+1} = v_t)
        x_{t+1} = x_t - gamma_t m_t / sqrt(v_t + eps)

    (update_v = None updates at every step).  Returns (x, m, v) after every step."""
    b1 = float(np.float32(beta1))
    b2 = float(np.float32(beta2))
    e = float(np.float32(eps))
    x = np.asarray(x0, dtype=np.float64).copy()
    m = np.zeros_like(x)
    v = np.zeros_like(x)
    out = []
    for t, (g, gamma) in enumerate(zip(grads, gammas)):
        g = np.asarray(g, dtype=np.float64)
        x_new = x - float(np.float32(gamma)) * m / np.sqrt(v + e)
        m_new = b1 * m + (1.0 - b1) * g
        v_new = b2 * v + (1.0 - b2) * g * g if (update_v is None or update_v(t)) else v
        x, m, v = x_new, m_new, v_new
        out.append((x.copy(), m.copy(), v.copy()))
    return out

