"""TEST INFRASTRUCTURE ONLY -- reference definitions of the training-step
operations around the path (used by tests/, never by the product path).

Plain fp64 numpy, written from the definitions:
* L1 photometric loss sum_k |C_k - C*_k| and its gradient sign(C_k - C*_k)
  (0 where equal), the upstream gradient of the backward.
* Adam (Kingma and Ba, "Adam: A Method for Stochastic Optimization",
  Algorithm 1): m_t = b1 m_{t-1} + (1 - b1) g_t, v_t = b2 v_{t-1} +
  (1 - b2) g_t^2, m_hat = m_t / (1 - b1^t), v_hat = v_t / (1 - b2^t),
  p_t = p_{t-1} - lr m_hat / (sqrt(v_hat) + eps).
"""
import numpy as np


def l1_loss_grad(image, target):
    """(sign(image - target), sum |image - target|) in fp64."""
    d = np.asarray(image, np.float64) - np.asarray(target, np.float64)
    return np.sign(d), float(np.abs(d).sum())


def adam_step(p, g, m, v, t, lr, b1, b2, eps):
    """One Adam step at iteration t >= 1; returns new (p, m, v) in fp64."""
    p, g, m, v = (np.asarray(a, np.float64) for a in (p, g, m, v))
    m = b1 * m + (1.0 - b1) * g
    v = b2 * v + (1.0 - b2) * g * g
    m_hat = m / (1.0 - b1 ** t)
    v_hat = v / (1.0 - b2 ** t)
    return p - lr * m_hat / (np.sqrt(v_hat) + eps), m, v
