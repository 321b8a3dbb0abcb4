"""Adam in fp64 -- test infrastructure, never called by the product path.

The paper's experiments train every model with Adam and no weight decay
(appendix on experimental settings); it names the optimizer only through
its citation of Kingma & Ba, "Adam: A Method for Stochastic Optimization"
(ICLR 2015), whose Algorithm 1 this module follows:

    m_k = beta1 m_{k-1} + (1 - beta1) g_k          (first moment)
    v_k = beta2 v_{k-1} + (1 - beta2) g_k^2        (second moment)
    mhat = m_k / (1 - beta1^k),  vhat = v_k / (1 - beta2^k)
    theta_k = theta_{k-1} - lr mhat / (sqrt(vhat) + eps)

with the defaults that paper recommends (beta1 = 0.9, beta2 = 0.999,
eps = 1e-8) and k counting from 1.
"""

import numpy as np

from .layers import as_f64

BETA1, BETA2, EPS = 0.9, 0.999, 1e-8


def adam(W, dW, m, v, step, lr, beta1=BETA1, beta2=BETA2, eps=EPS):
    """One Adam step; returns (W', m', v').  ``step`` is k >= 1."""
    if step < 1:
        raise ValueError("Adam step counts from 1")
    g = as_f64(dW)
    m1 = beta1 * as_f64(m) + (1.0 - beta1) * g
    v1 = beta2 * as_f64(v) + (1.0 - beta2) * g * g
    mhat = m1 / (1.0 - beta1 ** step)
    vhat = v1 / (1.0 - beta2 ** step)
    return as_f64(W) - lr * mhat / (np.sqrt(vhat) + eps), m1, v1
