"""Input rules that decide y^m_t online (test infrastructure).

The synthetic workloads replace each model block by an elementwise chain
(a stand-in for the MLP blocks and sampler of the paper's synthetic model,
Sec. 5):

* layer 0, position 0:  y^0_0 = x^0_0
* layer 0, position t:  y^0_t = 0.5 * tanh(z^{M-1}_{t-1}) + x^0_t
  (the "sampler": the next token's input comes from the last layer's output)
* layer m >= 1:         y^m_t = 0.5 * tanh(z^{m-1}_t) + x^m_t
  (the "block" between mixers, Alg. 2 / Alg. 3: a^l_i = block(b^l_i))

With M = 1 this is y_0 = x_0, y_{t+1} = 0.5 tanh(z_t) + x_{t+1}.

A rule is called as ``rule(t, m, z_now, z_prev)`` where ``z_now`` holds the
outputs of layers < m at position t and ``z_prev`` the outputs of all layers
at t-1 (None at t = 0); it returns y^m_t for every column of layer m.
"""
from __future__ import annotations

import numpy as np


def teacher_forced(y):
    """Inputs fixed in advance: y[t, m, ...] (no dependence on z)."""
    y = np.asarray(y, dtype=np.float64)

    def rule(t, m, z_now, z_prev):
        return y[t, m]

    return rule


def tanh_chain(x, M):
    """The chained rule above, with additive inputs x[t, m, ...]."""
    x = np.asarray(x, dtype=np.float64)

    def rule(t, m, z_now, z_prev):
        if m == 0:
            if t == 0:
                return x[0, 0]
            return 0.5 * np.tanh(z_prev[M - 1]) + x[t, 0]
        return 0.5 * np.tanh(z_now[m - 1]) + x[t, m]

    return rule
