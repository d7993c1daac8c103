"""The blocks and sampler of the paper's synthetic model (test infrastructure).

Sec. 5 (Experiments) defines the synthetic setup: every block is an MLP with
hidden width 2D and a GELU activation, and the sampler makes the next
token's input the last layer's output at the current position plus noise.
Weights are random (they do not affect the run time).  Readings where the
text is silent:

* GELU is the exact form x * Phi(x) = x/2 * (1 + erf(x / sqrt 2)) (not the
  tanh approximation);
* each MLP is Linear(D -> 2D) with bias, GELU, Linear(2D -> D) with bias,
  no residual connection; weights in the [out][in] layout;
* with layers m = 0..M-1 (mixer m reads y^m = a^m and emits z^m), the block
  gives a^{m+1}_t = MLP_m(z^m_t); the sampler gives the first token
  a^0_0 = eps_0 and a^0_{t+1} = a^M_t + eps_{t+1} (Alg. 3's sampler line).

fp64 throughout; erf is scipy's.
"""
from __future__ import annotations

import numpy as np
from scipy.special import erf


def gelu(x):
    """x * Phi(x), Phi the standard normal CDF."""
    x = np.asarray(x, dtype=np.float64)
    return 0.5 * x * (1.0 + erf(x / np.sqrt(2.0)))


def mlp(x, w_up, b_up, w_down, b_down):
    """One block on rows x [..., D]: w_up [2D, D], b_up [2D], w_down [D, 2D],
    b_down [D] -> [..., D]."""
    x = np.asarray(x, dtype=np.float64)
    hidden = gelu(x @ np.asarray(w_up, np.float64).T + np.asarray(b_up, np.float64))
    return hidden @ np.asarray(w_down, np.float64).T + np.asarray(b_down, np.float64)


def mlp_chain(weights, eps, M, B, D):
    """Input rule (see ``oracle.feedback``) of the synthetic model.

    weights: (w_up [M, 2D, D], b_up [M, 2D], w_down [M, D, 2D], b_down [M, D]);
    eps: sampler noise [L, B, D].  Columns of a layer are c = b*D + d.
    """
    w_up, b_up, w_down, b_down = (np.asarray(a, dtype=np.float64) for a in weights)
    eps = np.asarray(eps, dtype=np.float64)

    def block(m, z):
        return mlp(z.reshape(B, D), w_up[m], b_up[m], w_down[m], b_down[m]).reshape(B * D)

    def rule(t, m, z_now, z_prev):
        if m == 0:
            if t == 0:
                return eps[0].reshape(B * D)
            return block(M - 1, z_prev[M - 1]) + eps[t].reshape(B * D)
        return block(m - 1, z_now[m - 1])

    return rule


def activations(z, weights, B, D):
    """Block outputs a^{m+1}_t = MLP_m(z^m_t) of every layer: z [L, M, B*D]
    mixer outputs -> [L, M, B*D]."""
    w_up, b_up, w_down, b_down = (np.asarray(a, dtype=np.float64) for a in weights)
    z = np.asarray(z, dtype=np.float64)
    L, M, C = z.shape
    out = np.empty_like(z)
    for m in range(M):
        out[:, m] = mlp(z[:, m].reshape(L, B, D), w_up[m], b_up[m], w_down[m],
                        b_down[m]).reshape(L, C)
    return out
