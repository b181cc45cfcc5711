"""The last layer of the forward f_theta in Alg. 1 -- the LM head Z = H W^T --
followed by the vocabulary reduction of Eq. 1's symbols, as the plain
definition.  TEST INFRASTRUCTURE ONLY, like the rest of ``oracle/``.

hidden: float64 [n, D] (the rows' final hidden states), weight: float64 [V, D]
(one row per vocabulary id, the usual [out, in] layout of a linear layer).
Z = hidden @ weight.T in float64, then ``update.vocab_reduce`` row by row:
x_hat = lowest index of the maximum, p = 1 / sum_v exp(z_v - max z).

``accumulation_bound`` gives, per row, a bound on how far a float32
evaluation of any logit of the row may be from the exact one (the standard
bound gamma_D * sum_i |h_i w_i| with gamma_D = D u / (1 - D u), u = 2^-24;
Higham, "Accuracy and Stability of Numerical Algorithms", Sec. 3.1), so a
test can tell a genuine difference from rounding.
"""
import numpy as np

from . import update


def lm_logits(hidden, weight):
    return np.asarray(hidden, dtype=np.float64) @ np.asarray(weight, dtype=np.float64).T


def lmhead_reduce(hidden, weight):
    """(x_hat, p) per row of Z = hidden @ weight^T."""
    return update.vocab_reduce(lm_logits(hidden, weight))


def accumulation_bound(hidden, weight):
    """Per row: gamma_D * max_v sum_i |h_i w_vi|."""
    hidden = np.abs(np.asarray(hidden, dtype=np.float64))
    weight = np.abs(np.asarray(weight, dtype=np.float64))
    D = hidden.shape[1]
    u = 2.0 ** -24
    gamma = D * u / (1.0 - D * u)
    return gamma * (hidden @ weight.T).max(axis=1)
