"""Rotary position embedding at absolute positions (the "absolute RoPE
position ids" of Sec. 4.2 / Fig. 2b), and the window prologue built on it:
RoPE on the live rows' queries and keys, then the Eq. 6 window KV write.
TEST INFRASTRUCTURE ONLY, like the rest of ``oracle/``.

RoPE (Su et al., "RoFormer", 2021), in the rotate-half arrangement: a head
vector x of dimension d is split into halves x[:d/2], x[d/2:]; pair j
(x_j, x_{j+d/2}) is rotated by the angle p * base^(-2j/d) for position p:

    x'_j       = x_j cos a - x_{j+d/2} sin a
    x'_{j+d/2} = x_{j+d/2} cos a + x_j sin a

All in float64.
"""
import numpy as np

from . import attention


def angles(positions, d, base):
    """float64 [len(positions), d/2]: p * base^(-2j/d)."""
    j = np.arange(d // 2, dtype=np.float64)
    inv = base ** (-2.0 * j / d)
    return np.asarray(positions, dtype=np.float64)[:, None] * inv[None, :]


def rope(x, positions, base):
    """x: float64 [n, H, d]; positions: [n].  Returns the rotated copy."""
    x = np.asarray(x, dtype=np.float64)
    d = x.shape[-1]
    a = angles(positions, d, base)[:, None, :]          # [n, 1, d/2]
    c, s = np.cos(a), np.sin(a)
    lo, hi = x[..., : d // 2], x[..., d // 2:]
    return np.concatenate([lo * c - hi * s, hi * c + lo * s], axis=-1)


def window_prologue(q, k_new, v_new, K, V, packed, base):
    """RoPE on the live rows' q and k at their absolute positions, then the
    Eq. 6 write of (rope(k), v) into the logical caches.  q, k_new, v_new are
    float64 in the packed layout; rows that are not live stay as they are.
    Returns (q_rot, K, V)."""
    live = np.flatnonzero(packed["row_req"] >= 0)
    pos = packed["row_pos"][live]
    q_rot = np.array(q, dtype=np.float64, copy=True)
    k_rot = np.array(k_new, dtype=np.float64, copy=True)
    q_rot[live] = rope(q[live], pos, base)
    k_rot[live] = rope(k_new[live], pos, base)
    K2, V2 = attention.write_window_kv(K, V, k_rot, v_new, packed)
    return q_rot, K2, V2
