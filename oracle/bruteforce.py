"""Eq. 5 applied literally, on the paper's own physical tail layout.

An independent route to the window attention output, used to pin
``attention.window_attention``.  It follows Sec. 4.2 as printed:

* every request row b of the batch has one physical KV buffer of a shared
  length C; the frozen prefix sits at its absolute positions [0, o_b);
* the fresh window KV of the current forward ("present") sits in the shared
  physical tail [t, t+q) with t = C - q and q = W*bl; window slot delta holds
  position o_b + delta;
* the region [o_b, t) is the "stale middle" -- filled here with random junk
  that a correct mask must never let through;
* the dense mask M[b, i, j] = [j < o_b] or [t <= j < t + (s+1)*bl] with
  s = floor(i / bl) (Eq. 5) is materialised and applied before a dense
  softmax over all C keys.

Nothing here uses the kv_len rule of ``attention`` or the Eq. 6 write-back.
"""
import numpy as np


def dense_mask(o_b, t, q, bl, C):
    """M[i, j] of Eq. 5 for one batch row, as a bool array [q, C]."""
    M = np.zeros((q, C), dtype=bool)
    for i in range(q):
        s = i // bl
        for j in range(C):
            M[i, j] = (j < o_b) or (t <= j < t + (s + 1) * bl)
    return M


def tail_layout_attention(q_win, K_prefix, V_prefix, k_win, v_win, o, w, W, bl,
                          Hq, Hkv, sm_scale=None, junk_seed=12345):
    """Dense masked attention on the physical tail layout.

    q_win      : list over requests of float64 [w_b*bl, Hq, d], window queries
                 in slot order (slot delta = position o_b + delta)
    K_prefix   : list of float64 [>= o_b, Hkv, d] logical prefix keys
    k_win      : list of float64 [w_b*bl, Hkv, d] fresh window keys, slot order
    o, w       : per-request prefix length and live block count
    W          : window capacity (q = W*bl physical tail slots)
    returns    : list of float64 [w_b*bl, Hq, d]
    """
    B = len(o)
    q_len = W * bl
    C = int(max(o)) + q_len
    t = C - q_len
    rng = np.random.default_rng(junk_seed)
    g = Hq // Hkv
    out = []
    for b in range(B):
        d = K_prefix[b].shape[-1]
        scale = sm_scale if sm_scale is not None else 1.0 / np.sqrt(d)
        # Physical buffer: junk everywhere, then prefix and window tail.
        Kp = rng.normal(0.0, 3.0, size=(C, Hkv, d))
        Vp = rng.normal(0.0, 3.0, size=(C, Hkv, d))
        Kp[:o[b]] = K_prefix[b][:o[b]]
        Vp[:o[b]] = V_prefix[b][:o[b]]
        nlive = w[b] * bl
        Kp[t:t + nlive] = k_win[b]
        Vp[t:t + nlive] = v_win[b]
        M = dense_mask(int(o[b]), t, q_len, bl, C)
        res = np.zeros((nlive, Hq, d))
        for i in range(nlive):
            for h in range(Hq):
                c = h // g
                S = scale * (Kp[:, c, :] @ q_win[b][i, h])
                S = np.where(M[i], S, -np.inf)
                P = np.exp(S - S.max())
                P = P / P.sum()
                res[i, h] = P @ Vp[:, c, :]
        out.append(res)
    return out
