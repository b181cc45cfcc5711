"""Window KV write-back (Eq. 6) and W-shaped block-causal attention (Sec. 4.1).

All arrays are float64 and *logical*: request b's keys and values are
``K[b], V[b]`` of shape ``[T_b, Hkv, d]`` indexed by absolute position, which is
exactly the absolute KV layout of Sec. 4.2 ("each row storing KV at its
absolute positions").  How a cache is paged in memory is not the oracle's
concern: the caller gathers pages into these arrays with its own code.
"""
import numpy as np


def write_window_kv(K, V, k_new, v_new, packed):
    """Eq. 6: scatter the fresh window K/V of every live packed row to its
    absolute position, ``data[b, o_b + delta] <- present[row]``.

    K, V        : lists of float64 arrays [T_b, Hkv, d] (copied, not modified)
    k_new, v_new: float64 [rows, Hkv, d] in the packed row layout
    packed      : the result of ``pack.pack_wavefronts``
    Positions outside the live windows -- in particular the frozen prefix
    [0, o_b) -- are left untouched (Sec. 4.2: committed KV is never modified).
    """
    K = [k.copy() for k in K]
    V = [v.copy() for v in V]
    for r in range(len(packed["row_req"])):
        b = packed["row_req"][r]
        if b < 0:
            continue
        p = packed["row_pos"][r]
        K[b][p] = k_new[r]
        V[b][p] = v_new[r]
    return K, V


def block_attention(q_blk, K_vis, V_vis, sm_scale):
    """softmax(sm_scale * q k^T) v over the visible keys, for one block and one
    query head; q_blk [rows, d], K_vis/V_vis [kv_len, d].  Plain definition:
    max-subtracted exponentials normalised by their sum."""
    S = sm_scale * (q_blk @ K_vis.T)                 # [rows, kv_len]
    S = S - S.max(axis=1, keepdims=True)
    P = np.exp(S)
    P = P / P.sum(axis=1, keepdims=True)
    return P @ V_vis


def window_attention(q, K, V, packed, Hq, Hkv, sm_scale=None):
    """Sec. 4.1 / Eq. 5: every query row of window block s of request b attends
    to keys ``[0, kv_len)`` with ``kv_len = o_b + (s+1)*bl`` -- the committed
    prefix [0, o_b) plus live blocks L_b..L_b+s, bidirectionally inside its own
    block and never to a later block.

    q      : float64 [rows, Hq, d] in the packed layout
    K, V   : logical per-request arrays after the window write (Eq. 6)
    returns: float64 [rows, Hq, d]; rows that are not live stay 0.
    Query head h reads kv-head h // (Hq // Hkv); sm_scale defaults to 1/sqrt(d).
    """
    rows, _, d = q.shape
    if Hq % Hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    g = Hq // Hkv
    if sm_scale is None:
        sm_scale = 1.0 / np.sqrt(d)
    out = np.zeros((rows, Hq, d), dtype=np.float64)
    for t in packed["tiles"]:
        b, kv_len, r0 = t["b"], t["kv_len"], t["row0"]
        bl = packed["bl"]
        for h in range(Hq):
            c = h // g
            out[r0:r0 + bl, h] = block_attention(
                q[r0:r0 + bl, h], K[b][:kv_len, c], V[b][:kv_len, c], sm_scale)
    return out


def attention_weights(q_row, K_vis, sm_scale):
    """The softmax weights of one query over its visible keys (used by the
    sum-to-one pin)."""
    S = sm_scale * (K_vis @ q_row)
    S = S - S.max()
    P = np.exp(S)
    return P / P.sum()
