"""One packed wavefront denoising step, and a multi-step driver of Alg. 1.

``wavefront_step`` chains the pieces in the order of Sec. 4.2 / Alg. 1: pack
the live windows (Eq. 4), write the fresh window KV to absolute positions
(Eq. 6), block-causal attention (Sec. 4.1, Eq. 5), then the vocab reduction
and the update / retire / admit of Alg. 1 from the step's logits.

``gwd_loop`` repeats Alg. 1's loop body with a caller-supplied deterministic
"model" in place of f_theta (test infrastructure: there are no weights here),
so loop-level properties -- W = 1 equals serial decoding, B requests stepped
together equal each stepped alone -- can be checked.
"""
import numpy as np

from . import attention, pack, update


def wavefront_step(state, tokens, pe, fin, q, k_new, v_new, K_prefix, V_prefix,
                   logits, params, W_max, bl, layout, Hq, Hkv, sm_scale=None):
    """All float inputs are float64 holding the exact values the GPU reads.

    logits: float64 [rows, V] in the packed layout (rows that are not live
    may hold anything; they are not read).
    Returns (packed, K, V, attn_out, update_result)."""
    packed = pack.pack_wavefronts(state, W_max, bl, layout)
    K, V = attention.write_window_kv(K_prefix, V_prefix, k_new, v_new, packed)
    out = attention.window_attention(q, K, V, packed, Hq, Hkv, sm_scale)
    live = np.flatnonzero(packed["row_req"] >= 0)
    xhat = np.full(packed["cap"], -1, dtype=np.int64)
    p64 = np.zeros(packed["cap"])
    if live.size:
        xh, pp = update.vocab_reduce(logits[live])
        xhat[live] = xh
        p64[live] = pp
    res = update.denoise_update(xhat, p64, tokens, state, pe, fin, packed,
                                params)
    return packed, K, V, out, res


def gwd_loop(model, state, tokens, pe, fin, params, W_max, bl, layout,
             max_steps=10_000):
    """Run Alg. 1's loop for every request until all are inactive.

    model(x_b, lo, hi) -> float64 logits [hi - lo, V] for positions [lo, hi) of
    request b given x_b[:hi] (the block-causal visibility of Sec. 4.1).
    Returns (tokens, state, steps, per-request forwards)."""
    tokens = np.array(tokens, copy=True)
    state = update.copy_state(state)
    pe = np.array(pe, copy=True)
    fin = np.array(fin, copy=True)
    B = len(state["L"])
    forwards = np.zeros(B, dtype=np.int64)
    steps = 0
    while np.any(state["active"]):
        steps += 1
        if steps > max_steps:
            raise RuntimeError("GWD loop did not finish")
        packed = pack.pack_wavefronts(state, W_max, bl, layout)
        xhat = np.full(packed["cap"], -1, dtype=np.int64)
        p64 = np.zeros(packed["cap"])
        for t in packed["tiles"]:
            z = model(tokens[t["b"]], t["pos0"], t["pos0"] + bl)
            xh, pp = update.vocab_reduce(z)
            xhat[t["row0"]:t["row0"] + bl] = xh
            p64[t["row0"]:t["row0"] + bl] = pp
        for b in range(B):
            if state["active"][b] and state["R"][b] > state["L"][b]:
                forwards[b] += 1
        res = update.denoise_update(xhat, p64, tokens, state, pe, fin, packed,
                                    params)
        tokens, state, pe, fin = res["tokens"], res["state"], res["pe"], res["fin"]
    return tokens, state, steps, forwards
