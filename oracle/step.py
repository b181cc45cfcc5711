"""One packed wavefront denoising step, and a multi-step driver of Alg. 1.

``wavefront_step`` chains the pieces in the order of Sec. 4.2 / Alg. 1: pack
the live windows (Eq. 4), write the fresh window KV to absolute positions
(Eq. 6), block-causal attention (Sec. 4.1, Eq. 5), then the vocab reduction
and the update / retire / admit of Alg. 1 from the step's logits.

``gwd_loop`` repeats Alg. 1's loop body with a caller-supplied deterministic
"model" in place of f_theta (test infrastructure: there are no weights here),
so loop-level properties -- W = 1 equals serial decoding, B requests stepped
together equal each stepped alone, one request with a shared window equals HWP
-- can be checked.
"""
import numpy as np

from . import attention, pack, update


def wavefront_step(state, tokens, pe, fin, q, k_new, v_new, K_prefix, V_prefix,
                   logits, params, W_max, bl, layout, Hq, Hkv, sm_scale=None,
                   with_attention=True):
    """One whole step: pack (Eq. 4), window KV write (Eq. 6), block-causal
    attention over the written caches (Sec. 4.1, Eq. 5), then the vocab
    reduction and Alg. 1's update / retire / admit (Eq. 1-3).

    All float inputs are float64 holding the exact values the GPU reads;
    q, k_new, v_new are in the packed row layout of ``layout``; K_prefix and
    V_prefix are logical per-request caches [T_b, Hkv, d] (not modified).
    logits: float64 [rows, V] in the packed layout, or a callable
    ``logits(rows) -> float64 [len(rows), V]`` returning the given packed rows
    (a large step need not hold every row at once; every row is reduced on
    its own, so fetching rows in groups changes no value).  Rows that are not
    live are never read.

    Returns dict(packed, K, V, out (None without attention), xhat, p64,
    update) with ``update`` the result of ``update.denoise_update``."""
    packed = pack.pack_wavefronts(state, W_max, bl, layout)
    K, V = attention.write_window_kv(K_prefix, V_prefix, k_new, v_new, packed)
    out = None
    if with_attention:
        out = attention.window_attention(q, K, V, packed, Hq, Hkv, sm_scale)
    live = np.flatnonzero(packed["row_req"] >= 0)
    xhat = np.full(packed["cap"], -1, dtype=np.int64)
    p64 = np.zeros(packed["cap"])
    for c0 in range(0, live.size, 128):
        rows = live[c0:c0 + 128]
        z = logits(rows) if callable(logits) else logits[rows]
        xhat[rows], p64[rows] = update.vocab_reduce(z)
    res = update.denoise_update(xhat, p64, tokens, state, pe, fin, packed,
                                params)
    return dict(packed=packed, K=K, V=V, out=out, xhat=xhat, p64=p64, update=res)


def gwd_loop(model, state, tokens, pe, fin, params, W_max, bl, layout,
             max_steps=10_000, kv=None):
    """Run Alg. 1's loop for every request until all are inactive.

    model(x_b, lo, hi, gen_start=...) -> float64 logits [hi - lo, V] for
    positions [lo, hi) of request b given x_b[:hi] (the block-causal
    visibility of Sec. 4.1).  With params["sync_window"] the batch shares one
    window (the synchronous variant of the Sec. 5 ablation), else every
    request keeps its own (HWP).

    kv (optional): dict(seed, Hq, Hkv, d, K, V) -- run the window KV write
    (Eq. 6) and the attention (Sec. 4.1) of every step as well, on synthetic
    q/k/v rows (``synth_model.embed_rows`` of each live row's position and its
    token at the start of the step); K, V are the logical per-request caches
    (float64 [T, Hkv, d]), updated in place.  The attention output of the last
    step is returned under "out_last" as {(b, pos): [Hq, d]}, that step's
    packed rows under "packed_last".

    Returns dict(tokens, state, pe, fin, steps, forwards) (+ out, K, V)."""
    from . import synth_model
    tokens = np.array(tokens, copy=True)
    state = update.copy_state(state)
    pe = np.array(pe, copy=True)
    fin = np.array(fin, copy=True)
    B = len(state["L"])
    forwards = np.zeros(B, dtype=np.int64)
    steps = 0
    last_out, last_packed = {}, None
    while np.any(state["active"]):
        steps += 1
        if steps > max_steps:
            raise RuntimeError("GWD loop did not finish")
        packed = pack.pack_wavefronts(state, W_max, bl, layout)
        if kv is not None:
            live = np.flatnonzero(packed["row_req"] >= 0)
            pos = packed["row_pos"][live]
            tok = [int(tokens[packed["row_req"][r], packed["row_pos"][r]]) for r in live]
            cap = len(packed["row_req"])
            q = np.zeros((cap, kv["Hq"], kv["d"]))
            kn = np.zeros((cap, kv["Hkv"], kv["d"]))
            vn = np.zeros((cap, kv["Hkv"], kv["d"]))
            q[live] = synth_model.embed_rows(kv["seed"], 0, pos, tok, kv["Hq"], kv["d"])
            kn[live] = synth_model.embed_rows(kv["seed"], 1, pos, tok, kv["Hkv"], kv["d"])
            vn[live] = synth_model.embed_rows(kv["seed"], 2, pos, tok, kv["Hkv"], kv["d"])
            kv["K"], kv["V"] = attention.write_window_kv(kv["K"], kv["V"], kn, vn, packed)
            out = attention.window_attention(q, kv["K"], kv["V"], packed,
                                             kv["Hq"], kv["Hkv"])
            last_out = {(int(packed["row_req"][r]), int(packed["row_pos"][r])): out[r]
                        for r in live}
            last_packed = packed
        xhat = np.full(packed["cap"], -1, dtype=np.int64)
        p64 = np.zeros(packed["cap"])
        for t in packed["tiles"]:
            z = model(tokens[t["b"]], t["pos0"], t["pos0"] + bl,
                      gen_start=int(state["gen_start"][t["b"]]))
            xh, pp = update.vocab_reduce(z)
            xhat[t["row0"]:t["row0"] + bl] = xh
            p64[t["row0"]:t["row0"] + bl] = pp
        for b in range(B):
            if state["active"][b] and state["R"][b] > state["L"][b]:
                forwards[b] += 1
        res = update.denoise_update(xhat, p64, tokens, state, pe, fin, packed,
                                    params)
        tokens, state, pe, fin = res["tokens"], res["state"], res["pe"], res["fin"]
    out = dict(tokens=tokens, state=state, pe=pe, fin=fin, steps=steps,
               forwards=forwards)
    if kv is not None:
        out.update(out_last=last_out, packed_last=last_packed, K=kv["K"], V=kv["V"])
    return out
