"""Vocab reduction, joint M2T/T2T update, block bookkeeping, in-order retire
and readiness-gated admission -- Eq. 1, Eq. 2, Eq. 3, Sec. 3.1 and Alg. 1.

Plain per-request, per-block, per-row loops in float64.  The state of request
b is ``gen_start, prompt_len, n_blocks, L, R, active, eos_hit``; block g covers
absolute positions ``gen_start + g*bl + [0, bl)``; ``pe[b][g]`` counts the
post-edit steps block g has taken and ``fin[b][g]`` is its locally-finished
flag (Sec. 3.1, last sentences of "Joint M2T-T2T decoding").

Readings of silent or ambiguous points (the package docstring lists them):
Delta excludes masked positions unless ``edit_masked``; a prediction equal to
mask_id is never written; rho uses the masked set before the update; fin is
sticky; a block admitted in this step has rho = 0; an empty window after
retirement admits one block unconditionally (Alg. 1 admits B_0 that way).
"""
import numpy as np

BAND = 1e-5


def vocab_reduce(z):
    """Per row of float64 logits z [n, V]: the top-1 prediction
    x_hat = min{v : z_v = max z} and its softmax confidence
    p = exp(max z) / sum_v exp(z_v) = 1 / sum_v exp(z_v - max z)  (Eq. 1 symbols).
    """
    z = np.asarray(z, dtype=np.float64)
    m = z.max(axis=1)
    xhat = np.empty(z.shape[0], dtype=np.int64)
    for r in range(z.shape[0]):
        xhat[r] = np.flatnonzero(z[r] == m[r])[0]
    p = 1.0 / np.exp(z - m[:, None]).sum(axis=1)
    return xhat, p


def _gt(conf32, tau):
    """Threshold compare in the kernel's precision: the float32 confidence,
    widened exactly to float64, against the float64 threshold."""
    return float(conf32) > tau


def _ge(conf32, tau):
    return float(conf32) >= tau


def copy_state(state):
    return {k: np.array(v, copy=True) for k, v in state.items()}


def denoise_update(xhat, p64, tokens, state, pe, fin, packed, params):
    """One application of Alg. 1's loop body after the forward.

    xhat, p64 : per packed row (the layout of ``packed``), from vocab_reduce
    tokens    : int64 [B, T_max]; not modified (a copy is returned)
    state     : dict of per-request int arrays; pe, fin: int [B, n_max]
    params    : dict tau_mask, tau_edit, theta, mask_id, eos_id, S_pe, W,
                edit_masked (bool), force_progress (bool), sync_window (bool:
                one window shared by the batch, the synchronous variant that
                the Sec. 5 ablation compares HWP with)
    returns dict: tokens, conf (float32 per row, 0 for dead rows),
                  argmax (per row, -1 for dead rows), state, pe, fin,
                  stats (per request), band_rows, band_reqs
    """
    bl = packed["bl"]
    tm, te, theta = params["tau_mask"], params["tau_edit"], params["theta"]
    mask_id, eos_id = params["mask_id"], params["eos_id"]
    S_pe, W = params["S_pe"], params["W"]
    edit_masked = params.get("edit_masked", False)
    force = params.get("force_progress", False)

    tokens = np.array(tokens, copy=True)
    st = copy_state(state)
    pe = np.array(pe, copy=True)
    fin = np.array(fin, copy=True)
    cap = len(packed["row_req"])
    conf = np.zeros(cap, dtype=np.float32)
    argmax = np.full(cap, -1, dtype=np.int64)
    B = len(st["L"])
    stats = [dict(m2t=0, t2t=0, committed=0, spawned=0, eos=0, done=0, rho=-1.0)
             for _ in range(B)]
    band_rows = []

    tiles_of = [[] for _ in range(B)]
    for t in packed["tiles"]:
        tiles_of[t["b"]].append(t)

    rho_of = [None] * B
    for b in range(B):
        tl = tiles_of[b]
        rho = {}
        # --- Eq. 1 on every live block, then Eq. 2 / Sec. 3.1 bookkeeping ---
        for t in tl:
            g = t["g"]
            rows = range(t["row0"], t["row0"] + bl)
            x_old = {}
            for r in rows:
                pos = packed["row_pos"][r]
                c32 = np.float32(p64[r])
                conf[r] = c32
                argmax[r] = xhat[r]
                if abs(p64[r] - tm) < BAND or abs(p64[r] - te) < BAND:
                    band_rows.append(r)
                x = int(tokens[b, pos])
                x_old[r] = x
                masked = x == mask_id
                prompt = pos < st["prompt_len"][b]
                in_gamma = masked and _gt(c32, tm) and xhat[r] != mask_id
                in_delta = ((edit_masked or not masked) and not prompt
                            and xhat[r] != x and _gt(c32, te)
                            and xhat[r] != mask_id)
                if in_gamma or in_delta:
                    tokens[b, pos] = xhat[r]
                    if masked:
                        stats[b]["m2t"] += 1
                    else:
                        stats[b]["t2t"] += 1
            m_before = sum(1 for r in rows if x_old[r] == mask_id)
            revealed = sum(1 for r in rows if x_old[r] == mask_id and
                           int(tokens[b, packed["row_pos"][r]]) != mask_id)
            if force and m_before > 0 and revealed == 0:
                # Optional forced progress for a block where no masked row
                # was revealed this step (neither by Gamma nor, under
                # EDIT_MASKED, by Delta): unmask the most confident masked row
                # (ties to the lowest position) whose prediction is not [M].
                # Every masked row is then still masked, so none is counted
                # twice.
                best = None
                for r in rows:
                    if x_old[r] == mask_id and xhat[r] != mask_id:
                        if best is None or conf[r] > conf[best]:
                            best = r
                if best is not None:
                    tokens[b, packed["row_pos"][best]] = xhat[best]
                    stats[b]["m2t"] += 1
            dec = sum(1 for r in rows
                      if x_old[r] == mask_id and _ge(conf[r], tm))
            rho[g] = 1.0 if m_before == 0 else float(dec) / float(m_before)
            u = sum(1 for r in rows
                    if int(tokens[b, packed["row_pos"][r]]) != x_old[r])
            m_after = sum(1 for r in rows
                          if int(tokens[b, packed["row_pos"][r]]) == mask_id)
            if m_before == 0:                    # a post-edit step (Sec. 3.1)
                pe[b, g] += 1
                if u == 0 or pe[b, g] >= S_pe:
                    fin[b, g] = 1
            elif m_after == 0 and S_pe == 0:
                fin[b, g] = 1
        if tl:
            stats[b]["rho"] = rho[tl[-1]["g"]]
        rho_of[b] = rho

    if params.get("sync_window", False):
        _sync_retire_admit(tokens, st, pe, fin, rho_of, stats, bl, params)
    else:
        for b in range(B):
            _retire_admit(b, tokens, st, pe, fin, rho_of[b], stats, bl, params)

    band_reqs = sorted({int(packed["row_req"][r]) for r in band_rows})
    return dict(tokens=tokens, conf=conf, argmax=argmax, state=st, pe=pe,
                fin=fin, stats=stats, band_rows=sorted(band_rows),
                band_reqs=band_reqs)


def _retire_admit(b, tokens, st, pe, fin, rho, stats, bl, params):
    """Alg. 1's two inner loops for request b alone (HWP, Sec. 4.2: every
    request keeps its own window)."""
    eos_id, W, theta = params["eos_id"], params["W"], params["theta"]
    if not st["active"][b]:
        return
    n = int(st["n_blocks"][b])
    # --- in-order retirement (Alg. 1 inner while; Sec. 4.1 last para) ---
    while st["L"][b] < st["R"][b] and fin[b, st["L"][b]]:
        g = int(st["L"][b])
        st["L"][b] += 1
        stats[b]["committed"] += 1
        if eos_id >= 0:
            lo = int(st["gen_start"][b]) + g * bl
            if np.any(tokens[b, lo:lo + bl] == eos_id):
                st["active"][b] = 0
                st["eos_hit"][b] = 1
                stats[b]["eos"] = 1
                stats[b]["done"] = 1
                break
    if st["active"][b] and st["L"][b] >= n:
        st["active"][b] = 0
        stats[b]["done"] = 1
    if not st["active"][b]:
        return
    # --- gated admission (Eq. 3; Alg. 1 second inner while) ---
    if st["L"][b] == st["R"][b] and st["R"][b] < n:
        g = int(st["R"][b])
        st["R"][b] += 1
        pe[b, g] = 0
        fin[b, g] = 0
        rho[g] = 0.0
        stats[b]["spawned"] += 1
    while (st["R"][b] - st["L"][b] < W and st["R"][b] < n
           and _rho_of(rho, int(st["R"][b]) - 1, int(st["L"][b])) >= theta):
        g = int(st["R"][b])
        st["R"][b] += 1
        pe[b, g] = 0
        fin[b, g] = 0
        rho[g] = 0.0
        stats[b]["spawned"] += 1


def _sync_retire_admit(tokens, st, pe, fin, rho_of, stats, bl, params):
    """The batch-synchronous wavefront that the ablation of Sec. 5 compares
    HWP against (and Sec. 4.2 describes): all active requests share one window
    [L, R); block L retires only when it is finished in every active request
    (finished.all()), and the gate of Eq. 3 uses the smallest rho over the
    active requests.  A request whose committed block holds eos_id stops; the
    others go on.  With one request this is exactly ``_retire_admit``."""
    eos_id, W, theta = params["eos_id"], params["W"], params["theta"]
    act = [b for b in range(len(st["L"])) if st["active"][b]]
    if not act:
        return
    L, R, n = (int(st[k][act[0]]) for k in ("L", "R", "n_blocks"))
    for b in act:
        if (int(st["L"][b]), int(st["R"][b]), int(st["n_blocks"][b])) != (L, R, n):
            raise ValueError("a synchronous wavefront needs one shared window")
    # --- retirement: the shared block L goes when every active request finished it
    while L < R and act and all(fin[b, L] for b in act):
        g = L
        L += 1
        still = []
        for b in act:
            st["L"][b] = L
            stats[b]["committed"] += 1
            lo = int(st["gen_start"][b]) + g * bl
            if eos_id >= 0 and np.any(tokens[b, lo:lo + bl] == eos_id):
                st["active"][b] = 0
                st["eos_hit"][b] = 1
                stats[b]["eos"] = 1
                stats[b]["done"] = 1
            else:
                still.append(b)
        act = still
    if L >= n:
        for b in act:
            st["active"][b] = 0
            stats[b]["done"] = 1
        act = []
    if not act:
        return
    # --- admission gated by the minimum readiness over the batch (Eq. 3)
    def admit(R):
        for b in act:
            pe[b, R] = 0
            fin[b, R] = 0
            rho_of[b][R] = 0.0
            stats[b]["spawned"] += 1
        return R + 1
    if L == R and R < n:
        R = admit(R)
    while (R - L < W and R < n
           and min(_rho_of(rho_of[b], R - 1, L) for b in act) >= theta):
        R = admit(R)
    for b in act:
        st["R"][b] = R


def _rho_of(rho, g, L):
    """rho of block g for the gate: computed this step if g was live, 0 if it
    was admitted this step (no logits yet), 1 if committed (no masks left)."""
    if g < L:
        return 1.0
    return rho[g]
