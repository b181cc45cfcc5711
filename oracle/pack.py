"""Heterogeneous Wavefront Packing, Eq. 4 (Sec. 4.2), as a plain loop.

Each request b owns an independent wavefront [L_b, R_b) over its blocks
(Sec. 4.2, first paragraph).  Block g of request b covers the absolute
positions ``gen_start_b + g*bl + [0, bl)``; the window offset is
``o_b = gen_start_b + L_b*bl`` (the start of block L_b).  Eq. 4 gathers the
window positions ``o_b + [0, q)`` of every request into a dense batch; the
live part of the window is ``w_b = R_b - L_b`` blocks.

Two row layouts of the packed batch are produced:

* ``padded`` -- the paper's dense [B, q] batch with q = W_max*bl: request b
  owns rows ``[b*q, (b+1)*q)``; window slot s of b starts at row
  ``(b*W_max + s)*bl``.  Slots s >= w_b are padding (row maps = -1).
* ``ragged`` -- padding slots dropped: the live blocks of all requests are laid
  back to back in request order, slot s of b starting at row
  ``bl*(sum_{b'<b} w_b' + s)``; rows past the last live row are -1.

Both layouts have capacity ``B*W_max*bl`` rows.  A request takes part only when
it is active and its window is non-empty.
"""
import numpy as np

PADDED = "padded"
RAGGED = "ragged"


def validate_state(state, W_max):
    """Raise ValueError if an active request's wavefront is not well formed.

    Well formed (Alg. 1 invariants): 0 <= L <= R <= n, R - L <= W_max and
    gen_start >= 0.
    """
    B = len(state["L"])
    for b in range(B):
        if not state["active"][b]:
            continue
        L, R, n = int(state["L"][b]), int(state["R"][b]), int(state["n_blocks"][b])
        if not (0 <= L <= R <= n) or R - L > W_max or state["gen_start"][b] < 0:
            raise ValueError(f"request {b}: ill-formed wavefront L={L} R={R} n={n}")


def live_blocks(state):
    """w_b = R_b - L_b for active requests, else 0 (Sec. 4.2)."""
    B = len(state["L"])
    w = np.zeros(B, dtype=np.int64)
    for b in range(B):
        if state["active"][b]:
            w[b] = int(state["R"][b]) - int(state["L"][b])
    return w


def pack_wavefronts(state, W_max, bl, layout):
    """Eq. 4: per-row gather of every live window into one packed batch.

    Returns a dict with
      tiles   : list of dicts, one per live block (b, s), in (b, s) order, with
                b, s, g = L_b + s (absolute block index), row0 (first packed row),
                pos0 = o_b + s*bl (its first absolute position),
                o (= o_b, the frozen-prefix length) and kv_len = o_b + (s+1)*bl
                (the keys block s may see, Sec. 4.1 / Eq. 5),
      row_req : int64[B*W_max*bl], request of each packed row or -1,
      row_pos : int64[B*W_max*bl], absolute position of each packed row or -1,
      n_rows  : number of live rows (sum_b w_b*bl),
      n_tiles : number of live blocks.
    """
    validate_state(state, W_max)
    if layout not in (PADDED, RAGGED):
        raise ValueError(layout)
    B = len(state["L"])
    cap = B * W_max * bl
    row_req = np.full(cap, -1, dtype=np.int64)
    row_pos = np.full(cap, -1, dtype=np.int64)
    w = live_blocks(state)
    tiles = []
    next_ragged_block = 0
    for b in range(B):
        o_b = int(state["gen_start"][b]) + int(state["L"][b]) * bl
        for s in range(int(w[b])):
            if layout == PADDED:
                row0 = (b * W_max + s) * bl
            else:
                row0 = (next_ragged_block + s) * bl
            pos0 = o_b + s * bl
            tiles.append(dict(b=b, s=s, g=int(state["L"][b]) + s, row0=row0,
                              pos0=pos0, o=o_b, kv_len=o_b + (s + 1) * bl))
            for i in range(bl):
                row_req[row0 + i] = b
                row_pos[row0 + i] = pos0 + i
        next_ragged_block += int(w[b])
    return dict(tiles=tiles, row_req=row_req, row_pos=row_pos,
                n_rows=int(w.sum()) * bl, n_tiles=len(tiles), cap=cap,
                bl=bl, W_max=W_max, layout=layout)
