"""Serial block-wise decoding (the LLaDA-2.1 baseline of Sec. 5.1), written
independently of ``pack``/``attention``/``update``.

Alg. 1 with W = 1 keeps exactly one live block, admits the next block only
when the previous one has been retired, and gives that block the visibility of
serial block-wise decoding (Sec. 4.1, "In-order retirement": the retiring
block's visibility matches serial decoding).  This module is that serial
decoder, one block at a time, so tests can check the W = 1 reduction.
"""
import math

import numpy as np


def serial_block_attention(q_blk, K_b, V_b, lo, bl, Hq, Hkv, sm_scale=None):
    """Attention of the queries of the block starting at absolute position lo
    over keys [0, lo + bl) -- the committed prefix plus the block itself,
    bidirectional inside the block.  Row by row, head by head, with an explicit
    loop over keys for the softmax normaliser.

    q_blk: float64 [bl, Hq, d]; K_b, V_b: float64 [T, Hkv, d] (logical)."""
    _, _, d = q_blk.shape
    scale = sm_scale if sm_scale is not None else 1.0 / math.sqrt(d)
    g = Hq // Hkv
    n_keys = lo + bl
    out = np.zeros_like(q_blk)
    for i in range(bl):
        for h in range(Hq):
            c = h // g
            scores = [scale * float(np.dot(q_blk[i, h], K_b[j, c]))
                      for j in range(n_keys)]
            top = max(scores)
            weights = [math.exp(s - top) for s in scores]
            total = math.fsum(weights)
            acc = np.zeros(d)
            for j in range(n_keys):
                acc += (weights[j] / total) * V_b[j, c]
            out[i, h] = acc
    return out


def _top1(row):
    """Top-1 index (first maximum) and its softmax probability, by plain loops."""
    best, best_v = 0, row[0]
    for v in range(1, len(row)):
        if row[v] > best_v:
            best, best_v = v, row[v]
    total = math.fsum(math.exp(z - best_v) for z in row)
    return best, 1.0 / total


def serial_decode(model, x, prompt_len, gen_start, n, bl, params,
                  max_forwards=10_000):
    """Decode one sequence block by block.

    model(x, lo, hi, gen_start=...) -> float64 logits [hi - lo, V] for
    positions [lo, hi) given the context x[:hi].  Each block is refined by the joint M2T/T2T rule
    (Eq. 1) until it is locally finished (Sec. 3.1): once it has no masks, up
    to S_pe post-edit steps, stopping early after a step with no change.  The
    block then commits; a committed eos_id ends decoding.
    Returns (final tokens, number of forwards, number of committed blocks).
    """
    x = np.array(x, copy=True)
    tm, te = params["tau_mask"], params["tau_edit"]
    M, eos, S_pe = params["mask_id"], params["eos_id"], params["S_pe"]
    edit_masked = params.get("edit_masked", False)
    forwards = 0
    committed = 0
    for g in range(n):
        lo = gen_start + g * bl
        post_edits = 0
        while True:
            z = model(x, lo, lo + bl, gen_start=gen_start)
            forwards += 1
            if forwards > max_forwards:
                raise RuntimeError("serial decoder did not converge")
            had_mask = any(int(x[lo + i]) == M for i in range(bl))
            changed = 0
            new = x.copy()
            for i in range(bl):
                pos = lo + i
                k, p = _top1(z[i])
                p32 = float(np.float32(p))
                cur = int(x[pos])
                if k == M:
                    continue
                if cur == M and p32 > tm:
                    new[pos] = k
                    changed += 1
                elif ((edit_masked or cur != M) and pos >= prompt_len
                      and k != cur and p32 > te):
                    new[pos] = k
                    changed += 1
            x = new
            if not had_mask:
                post_edits += 1
                if changed == 0 or post_edits >= S_pe:
                    break
            elif S_pe == 0 and not any(int(x[lo + i]) == M for i in range(bl)):
                break
        committed += 1
        if eos >= 0 and any(int(x[lo + i]) == eos for i in range(bl)):
            break
    return x, forwards, committed
