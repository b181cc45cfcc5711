"""A deterministic stand-in for the model f_theta of Alg. 1 (the forward that
maps the visible tokens to logits), for multi-step tests of the decode loop.
TEST INFRASTRUCTURE ONLY, like the rest of ``oracle/``.

There are no trained weights here, so the loop is driven by a hash model whose
logits depend on exactly what Sec. 4.1 lets a block see: the tokens of
positions [0, lo + bl) for the block at [lo, lo + bl).  It mimics the
behaviour the paper builds on (Sec. 1, Sec. 3): a block drafted while an
upstream block is still masked may draft wrong tokens, and once the upstream
context is complete the model predicts the "true" token, so T2T edits repair
the early drafts.

Hash: SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number
generators", OOPSLA 2014) used as a counter-based generator: the n-th output
(n = 0, 1, ...) of the generator seeded with s is

    H(s, n) = mix(s + (n + 1) * GAMMA  mod 2^64),
    mix(z)  : z ^= z >> 30; z *= 0xBF58476D1CE4E5B9;
              z ^= z >> 27; z *= 0x94D049BB133111EB; z ^= z >> 31   (mod 2^64)
    GAMMA   = 0x9E3779B97F4A7C15.

Model (seed s, peak heights a[0..3] > 0, vocabulary V, mask id M = V - 1):

* token contribution     c(j, x) = H(s, j * 2^32 + x)
* true token             t(p)    = H(s, 2^63 + p) mod (V - 1)
* for the block [lo, hi = lo + bl) of a request whose block 0 starts at gen_start:
    ctx   = sum over j < hi with x_j != M of c(j, x_j)    (mod 2^64)
    stale = number of j in [gen_start, lo) with x_j == M   (upstream still masked)
    first = the lowest position of the block holding M, if any
* for each position p of the block, with h = H(ctx, p):
    k = t(p)            if stale == 0 or the top bit of h is 0
        h mod (V - 1)   otherwise (a draft from stale context)
    l = (h >> 32) mod 4, raised to 3 at p == first
    logits z_v = 0 for v != k and z_k = a[l].

Since every z_v other than z_k is 0, argmax = k (never M) and the confidence
is the closed form p = e^a / (e^a + V - 1); the heights are chosen far from
the thresholds so the kernel's float32 confidence and this float64 one decide
alike.  The raised level at ``first`` makes every forward reveal at least one
token per block with masks (a[3] > tau_mask), so the loop always ends.

Synthetic Q/K/V rows ("embeddings") for the attention inside the loop, kind
0 = q, 1 = k, 2 = v, head hd, dimension i of a row at position p holding token
x:  e = ((H(H(H(s, 2^62 + kind * 2^59 + p), x), hd * d + i) >> 56) - 128) / 256,
exact in bf16 and float32.
"""
import numpy as np

MASK64 = (1 << 64) - 1
GAMMA = 0x9E3779B97F4A7C15


def mix(z):
    """SplitMix64's output function on a Python int (mod 2^64)."""
    z &= MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


def H(seed, n):
    """The n-th output (0-based) of SplitMix64 seeded with ``seed``."""
    return mix((seed + (n + 1) * GAMMA) & MASK64)


def splitmix64_stream(seed, count):
    """The first ``count`` outputs of SplitMix64 seeded with ``seed``, by the
    generator's own state update (state += GAMMA, output mix(state))."""
    out, state = [], seed & MASK64
    for _ in range(count):
        state = (state + GAMMA) & MASK64
        out.append(mix(state))
    return out


def true_token(seed, p, V):
    return H(seed, (1 << 63) + p) % (V - 1)


def block_context(seed, x, lo, hi, gen_start, mask_id):
    """(ctx, stale, first) of the block [lo, hi) given the token row x."""
    ctx = 0
    for j in range(hi):
        xj = int(x[j])
        if xj != mask_id:
            ctx = (ctx + H(seed, (j << 32) + xj)) & MASK64
    stale = sum(1 for j in range(gen_start, lo) if int(x[j]) == mask_id)
    first = next((p for p in range(lo, hi) if int(x[p]) == mask_id), None)
    return ctx, stale, first


def block_predictions(seed, x, lo, hi, gen_start, V):
    """Per position of [lo, hi): (k, level)."""
    M = V - 1
    ctx, stale, first = block_context(seed, x, lo, hi, gen_start, M)
    preds = []
    for p in range(lo, hi):
        h = H(ctx, p)
        if stale == 0 or (h >> 63) == 0:
            k = true_token(seed, p, V)
        else:
            k = h % (V - 1)
        lvl = 3 if p == first else (h >> 32) % 4
        preds.append((k, lvl))
    return preds


def make_model(seed, levels, V):
    """model(x, lo, hi, gen_start) -> float64 logits [hi - lo, V] for the
    block [lo, hi), the interface of ``step.gwd_loop`` and ``serial``."""
    levels = [float(a) for a in levels]
    if len(levels) != 4 or min(levels) <= 0:
        raise ValueError("four positive peak heights")

    def model(x, lo, hi, gen_start=0):
        z = np.zeros((hi - lo, V))
        for i, (k, lvl) in enumerate(block_predictions(seed, x, lo, hi, gen_start, V)):
            z[i, k] = levels[lvl]
        return z
    return model


def embed_rows(seed, kind, positions, tokens, heads, d):
    """float64 [len(positions), heads, d] embeddings of (position, token) rows."""
    out = np.zeros((len(positions), heads, d))
    for r, (p, x) in enumerate(zip(positions, tokens)):
        h1 = H(seed, (1 << 62) + (kind << 59) + int(p))
        h2 = H(h1, int(x))
        for hd in range(heads):
            for i in range(d):
                out[r, hd, i] = ((H(h2, hd * d + i) >> 56) - 128) / 256.0
    return out
