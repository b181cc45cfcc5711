"""Seeded synthetic workloads for the wavefront denoising step.

Input generation only: this module draws request states, token arrays, paged
K/V caches, queries and logits with the shapes and value distributions of the
five workloads below.  It holds none of the method's arithmetic (no packing,
no attention, no reduction, no update rule) and imports neither the HIP
binding nor the oracle, so both can be fed from it.

Workloads (FlowBlock's decoding setup: block length 32, generation length
2048, i.e. 64 blocks per request; LLaDA-2.1-mini-like head shapes):

* ``tiny``     -- 1 request, 2/2 heads, d=32, bl=4, prefix 8, W=2, fp32, V=1000
* ``single``   -- 1 request, 16/4 heads, d=128, bl=32, prefix 1024, W=3, bf16,
                  V=157184
* ``hetero64`` -- 64 requests, 16/4 heads, prefixes U[256,4096], windows
                  U{1..4} packed padded to W_max=4
* ``long8``    -- 8 requests, 32/8 heads, prefixes U[16384,32768], W=4
* ``serve256`` -- 256 requests, 32/8 heads, prefixes log-uniform [128,8192],
                  windows U{1..4}, ragged packing

Distributions: Q/K/V i.i.d. N(0,1)/sqrt(d) rounded to the compute dtype
(round-to-nearest-even); logits z = sigma_row * N(0,1) with sigma_row uniform
in [sigma_lo, sigma_hi] and, on a seeded fraction of rows, one planted peak
z_k = max(z) + 4 at k uniform over the non-mask ids; unmasked tokens uniform
over the non-mask ids; mask id = V - 1.  Prefixes are floored to a multiple of
bl (at least bl).  Request b's generation starts at gen_start_b = o_b - L_b*bl
with L_b uniform in {0 .. min(o_b/bl, n - W_max)}; the prompt is
[0, gen_start_b).  Masks in the live window: exactly half of each request's
window rows (seeded permutation) for tiny/single/long8; a per-block fraction
f ~ U[0,1] with Bernoulli(f) rows for hetero64/serve256.  Mask-free live
blocks carry pe ~ U{0..S_pe-1}; mask-free blocks that are not leftmost are
finished with probability 1/2 (so several blocks can retire in one step).
"""
from dataclasses import dataclass, replace

import numpy as np

MASK_HALF = "half"
MASK_BLOCK_UNIFORM = "block_uniform"


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    Hq: int
    Hkv: int
    d: int
    bl: int
    page_size: int
    W_max: int
    layout: str                  # "ragged" | "padded"
    dtype: str                   # "f32" | "bf16"
    V: int
    sigma: tuple
    planted: float
    prefix: tuple                # ("fixed", o) | ("uniform", lo, hi) | ("loguniform", lo, hi)
    window: tuple                # ("fixed", w) | ("uniform", lo, hi)
    mask: str
    n_blocks: int = 64
    S_pe: int = 2
    tau_mask: float = 0.9
    tau_edit: float = 0.8
    theta: float = 0.5
    eos_id: int = -1
    W: int = 0                   # admission cap; 0 means W_max
    prefix_jitter: int = 0       # adds U{0..jitter} to each prefix (unaligned)

    @property
    def mask_id(self):
        return self.V - 1

    @property
    def row_cap(self):
        return self.B * self.W_max * self.bl

    def params(self):
        return dict(tau_mask=self.tau_mask, tau_edit=self.tau_edit,
                    theta=self.theta, mask_id=self.mask_id, eos_id=self.eos_id,
                    S_pe=self.S_pe, W=self.W or self.W_max,
                    edit_masked=False, force_progress=False)


WORKLOADS = {
    "tiny": Workload("tiny", B=1, Hq=2, Hkv=2, d=32, bl=4, page_size=4,
                     W_max=2, layout="ragged", dtype="f32", V=1000,
                     sigma=(1.0, 6.0), planted=0.3, prefix=("fixed", 8),
                     window=("fixed", 2), mask=MASK_HALF, n_blocks=4),
    "single": Workload("single", B=1, Hq=16, Hkv=4, d=128, bl=32,
                       page_size=32, W_max=3, layout="ragged", dtype="bf16",
                       V=157184, sigma=(1.0, 8.0), planted=0.4,
                       prefix=("fixed", 1024), window=("fixed", 3),
                       mask=MASK_HALF),
    "hetero64": Workload("hetero64", B=64, Hq=16, Hkv=4, d=128, bl=32,
                         page_size=32, W_max=4, layout="padded", dtype="bf16",
                         V=157184, sigma=(1.0, 8.0), planted=0.4,
                         prefix=("uniform", 256, 4096), window=("uniform", 1, 4),
                         mask=MASK_BLOCK_UNIFORM),
    "long8": Workload("long8", B=8, Hq=32, Hkv=8, d=128, bl=32, page_size=32,
                      W_max=4, layout="ragged", dtype="bf16", V=157184,
                      sigma=(1.0, 8.0), planted=0.4,
                      prefix=("uniform", 16384, 32768), window=("fixed", 4),
                      mask=MASK_HALF),
    "serve256": Workload("serve256", B=256, Hq=32, Hkv=8, d=128, bl=32,
                         page_size=32, W_max=4, layout="ragged", dtype="bf16",
                         V=157184, sigma=(1.0, 8.0), planted=0.4,
                         prefix=("loguniform", 128, 8192),
                         window=("uniform", 1, 4), mask=MASK_BLOCK_UNIFORM),
}

# Order in which the workloads are listed (smallest first).
WORKLOAD_ORDER = ["tiny", "single", "hetero64", "long8", "serve256"]


def workload(name, **overrides):
    w = WORKLOADS[name]
    return replace(w, **overrides) if overrides else w


def _rng(seed, stream):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, stream])))


def _draw_prefixes(wl, rng):
    kind = wl.prefix[0]
    if kind == "fixed":
        o = np.full(wl.B, wl.prefix[1], dtype=np.int64)
    elif kind == "uniform":
        o = rng.integers(wl.prefix[1], wl.prefix[2] + 1, size=wl.B)
    elif kind == "loguniform":
        lo, hi = np.log(wl.prefix[1]), np.log(wl.prefix[2])
        o = np.exp(rng.uniform(lo, hi, size=wl.B)).astype(np.int64)
    else:
        raise ValueError(kind)
    o = np.maximum((o // wl.bl) * wl.bl, wl.bl)
    if wl.prefix_jitter:
        o = o + rng.integers(0, wl.prefix_jitter + 1, size=wl.B)
    return o


def _draw_windows(wl, rng):
    kind = wl.window[0]
    if kind == "fixed":
        return np.full(wl.B, wl.window[1], dtype=np.int64)
    return rng.integers(wl.window[1], wl.window[2] + 1, size=wl.B)


def make_host_state(wl, seed=0):
    """Request states, tokens, per-block pe/fin and the page table (numpy).

    Returns a dict with
      state      : gen_start, prompt_len, n_blocks, L, R, active, eos_hit
                   (int64 arrays of length B)
      tokens     : int64 [B, T_max]
      pe, fin    : int64 [B, n_max]
      page_table : int64 [B, max_pages] (-1 past a request's allocation)
      num_pages, T_max, n_max, o (prefix lengths), w (live blocks)
    """
    rng = _rng(seed, 1)
    B, bl, n, M = wl.B, wl.bl, wl.n_blocks, wl.mask_id
    o = _draw_prefixes(wl, rng)
    w = _draw_windows(wl, rng)
    L = np.array([rng.integers(0, max(0, min(ob // bl, n - wl.W_max)) + 1)
                  for ob in o], dtype=np.int64)
    gen_start = o - L * bl
    R = L + w
    T_need = gen_start + n * bl
    ps = wl.page_size
    T_max = int(-(-T_need.max() // ps) * ps)
    tokens = np.full((B, T_max), M, dtype=np.int64)
    pe = np.zeros((B, n), dtype=np.int64)
    fin = np.zeros((B, n), dtype=np.int64)
    for b in range(B):
        tokens[b, :o[b]] = rng.integers(0, M, size=o[b])
        nwin = int(w[b]) * bl
        win = rng.integers(0, M, size=nwin)
        if wl.mask == MASK_HALF:
            masked = np.zeros(nwin, dtype=bool)
            masked[rng.permutation(nwin)[: nwin // 2]] = True
        else:
            masked = np.zeros(nwin, dtype=bool)
            for s in range(int(w[b])):
                f = rng.uniform()
                masked[s * bl:(s + 1) * bl] = rng.uniform(size=bl) < f
        win[masked] = M
        tokens[b, o[b]:o[b] + nwin] = win
        fin[b, :L[b]] = 1
        for s in range(int(w[b])):
            if not masked[s * bl:(s + 1) * bl].any():
                pe[b, L[b] + s] = rng.integers(0, max(wl.S_pe, 1))
                if s > 0 and rng.uniform() < 0.5:
                    fin[b, L[b] + s] = 1
    pages_per_req = -(-T_need // ps)
    num_pages = int(pages_per_req.sum())
    max_pages = int(pages_per_req.max())
    perm = rng.permutation(num_pages)
    page_table = np.full((B, max_pages), -1, dtype=np.int64)
    k = 0
    for b in range(B):
        page_table[b, :pages_per_req[b]] = perm[k:k + pages_per_req[b]]
        k += pages_per_req[b]
    state = dict(gen_start=gen_start, prompt_len=gen_start.copy(),
                 n_blocks=np.full(B, n, dtype=np.int64), L=L, R=R,
                 active=np.ones(B, dtype=np.int64),
                 eos_hit=np.zeros(B, dtype=np.int64))
    return dict(state=state, tokens=tokens, pe=pe, fin=fin,
                page_table=page_table, num_pages=num_pages, T_max=T_max,
                n_max=n, o=o, w=w, max_pages=max_pages)


def torch_dtype(wl):
    import torch
    return torch.float32 if wl.dtype == "f32" else torch.bfloat16


def _normal(shape, gen, device, dtype, scale, chunk_rows=None):
    import torch
    out = torch.empty(shape, dtype=dtype, device=device)
    if chunk_rows is None:
        chunk_rows = shape[0]
    for r0 in range(0, shape[0], chunk_rows):
        r1 = min(shape[0], r0 + chunk_rows)
        x = torch.randn((r1 - r0,) + tuple(shape[1:]), generator=gen,
                        device=device, dtype=torch.float32)
        out[r0:r1] = (x * scale).to(dtype)
    return out


def make_device_tensors(wl, host, seed=0, device="cuda", with_logits=True):
    """Q, window K/V, paged K/V caches and logits as torch tensors.

    Layouts (those of the C ABI):
      q        [row_cap, Hq, d]        k_new, v_new [row_cap, Hkv, d]
      k_cache  [num_pages, Hkv, page_size, d]
      v_cache  [num_pages, Hkv, d, page_size]   (keys innermost)
      logits   [row_cap, V]
    Rows of q / k_new / v_new / logits are i.i.d., so their values do not
    depend on which packed row a position lands in.
    """
    import torch
    dt = torch_dtype(wl)
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed) * 1_000_003 + 7)
    s = 1.0 / np.sqrt(wl.d)
    cap, P = wl.row_cap, host["num_pages"]
    t = {}
    t["q"] = _normal((cap, wl.Hq, wl.d), gen, device, dt, s)
    t["k_new"] = _normal((cap, wl.Hkv, wl.d), gen, device, dt, s)
    t["v_new"] = _normal((cap, wl.Hkv, wl.d), gen, device, dt, s)
    t["k_cache"] = _normal((P, wl.Hkv, wl.page_size, wl.d), gen, device, dt, s,
                           chunk_rows=4096)
    t["v_cache"] = _normal((P, wl.Hkv, wl.d, wl.page_size), gen, device, dt, s,
                           chunk_rows=4096)
    if with_logits:
        t["logits"] = make_logits(wl, cap, gen, device)
    return t


def make_logits(wl, rows, gen, device, chunk_rows=2048):
    """[rows, V] logits: sigma_row * N(0,1), with a planted max+4 peak on a
    seeded fraction of rows at a non-mask index."""
    import torch
    dt = torch_dtype(wl)
    out = torch.empty((rows, wl.V), dtype=dt, device=device)
    lo, hi = wl.sigma
    for r0 in range(0, rows, chunk_rows):
        r1 = min(rows, r0 + chunk_rows)
        n = r1 - r0
        sig = lo + (hi - lo) * torch.rand((n, 1), generator=gen, device=device)
        z = torch.randn((n, wl.V), generator=gen, device=device) * sig
        plant = torch.rand((n,), generator=gen, device=device) < wl.planted
        k = torch.randint(0, wl.V - 1, (n,), generator=gen, device=device)
        peak = z.max(dim=1).values + 4.0
        idx = torch.nonzero(plant).flatten()
        z[idx, k[idx]] = peak[idx]
        out[r0:r1] = z.to(dt)
    return out


def host_to_device_state(host, device="cuda"):
    """int32 device copies of the integer host arrays (tokens, pe/fin as uint8,
    page table) and the packed fb_req_state records."""
    import torch
    st = host["state"]
    B = len(st["L"])
    rec = np.zeros((B, 8), dtype=np.int32)
    rec[:, 0] = st["gen_start"]
    rec[:, 1] = st["prompt_len"]
    rec[:, 2] = st["n_blocks"]
    rec[:, 3] = st["L"]
    rec[:, 4] = st["R"]
    rec[:, 5] = st["active"]
    rec[:, 6] = st["eos_hit"]
    return dict(
        req_state=torch.from_numpy(rec).to(device),
        tokens=torch.from_numpy(host["tokens"].astype(np.int32)).to(device),
        pe=torch.from_numpy(host["pe"].astype(np.uint8)).to(device),
        fin=torch.from_numpy(host["fin"].astype(np.uint8)).to(device),
        page_table=torch.from_numpy(host["page_table"].astype(np.int32)).to(device),
    )


def state_from_records(rec):
    """Inverse of the fb_req_state packing above (numpy int32 [B, 8])."""
    rec = np.asarray(rec)
    return dict(gen_start=rec[:, 0].astype(np.int64),
                prompt_len=rec[:, 1].astype(np.int64),
                n_blocks=rec[:, 2].astype(np.int64),
                L=rec[:, 3].astype(np.int64), R=rec[:, 4].astype(np.int64),
                active=rec[:, 5].astype(np.int64),
                eos_hit=rec[:, 6].astype(np.int64))


# ------------------------------------------------------- multi-step loop ----
def loop_levels(V, targets=(0.3, 0.85, 0.955, 0.99)):
    """Peak heights of the synthetic model for vocabulary V: the logit a whose
    two-level confidence e^a / (e^a + V - 1) is near each target, rounded to a
    multiple of 1/8 (exact in bf16 below 32).  The default targets sit far from
    the thresholds 0.9 / 0.8 the workloads use."""
    out = []
    for p in targets:
        a = np.log(p / (1.0 - p) * (V - 1))
        out.append(float(np.round(a * 8.0) / 8.0))
    return tuple(out)


def make_loop_host_state(B, prompts, n_blocks, bl, V, page_size, seed=0):
    """Fresh requests for a whole decode: request b has a random prompt of
    prompts[b] tokens (never the mask id V - 1), then n_blocks masked blocks
    starting at gen_start = prompt length; L = 0, R = 1 (B_0 admitted), pe =
    fin = 0.  Pages cover each request's full length, ids a seeded
    permutation.  Same dict layout as ``make_host_state``."""
    rng = _rng(seed, 11)
    M = V - 1
    prompts = np.asarray(prompts, dtype=np.int64)
    assert len(prompts) == B
    T_need = prompts + n_blocks * bl
    T_max = int(-(-T_need.max() // page_size) * page_size)
    tokens = np.full((B, T_max), M, dtype=np.int64)
    for b in range(B):
        tokens[b, :prompts[b]] = rng.integers(0, M, size=prompts[b])
    pages_per_req = -(-T_need // page_size)
    num_pages = int(pages_per_req.sum())
    max_pages = int(pages_per_req.max())
    perm = rng.permutation(num_pages)
    page_table = np.full((B, max_pages), -1, dtype=np.int64)
    k = 0
    for b in range(B):
        page_table[b, :pages_per_req[b]] = perm[k:k + pages_per_req[b]]
        k += pages_per_req[b]
    state = dict(gen_start=prompts.copy(), prompt_len=prompts.copy(),
                 n_blocks=np.full(B, n_blocks, dtype=np.int64),
                 L=np.zeros(B, dtype=np.int64), R=np.ones(B, dtype=np.int64),
                 active=np.ones(B, dtype=np.int64), eos_hit=np.zeros(B, dtype=np.int64))
    return dict(state=state, tokens=tokens,
                pe=np.zeros((B, n_blocks), dtype=np.int64),
                fin=np.zeros((B, n_blocks), dtype=np.int64),
                page_table=page_table, num_pages=num_pages, T_max=T_max,
                n_max=n_blocks, max_pages=max_pages)


# ----------------------------------------------------------- LM head ------
def make_lmhead_tensors(wl, D, seed=0, device="cuda", planted=None):
    """Hidden rows [row_cap, D] and an LM-head weight [V, D], bf16, whose
    product has the logit statistics of the workload: weight rows ~ N(0, 1/D)
    (norm about 1), hidden rows sigma_row * N(0, 1) with sigma_row ~ U[sigma],
    so a row's logits are about N(0, sigma_row^2); on a seeded fraction of rows
    (the workload's planted share) the hidden row also gets a component along
    one weight row that lifts that logit about 4 above the row's maximum."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed) * 7919 + 13)
    V, cap = wl.V, wl.row_cap
    weight = torch.empty((V, D), dtype=torch.bfloat16, device=device)
    for v0 in range(0, V, 16384):
        v1 = min(V, v0 + 16384)
        weight[v0:v1] = (torch.randn((v1 - v0, D), generator=gen, device=device)
                         / np.sqrt(D)).to(torch.bfloat16)
    lo, hi = wl.sigma
    sig = lo + (hi - lo) * torch.rand((cap, 1), generator=gen, device=device)
    hid = torch.randn((cap, D), generator=gen, device=device) * sig
    frac = wl.planted if planted is None else planted
    plant = torch.rand((cap,), generator=gen, device=device) < frac
    k = torch.randint(0, V - 1, (cap,), generator=gen, device=device)
    idx = torch.nonzero(plant).flatten()
    if len(idx):
        wk = weight[k[idx]].float()
        # the maximum of V Gaussian logits is about sigma * sqrt(2 ln V)
        lift = sig[idx, 0] * float(np.sqrt(2 * np.log(V))) + 4.0
        hid[idx] += wk * (lift / (wk * wk).sum(dim=1))[:, None]
    return hid.to(torch.bfloat16), weight
