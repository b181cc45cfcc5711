"""GPU parity of the LM head with the fused vocabulary reduction
(fb_lmhead_reduce): argmax and confidence of every sampled live row against
the oracle's float64 product and reduction, then the whole update
(fb_denoise_apply) on those results against the oracle's update.

The kernel accumulates the logits in float32, the oracle exactly, so a row's
logits may differ by up to the accumulation bound E of the oracle
(gamma_D * max_v sum |h w|).  Where the oracle's top two logits are closer than
2E either index is a correct argmax: the test checks the kernel's choice is
within 2E of the maximum and leaves that row's decisions out, as it does for
confidences within the error of a threshold."""
import numpy as np
import pytest
import torch

from oracle import lmhead as olm
from oracle import pack as opack
from oracle import update as oupd
from paper_2607_17652_amd import binding as fb
from paper_2607_17652_amd import synth
from paper_2607_17652_amd.runner import WavefrontStep

from harness import gpu_results, log

pytestmark = pytest.mark.gpu


def oracle_rows(hid, weight, rows, chunk=16384):
    """x_hat, p, top-2 gap and accumulation bound of the given rows, in float64,
    with the product taken over vocabulary chunks."""
    H = hid[torch.from_numpy(rows).cuda()].double().cpu().numpy()
    V = weight.shape[0]
    bound = np.zeros(len(rows))
    Z_parts = []
    for v0 in range(0, V, chunk):
        Wc = weight[v0:v0 + chunk].double().cpu().numpy()
        Z_parts.append(olm.lm_logits(H, Wc))
        bound = np.maximum(bound, olm.accumulation_bound(H, Wc))
    Z = np.concatenate(Z_parts, axis=1)
    xhat, p = oupd.vocab_reduce(Z)
    srt = np.sort(Z, axis=1)
    m, second = srt[:, -1], srt[:, -2]
    return dict(Z=Z, xhat=xhat, p=p, gap=m - second, bound=bound)


def run_case(name, V, D, seed, sample=None, edit=None, **overrides):
    wl = synth.workload(name, V=V, **overrides)
    host = synth.make_host_state(wl, seed)
    log(f"[lmhead] {name} V={V} D={D} B={wl.B} rows={wl.row_cap}")
    t = synth.make_device_tensors(wl, host, seed, device="cuda", with_logits=False)
    step = WavefrontStep(wl, host, dict(t, logits=None))
    hid, weight = synth.make_lmhead_tensors(wl, D, seed)
    if edit is not None:
        edit(hid, weight)
    lm_ws = torch.empty(fb.fb_lmhead_workspace_bytes(step.pack, V, D), dtype=torch.uint8,
                        device="cuda")
    tokens_before = host["tokens"].copy()
    step.pack_step()
    fb.fb_lmhead_reduce(hid, weight, step.pack, lm_ws, step.upd_ws)
    fb.fb_denoise_apply(V, step.tokens, step.conf, step.argmax, step.st, step.pe, step.fin,
                        step.pack, step.params, step.stats, step.upd_ws)
    torch.cuda.synchronize()
    g = gpu_results(step)
    packed = opack.pack_wavefronts(host["state"], wl.W_max, wl.bl, wl.layout)
    live = np.flatnonzero(packed["row_req"] >= 0)
    rows = live if sample is None else np.sort(
        np.random.default_rng(seed).choice(live, size=min(sample, len(live)), replace=False))
    o = oracle_rows(hid, weight, rows)
    # argmax: exact where unique beyond the accumulation error, else near-max
    tie = o["gap"] <= 2 * o["bound"]
    ga = g["argmax"][rows]
    assert np.array_equal(ga[~tie], o["xhat"][~tie])
    for i in np.flatnonzero(tie):
        assert o["Z"][i, ga[i]] >= o["Z"][i].max() - 2 * o["bound"][i]
    # confidence: p moves by at most a factor e^(2E) under logit errors <= E,
    # plus the float32 sum over the vocabulary
    tol = o["p"] * (np.expm1(2 * o["bound"]) + 2e-5)
    err = np.abs(g["conf"][rows].astype(np.float64) - o["p"])
    assert np.all(err <= tol), float(np.max(err / tol))
    log(f"[lmhead] {name}: rows {len(rows)}, near ties {int(tie.sum())}, "
        f"max conf err {float(err.max()):.2e}, max bound {float(o['bound'].max()):.2e}")
    return wl, host, packed, g, rows, o, tie, tokens_before


@pytest.mark.parametrize("name,V,D,sample", [
    ("single", 5003, 512, None),          # partial last vocabulary tile, one token tile
    ("hetero64", 157184, 2048, 96),       # padded rows, full vocabulary
    ("long8", 157184, 1024, 64),
])
def test_lmhead_reduce_matches_oracle(name, V, D, sample):
    run_case(name, V, D, seed=3, sample=sample)


def test_lmhead_workgroups_that_take_two_blocks():
    """52 requests of four live blocks: 6656 rows = 26 token tiles, for which
    the partition choice on a 256-CU device asks for 26 x 88 = 2288 blocks,
    more than the 2048 workgroups launched, so 240 workgroups run a second
    block (the grid-stride path)."""
    run_case("long8", 157184, 512, seed=5, sample=64, B=52, prefix=("uniform", 64, 512))


@pytest.mark.parametrize("tied", [
    # lowest copy in the first 16-id group of its lane; copies in both lane
    # halves, both waves of a tile, another tile and the last partition
    [13, 14, 17, 45, 141, 269],
    # lowest copy in the third group of its lane (ids 69 and 101 share a lane:
    # groups 2 and 3), more in the other wave and the next tile
    [69, 101, 229, 325],
])
def test_lmhead_exact_ties_take_the_lowest_id(tied):
    """Vocabulary rows of W made equal to 256 e_0 and every hidden state given
    h_0 = 1: each row's logits then hold exact maxima of 256 (one nonzero
    product, so no rounding on either side) at the tied ids and the last id.
    The argmax is the lowest of them on every row."""

    def edit(hid, weight):
        V = weight.shape[0]
        ids = torch.tensor(tied + [V - 1], device=weight.device)
        hid[:, 0] = 1.0
        weight[ids] = 0
        weight[ids, 0] = 256.0

    wl, host, packed, g, rows, o, tie, tok0 = run_case(
        "hetero64", 157184, 256, seed=6, sample=96, edit=edit, B=16,
        prefix=("uniform", 64, 512))
    lo = min(tied)
    assert np.all(o["xhat"] == lo) and np.all(o["gap"] == 0)
    assert np.all(g["argmax"][rows] == lo)
    assert np.all(o["Z"][:, lo] == 256.0)


def test_lmhead_reduce_then_update_matches_oracle_update():
    """On a whole small workload: the update applied to the fused reduction
    equals the oracle's update on the oracle's (x_hat, p), outside rows whose
    decisions rounding could flip."""
    V, D = 4099, 256
    wl, host, packed, g, rows, o, tie, tok0 = run_case(
        "hetero64", V, D, seed=5, B=16, prefix=("uniform", 64, 512))
    cap = packed["cap"]
    xhat = np.full(cap, -1)
    p64 = np.zeros(cap)
    xhat[rows], p64[rows] = o["xhat"], o["p"]
    res = oupd.denoise_update(xhat, p64, tok0, host["state"], host["pe"], host["fin"], packed,
                              wl.params())
    unsure = set()
    tol = o["p"] * (np.expm1(2 * o["bound"]) + 2e-5)
    prm = wl.params()
    for i, r in enumerate(rows):
        near = min(abs(o["p"][i] - prm["tau_mask"]), abs(o["p"][i] - prm["tau_edit"]))
        if tie[i] or near <= tol[i]:
            unsure.add(int(packed["row_req"][r]))
    checked = 0
    for b in range(wl.B):
        if b in unsure:
            continue
        checked += 1
        assert np.array_equal(g["tokens"][b], res["tokens"][b]), b
        for k in ("L", "R", "active"):
            assert g["st"][k][b] == res["state"][k][b], (b, k)
        assert np.array_equal(g["fin"][b], res["fin"][b]), b
    log(f"[lmhead] update compared on {checked} of {wl.B} requests")
    assert checked >= wl.B // 2
