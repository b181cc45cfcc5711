"""GPU parity of the window prologue (fb_window_prologue): absolute-position
RoPE on the live rows' queries and keys fused with the Eq. 6 write, against
the oracle's float64 rotation and write; then the attention on the rotated
queries and cache against the oracle's attention.

Tolerance of a rotated value: its rounding to the dtype (2^-8 relative for
bf16, 2^-23 for fp32) plus the float32 products with cos/sin rounded to float
(a few 2^-24 of the pair's magnitude)."""
import numpy as np
import pytest
import torch

from oracle import attention as oatt
from oracle import rope as orope
from paper_2607_17652_amd import binding as fb

from harness import ATTN_TOL, OracleCase, gather_kv, log, setup

pytestmark = pytest.mark.gpu

BASE = 10000.0


def rot_tol(ref, pair_mag, dtype):
    rel = 2.0 ** -8 if dtype == "bf16" else 2.0 ** -23
    return rel * np.abs(ref) + 8 * 2.0 ** -24 * pair_mag + 1e-30


def pair_mag(x):
    d = x.shape[-1]
    m = np.sqrt(x[..., : d // 2] ** 2 + x[..., d // 2:] ** 2)
    return np.concatenate([m, m], axis=-1)


@pytest.mark.parametrize("name,reqs,overrides", [
    ("tiny", None, {}),
    ("single", None, {}),
    ("hetero64", list(range(0, 64, 9)), {}),                 # padded rows
    ("long8", [1, 6], {}),                                    # positions up to ~33K
    ("single", None, dict(d=64, Hq=8, Hkv=2, prefix_jitter=11)),   # unaligned window
])
def test_window_prologue_matches_oracle(name, reqs, overrides):
    wl, host, t, step = setup(name, seed=12, **overrides)
    reqs = list(range(wl.B)) if reqs is None else reqs
    log(f"[prologue] {name} {overrides} reqs={reqs}")
    case = OracleCase(wl, host, t, reqs, step.page_table)     # inputs copied before the run
    q_in = t["q"].clone()
    q_out = torch.full_like(t["q"], 3.0)
    step.pack_step()
    fb.fb_window_prologue(q_in, q_out, t["k_new"], t["v_new"], t["k_cache"], t["v_cache"],
                          step.page_table, step.pack, step.shape, BASE)
    fb.fb_wavefront_attention(q_out, t["k_cache"], t["v_cache"], step.page_table, step.pack,
                              step.shape, step.out, step.attn_ws)
    torch.cuda.synchronize()
    assert torch.equal(q_in, t["q"])                          # input untouched
    assert fb.fb_pack_read_status(step.pack)["code"] == fb.FB_DERR_NONE
    q_rot, K2, V2 = orope.window_prologue(case.q, case.k_new, case.v_new, case.K_pre,
                                          case.V_pre, case.sub_packed, BASE)
    out = oatt.window_attention(q_rot, K2, V2, case.sub_packed, wl.Hq, wl.Hkv)
    full_live = case.full_packed["row_req"] >= 0
    dead = torch.from_numpy(np.flatnonzero(~full_live)).cuda()
    if len(dead):
        assert torch.all(q_out[dead] == 3.0)                  # dead rows not written
    worst = 0.0
    for i, b in enumerate(case.reqs):
        rf, rs = case.map_rows[i]
        if len(rf):
            g = q_out[torch.from_numpy(rf).cuda()].double().cpu().numpy()
            tol = rot_tol(q_rot[rs], pair_mag(case.q[rs]), wl.dtype)
            assert np.all(np.abs(g - q_rot[rs]) <= tol), f"q req {b}"
            a = step.out[torch.from_numpy(rf).cuda()].double().cpu().numpy()
            err = float(np.max(np.abs(a - out[rs])))
            worst = max(worst, err)
            assert err <= ATTN_TOL[wl.dtype], f"attention req {b}: {err}"
        T = case.K_pre[i].shape[0]
        Kg, Vg = gather_kv(t["k_cache"], t["v_cache"], step.page_table[b], T, wl.page_size)
        assert np.array_equal(Vg, V2[i]), f"V cache req {b}"
        o, w = case.T_need[i]
        # outside the window the K cache is untouched, inside it is rope(k)
        assert np.array_equal(Kg[:o], case.K_pre[i][:o]), f"K prefix req {b}"
        assert np.array_equal(Kg[o + w * wl.bl:], case.K_pre[i][o + w * wl.bl:])
        if w:
            win = slice(o, o + w * wl.bl)
            kn = np.stack([case.k_new[r] for r in rs])
            tol = rot_tol(K2[i][win], pair_mag(kn), wl.dtype)
            assert np.all(np.abs(Kg[win] - K2[i][win]) <= tol), f"K window req {b}"
    log(f"[prologue] {name}: attention after the prologue max err {worst:.2e}")


def test_window_prologue_in_place():
    wl, host, t, step = setup("single", seed=13)
    log("[prologue] in place")
    q2 = t["q"].clone()
    step.pack_step()
    fb.fb_window_prologue(q2, q2, t["k_new"], t["v_new"], t["k_cache"], t["v_cache"],
                          step.page_table, step.pack, step.shape, BASE)
    q3 = torch.empty_like(t["q"])
    k2 = t["k_cache"].clone()
    v2 = t["v_cache"].clone()
    fb.fb_window_prologue(t["q"], q3, t["k_new"], t["v_new"], k2, v2,
                          step.page_table, step.pack, step.shape, BASE)
    torch.cuda.synchronize()
    live = torch.from_numpy(np.flatnonzero(
        step.pack.view()["row_req"].cpu().numpy() >= 0)).cuda()
    assert torch.equal(q2[live], q3[live])
