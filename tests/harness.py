"""Shared helpers of the GPU parity tests: run the HIP step through the C ABI,
gather its paged caches with the test's own indexing code, build the oracle
problem for a set of requests and compare.

The oracle side never sees a value produced by the HIP path: its inputs are
the generated tensors (copied to the host before the GPU step runs) and the
host-side request state."""
import sys

import numpy as np
import torch

from oracle import pack as opack
from oracle import step as ostep
from paper_2607_17652_amd import binding as fb
from paper_2607_17652_amd import synth
from paper_2607_17652_amd.runner import WavefrontStep

ATTN_TOL = {"bf16": 1e-2, "f32": 1e-5}
# Confidence: relative to the float64 value.  The kernel sums the row's
# exponentials in float32 with at most about 60 roundings in sequence (up to
# 40 groups of 8 per thread, the pairwise sum of a group, the wave and
# workgroup merges, the partition merge and the final reciprocal), each
# within 2^-24 relative on positive terms, plus one-ulp exp2 results: about
# 4e-6 at worst; 5e-6 covers it.  The floor only matters for p near 1/V.
CONF_RTOL = 5e-6
CONF_ATOL = 1e-12


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def setup(name, seed=0, host_edit=None, kv_split=0, **overrides):
    """Workload, host state, device tensors and a WavefrontStep."""
    wl = synth.workload(name, **overrides)
    host = synth.make_host_state(wl, seed)
    if host_edit is not None:
        host_edit(wl, host)
    t = synth.make_device_tensors(wl, host, seed, device="cuda")
    step = WavefrontStep(wl, host, t, kv_split=kv_split)
    return wl, host, t, step


# ------------------------------------------------------------- gathering ----
def gather_kv(k_cache, v_cache, pt_row, T, ps):
    """Logical [T, Hkv, d] float64 K and V of one request from the paged
    caches (K: [page][head][slot][d]; V: [page][head][d][slot])."""
    if T == 0:
        d = k_cache.shape[-1]
        z = np.zeros((0, k_cache.shape[1], d))
        return z, z
    pos = torch.arange(T, device=k_cache.device)
    pages = pt_row[(pos // ps)].long()
    slot = pos % ps
    K = k_cache[pages, :, slot, :]
    V = v_cache[pages, :, :, slot]
    return K.double().cpu().numpy(), V.double().cpu().numpy()


def state_subset(state, reqs):
    return {k: np.asarray(v)[reqs].copy() for k, v in state.items()}


def rows_by_pos(packed, b):
    r = np.flatnonzero(packed["row_req"] == b)
    return r[np.argsort(packed["row_pos"][r])]


class OracleCase:
    """Oracle inputs for a subset `reqs` of a workload's requests, taken from
    the generated tensors before the GPU step runs (the live rows' logits are
    copied to host memory then), and the oracle's whole step on them."""

    def __init__(self, wl, host, t, reqs, page_table):
        self.wl = wl
        self.reqs = list(reqs)
        st = host["state"]
        self.full_packed = opack.pack_wavefronts(st, wl.W_max, wl.bl, wl.layout)
        self.sub_state = state_subset(st, self.reqs)
        self.sub_packed = opack.pack_wavefronts(self.sub_state, wl.W_max, wl.bl,
                                                opack.RAGGED)
        cap = self.sub_packed["cap"]
        self.q = np.zeros((cap, wl.Hq, wl.d))
        self.k_new = np.zeros((cap, wl.Hkv, wl.d))
        self.v_new = np.zeros((cap, wl.Hkv, wl.d))
        self.map_rows = []          # (full rows, sub rows) per request
        full_of_sub = np.full(cap, -1, dtype=np.int64)
        for i, b in enumerate(self.reqs):
            rf = rows_by_pos(self.full_packed, b)
            rs = rows_by_pos(self.sub_packed, i)
            self.map_rows.append((rf, rs))
            full_of_sub[rs] = rf
            if len(rf):
                idx = torch.from_numpy(rf).cuda()
                self.q[rs] = t["q"][idx].double().cpu().numpy()
                self.k_new[rs] = t["k_new"][idx].double().cpu().numpy()
                self.v_new[rs] = t["v_new"][idx].double().cpu().numpy()
        # the live rows' logits, in the sub pack's row order, kept in their
        # own dtype on the host (widened to float64 a group at a time)
        live = np.flatnonzero(full_of_sub >= 0)
        self.logit_slot = np.full(cap, -1, dtype=np.int64)
        self.logit_slot[live] = np.arange(live.size)
        self.logits_host = t["logits"][torch.from_numpy(full_of_sub[live]).cuda()].cpu()
        self.T_need = []
        self.K_pre, self.V_pre = [], []
        for b in self.reqs:
            o = int(st["gen_start"][b] + st["L"][b] * wl.bl)
            w = int(st["R"][b] - st["L"][b]) if st["active"][b] else 0
            # the window plus two blocks past it (which must stay untouched)
            T = min(int(st["gen_start"][b] + st["n_blocks"][b] * wl.bl),
                    o + (w + 2) * wl.bl, host["max_pages"] * wl.page_size)
            K, V = gather_kv(t["k_cache"], t["v_cache"], page_table[b], T,
                             wl.page_size)
            self.K_pre.append(K)
            self.V_pre.append(V)
            self.T_need.append((o, w))
        self.tokens = host["tokens"][self.reqs].copy()
        self.pe = host["pe"][self.reqs].copy()
        self.fin = host["fin"][self.reqs].copy()

    def logits_rows(self, rows):
        """float64 logits of sub-pack rows (all live)."""
        slot = self.logit_slot[rows]
        assert np.all(slot >= 0)
        return self.logits_host[torch.from_numpy(slot)].double().numpy()

    def run(self, params, attention=True):
        wl = self.wl
        r = ostep.wavefront_step(self.sub_state, self.tokens, self.pe, self.fin,
                                 self.q, self.k_new, self.v_new, self.K_pre,
                                 self.V_pre, self.logits_rows, params, wl.W_max,
                                 wl.bl, opack.RAGGED, wl.Hq, wl.Hkv,
                                 with_attention=attention)
        self.K, self.V, self.out = r["K"], r["V"], r["out"]
        self.xhat, self.p64, self.upd = r["xhat"], r["p64"], r["update"]
        return self


# ------------------------------------------------------------ GPU results ---
def gpu_results(step):
    wl = step.wl
    view = step.pack.view()
    out = dict(
        header=view["header"].cpu().numpy().copy(),
        tiles=view["tiles"].cpu().numpy().copy(),
        req_w=view["req_w"].cpu().numpy().copy(),
        req_row0=view["req_row0"].cpu().numpy().copy(),
        row_req=view["row_req"].cpu().numpy().copy(),
        row_pos=view["row_pos"].cpu().numpy().copy(),
        row_tok=view["row_tok"].cpu().numpy().copy(),
        conf=step.conf.cpu().numpy().copy(),
        argmax=step.argmax.cpu().numpy().copy(),
        tokens=step.tokens.cpu().numpy().copy(),
        pe=step.pe.cpu().numpy().copy(),
        fin=step.fin.cpu().numpy().copy(),
        st=synth.state_from_records(step.st.cpu().numpy()),
        stats=fb.stats_to_numpy(step.stats, wl.B).copy(),
    )
    return out


# ------------------------------------------------------------- comparison ---
def compare_pack(wl, host, g, tokens_before):
    """The HIP pack equals the oracle's Eq. 4 pack bit for bit."""
    p = opack.pack_wavefronts(host["state"], wl.W_max, wl.bl, wl.layout)
    assert g["header"][0] == p["n_rows"]
    assert g["header"][1] == p["n_tiles"]
    assert g["header"][2] == 0x7fffffff
    assert np.array_equal(g["row_req"], p["row_req"])
    assert np.array_equal(g["row_pos"], p["row_pos"])
    tok = np.where(p["row_req"] >= 0,
                   tokens_before[np.maximum(p["row_req"], 0),
                                 np.maximum(p["row_pos"], 0)], -1)
    assert np.array_equal(g["row_tok"], tok)
    st = host["state"]
    for k, t in enumerate(p["tiles"]):
        w = int(st["R"][t["b"]] - st["L"][t["b"]])
        exp = [t["b"], t["s"], t["g"], t["row0"], t["pos0"], t["o"], t["kv_len"], w]
        assert list(g["tiles"][k]) == exp, (k, list(g["tiles"][k]), exp)


def compare_case(wl, case, g, step, check_attention=True, check_kv=True):
    """Compare the GPU step with the oracle on the case's requests.
    Returns a summary dict (max attention error, band requests)."""
    upd = case.upd
    band_sub = set(upd["band_reqs"])
    summary = dict(attn_max_err=0.0, band_requests=[case.reqs[i] for i in band_sub],
                   rows=0, conf_max_rel=0.0)
    for i, b in enumerate(case.reqs):
        rf, rs = case.map_rows[i]
        summary["rows"] += len(rf)
        if len(rf):
            # vocab reduction: argmax exact, confidence to fp32 accuracy
            assert np.array_equal(g["argmax"][rf], upd["argmax"][rs]), f"argmax req {b}"
            p64 = case.p64[rs]
            err = np.abs(g["conf"][rf].astype(np.float64) - p64)
            summary["conf_max_rel"] = max(summary["conf_max_rel"],
                                          float(np.max(err / p64)))
            assert np.all(err <= CONF_RTOL * p64 + CONF_ATOL), \
                f"conf req {b}: max rel {np.max(err / p64):.3e}"
            if check_attention:
                d = np.max(np.abs(step.out[torch.from_numpy(rf).cuda()].double()
                                  .cpu().numpy() - case.out[rs]))
                summary["attn_max_err"] = max(summary["attn_max_err"], float(d))
                assert d <= ATTN_TOL[wl.dtype], f"attention req {b}: {d}"
        if check_kv:
            o, w = case.T_need[i]
            T = case.K_pre[i].shape[0]
            K, V = gather_kv(step.t["k_cache"], step.t["v_cache"],
                             step.page_table[b], T, wl.page_size)
            assert np.array_equal(K, case.K[i]), f"K cache req {b}"
            assert np.array_equal(V, case.V[i]), f"V cache req {b}"
        if i in band_sub:
            continue
        assert np.array_equal(g["tokens"][b], upd["tokens"][i]), f"tokens req {b}"
        assert np.array_equal(g["pe"][b], upd["pe"][i]), f"pe req {b}"
        assert np.array_equal(g["fin"][b], upd["fin"][i]), f"fin req {b}"
        for k in ("L", "R", "active", "eos_hit"):
            assert g["st"][k][b] == upd["state"][k][i], f"state {k} req {b}"
        gs, os_ = g["stats"][b], upd["stats"][i]
        for k in ("m2t", "t2t", "committed", "spawned", "eos", "done"):
            assert gs[k] == os_[k], f"stats {k} req {b}: {gs[k]} vs {os_[k]}"
        assert gs["rho_frontier"] == os_["rho"], f"rho req {b}"
        assert gs["valid"] == 1
    return summary
