"""GPU parity of the multi-step decode loop (Alg. 1's outer loop) on the
synthetic model, through the C ABI: the synthetic logits and embeddings bit
for bit, whole decodes (tokens, windows, step and forward counts) against the
oracle's loop, the batch-synchronous window of the Sec. 5 ablation, graph
replay, and the attention leg (caches bit for bit, last-step output within
the attention tolerance)."""
import numpy as np
import pytest
import torch

from oracle import pack as opack
from oracle import step as ostep
from oracle import synth_model as osm
from paper_2607_17652_amd import binding as fb
from paper_2607_17652_amd import synth
from paper_2607_17652_amd.runner import DecodeLoop, WavefrontStep

from harness import ATTN_TOL, gather_kv, log

pytestmark = pytest.mark.gpu


def params(V, **kw):
    p = dict(tau_mask=0.9, tau_edit=0.8, theta=0.5, mask_id=V - 1, eos_id=-1,
             S_pe=2, W=2, edit_masked=False, force_progress=False, sync_window=False)
    p.update(kw)
    return p


# ------------------------------------------------------ synthetic model ----
@pytest.mark.parametrize("name,V,dtype", [("single", 1000, "bf16"),
                                          ("hetero64", 5003, "f32"),
                                          ("serve256", 157184, "bf16")])
def test_synth_logits_match_oracle(name, V, dtype):
    wl = synth.workload(name, V=V, B=min(synth.workload(name).B, 16))
    host = synth.make_host_state(wl, seed=5)
    log(f"[loop] synth logits {name} V={V} {dtype}")
    t = synth.make_device_tensors(wl, host, 5, device="cuda", with_logits=False)
    step = WavefrontStep(wl, host, dict(t, logits=None))
    step.pack_step()
    seed = 0x1234_5678_9ABC_DEF0
    levels = synth.loop_levels(V)
    model = fb.make_model(seed, levels)
    cap = wl.row_cap
    ldt = torch.bfloat16 if dtype == "bf16" else torch.float32
    logits = torch.full((cap, V), -7.0, dtype=ldt, device="cuda")
    pred = torch.full((cap, 2), -1, dtype=torch.int32, device="cuda")
    fb.fb_synth_logits(step.st, step.tokens, step.pack, model, pred, logits)
    torch.cuda.synchronize()
    packed = opack.pack_wavefronts(host["state"], wl.W_max, wl.bl, wl.layout)
    g_pred = pred.cpu().numpy()
    st = host["state"]
    checked = 0
    for t_ in packed["tiles"]:
        b = t_["b"]
        exp = osm.block_predictions(seed, host["tokens"][b], t_["pos0"], t_["pos0"] + wl.bl,
                                    int(st["gen_start"][b]), V)
        got = [tuple(g_pred[t_["row0"] + i]) for i in range(wl.bl)]
        assert got == [(int(k), int(l)) for k, l in exp], (b, t_["s"])
        checked += 1
    assert checked == len(packed["tiles"]) > 0
    # whole rows: zeros with the level at k (sampled rows at the full vocabulary)
    live = np.flatnonzero(packed["row_req"] >= 0)
    rng = np.random.default_rng(0)
    for r in rng.choice(live, size=min(24, len(live)), replace=False):
        row = logits[int(r)].float().cpu().numpy()
        k, l = g_pred[r]
        exp = np.zeros(V, dtype=np.float32)
        exp[k] = levels[l]
        assert np.array_equal(row, exp), r
    dead = np.flatnonzero(packed["row_req"] < 0)
    if len(dead):
        assert torch.all(logits[torch.from_numpy(dead).cuda()].float() == -7.0)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_synth_embed_matches_oracle(dtype):
    wl = synth.workload("single", dtype=dtype, B=2, window=("uniform", 1, 3))
    host = synth.make_host_state(wl, seed=2)
    log(f"[loop] synth embed {dtype}")
    t = synth.make_device_tensors(wl, host, 2, device="cuda", with_logits=False)
    step = WavefrontStep(wl, host, dict(t, logits=None))
    step.pack_step()
    seed = 987654321
    q = torch.zeros_like(t["q"])
    kn = torch.zeros_like(t["k_new"])
    vn = torch.zeros_like(t["v_new"])
    fb.fb_synth_embed(step.pack, step.shape, seed, q, kn, vn)
    torch.cuda.synchronize()
    packed = opack.pack_wavefronts(host["state"], wl.W_max, wl.bl, wl.layout)
    live = np.flatnonzero(packed["row_req"] >= 0)[::7]
    pos = packed["row_pos"][live]
    tok = [int(host["tokens"][packed["row_req"][r], packed["row_pos"][r]]) for r in live]
    idx = torch.from_numpy(live).cuda()
    for kind, (T, H) in enumerate([(q, wl.Hq), (kn, wl.Hkv), (vn, wl.Hkv)]):
        exp = osm.embed_rows(seed, kind, pos, tok, H, wl.d)
        assert np.array_equal(T[idx].double().cpu().numpy(), exp), kind


# ------------------------------------------------------------ whole loop ----
def run_both(B, prompts, n, bl, W_max, V, prm, seed=0, layout="ragged",
             logit_dtype="bf16", use_graph=False, check_every=4, model_seed=None):
    host = synth.make_loop_host_state(B, prompts, n, bl, V, page_size=bl, seed=seed)
    levels = synth.loop_levels(V)
    ms = 1000 + seed if model_seed is None else model_seed
    model = osm.make_model(ms, levels, V)
    z = np.zeros((B, n), dtype=np.int64)
    ores = ostep.gwd_loop(model, host["state"], host["tokens"], z, z, prm, W_max, bl,
                          layout)
    loop = DecodeLoop(host, bl, W_max, V, prm, ms, levels, layout=layout,
                      logit_dtype=logit_dtype)
    stream = torch.cuda.Stream() if use_graph else None
    enq, done = loop.run(max_steps=40 * n + 40, check_every=check_every,
                         use_graph=use_graph, stream=stream)
    torch.cuda.synchronize()
    g = loop.results()
    return host, ores, g, enq, done


def assert_same_decode(ores, g, B):
    assert np.array_equal(g["tokens"], ores["tokens"])
    for k in ("L", "R", "active", "eos_hit"):
        assert np.array_equal(g["st"][k], ores["state"][k]), k
    assert np.array_equal(g["pe"], ores["pe"])
    assert np.array_equal(g["fin"], ores["fin"])
    assert g["steps"] == ores["steps"]
    assert np.array_equal(g["forwards"], ores["forwards"])


LOOP_CASES = {
    "serial": dict(B=1, prompts=[5], n=6, bl=8, W_max=1, V=1000, prm=dict(W=1)),
    "w2": dict(B=4, prompts=[3, 17, 9, 30], n=6, bl=16, W_max=2, V=1000, prm=dict(W=2)),
    "w4_padded": dict(B=6, prompts=[4, 8, 15, 16, 23, 42], n=8, bl=8, W_max=4, V=1000,
                      prm=dict(W=4, theta=0.25, S_pe=1), layout="padded"),
    "w3_f32": dict(B=3, prompts=[7, 2, 11], n=5, bl=8, W_max=3, V=777,
                   prm=dict(W=3, theta=0.25), logit_dtype="f32"),
    "sync": dict(B=4, prompts=[3, 17, 9, 30], n=6, bl=8, W_max=3, V=1000,
                 prm=dict(W=3, theta=0.25, sync_window=True)),
    "full_vocab": dict(B=2, prompts=[40, 100], n=4, bl=32, W_max=3, V=157184,
                       prm=dict(W=3, theta=0.25)),
}


@pytest.mark.parametrize("case", list(LOOP_CASES))
def test_decode_loop_matches_oracle(case):
    c = dict(LOOP_CASES[case])
    prm = params(c["V"], **c.pop("prm"))
    log(f"[loop] decode {case}")
    host, ores, g, enq, done = run_both(prm=prm, **c)
    assert done and enq >= ores["steps"]
    assert_same_decode(ores, g, c["B"])
    log(f"[loop] {case}: steps {ores['steps']}, forwards {list(ores['forwards'])}")


def test_decode_loop_graph_replay_equals_eager():
    c = dict(LOOP_CASES["w2"])
    prm = params(c["V"], **c.pop("prm"))
    log("[loop] graph replay w2")
    _, ores, g, _, done = run_both(prm=prm, use_graph=True, check_every=3, **c)
    assert done
    assert_same_decode(ores, g, c["B"])


def test_synchronous_window_with_one_request_equals_hwp_on_gpu():
    log("[loop] sync B=1")
    V = 1000
    outs = []
    for sync in (False, True):
        prm = params(V, W=3, theta=0.25, sync_window=sync)
        _, ores, g, _, done = run_both(1, [9], 6, 8, 3, V, prm, seed=4)
        assert done
        assert_same_decode(ores, g, 1)
        outs.append(g)
    assert np.array_equal(outs[0]["tokens"], outs[1]["tokens"])
    assert outs[0]["steps"] == outs[1]["steps"]


def test_decode_loop_stops_on_eos():
    """Pick as eos_id a token the oracle commits in request 0's third block:
    that request must stop there on both sides."""
    V, n, bl = 1000, 6, 8
    base = params(V, W=2)
    host = synth.make_loop_host_state(3, [5, 9, 14], n, bl, V, page_size=bl, seed=8)
    model = osm.make_model(42, synth.loop_levels(V), V)
    z = np.zeros((3, n), dtype=np.int64)
    first = ostep.gwd_loop(model, host["state"], host["tokens"], z, z, base, 2, bl, "ragged")
    eos = int(first["tokens"][0, 5 + 2 * bl + 3])
    prm = dict(base, eos_id=eos)
    log(f"[loop] eos {eos}")
    _, ores, g, _, done = run_both(3, [5, 9, 14], n, bl, 2, V, prm, seed=8, model_seed=42)
    assert ores["state"]["eos_hit"][0] == 1 and ores["state"]["L"][0] <= 3
    assert done
    assert_same_decode(ores, g, 3)


def test_synchronous_window_rejects_diverged_windows():
    """FB_SYNC_WINDOW with active requests whose windows differ: the status
    word names FB_DERR_STATE and no window moves."""
    V = 1000
    host = synth.make_loop_host_state(2, [4, 6], 4, 8, V, page_size=8, seed=1)
    host["state"]["R"][1] = 2               # request 1 has a two-block window
    loop = DecodeLoop(host, 8, 2, V, params(V, sync_window=True), 7,
                      synth.loop_levels(V))
    log("[loop] sync diverged windows")
    fb.fb_pack_wavefronts(loop.st, loop.tokens, loop.n_max, loop.T_max, loop.pack)
    fb.fb_synth_logits(loop.st, loop.tokens, loop.pack, loop.model, loop.pred, loop.logits)
    fb.fb_denoise_update(loop.logits, loop.tokens, loop.conf, loop.argmax, loop.st,
                         loop.pe, loop.fin, loop.pack, loop.params, loop.stats,
                         loop.upd_ws)
    torch.cuda.synchronize()
    status = fb.fb_pack_read_status(loop.pack)
    assert status["code"] == fb.FB_DERR_STATE
    g = loop.results()
    assert list(g["st"]["L"]) == [0, 0] and list(g["st"]["R"]) == [1, 2]


# ------------------------------------------------------- attention leg ----
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_decode_loop_with_attention_leg(dtype):
    """Every step also writes the window K/V of the synthetic embeddings and
    runs the attention: the caches end bit-identical to the oracle's (frozen
    prefixes untouched, each position holding the K/V of its last window
    write) and the last step's attention agrees within tolerance."""
    V, n, bl, W_max, B = 1000, 4, 8, 2, 3
    prompts = [5, 12, 20]
    Hq, Hkv, d = 4, 2, 32
    prm = params(V, W=2)
    host = synth.make_loop_host_state(B, prompts, n, bl, V, page_size=bl, seed=6)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(6)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    P = host["num_pages"]
    k_cache = (torch.randn((P, Hkv, bl, d), generator=gen, device="cuda") * 0.2).to(tdt)
    v_cache = (torch.randn((P, Hkv, d, bl), generator=gen, device="cuda") * 0.2).to(tdt)
    pt = torch.from_numpy(host["page_table"].astype(np.int32)).cuda()
    T = [int(p + n * bl) for p in prompts]
    K0, V0 = zip(*[gather_kv(k_cache, v_cache, pt[b], T[b], bl) for b in range(B)])
    embed_seed = 555
    levels = synth.loop_levels(V)
    log(f"[loop] attention leg {dtype}")
    loop = DecodeLoop(host, bl, W_max, V, prm, 77, levels,
                      attn=dict(Hq=Hq, Hkv=Hkv, d=d, dtype=dtype, page_size=bl,
                                k_cache=k_cache, v_cache=v_cache, embed_seed=embed_seed))
    enq, done = loop.run(max_steps=200, check_every=5)
    torch.cuda.synchronize()
    assert done
    g = loop.results()
    model = osm.make_model(77, levels, V)
    z = np.zeros((B, n), dtype=np.int64)
    kv = dict(seed=embed_seed, Hq=Hq, Hkv=Hkv, d=d, K=list(K0), V=list(V0))
    ores = ostep.gwd_loop(model, host["state"], host["tokens"], z, z, prm, W_max, bl,
                          "ragged", kv=kv)
    assert_same_decode(ores, g, B)
    for b in range(B):
        K, Vv = gather_kv(k_cache, v_cache, pt[b], T[b], bl)
        assert np.array_equal(K, ores["K"][b]), b
        assert np.array_equal(Vv, ores["V"][b]), b
    # the last step's live rows, placed by the oracle's pack of that step
    # (later no-op steps write no attention rows)
    pk = ores["packed_last"]
    assert ores["out_last"] and pk is not None
    out = loop.out.double().cpu().numpy()
    err = 0.0
    for (b, pos), o in ores["out_last"].items():
        r = np.flatnonzero((pk["row_req"] == b) & (pk["row_pos"] == pos))
        assert len(r) == 1
        err = max(err, float(np.max(np.abs(out[int(r[0])] - o))))
    log(f"[loop] attention leg {dtype}: max err {err:.3g}")
    assert err <= ATTN_TOL[dtype]
