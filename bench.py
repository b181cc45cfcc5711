#!/usr/bin/env python
"""Benchmark of the packed wavefront denoising step on one MI355X.

One step = pack (Eq. 4) + window KV write (Eq. 6) + block-causal attention
(Sec. 4.1, one layer) + vocab reduction and denoise update (Eq. 1-3, Alg. 1)
over one batch of a seeded synthetic workload whose inputs are resident in
HBM before timing starts.  Every timed step starts from its own copy of the
same request state, so all K steps do identical work.

Prints ONE JSON line: active tokens/s (live window tokens, never padding) of
the K steps replayed from one HIP graph (the eager loop's figures beside them,
and the headline when the replay is skipped or differs from the eager outputs),
attention % of dense bf16 MFMA peak, update HBM GB/s, per-phase times from
HIP events recorded on the launch stream, a roofline entry for the dominant
kernel, the fp64 oracle timed on a bounded sample on the host cores, and
whole decodes on the synthetic model (serial, HWP and the batch-synchronous
window) under "loop".

    python bench.py [--gpus 1] [--steps 50] [--warmup 5] [--workload serve256]
"""
import argparse
import hashlib
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "active tokens/s per wavefront step; attn % MFMA peak; update HBM GB/s"
PEAK_BF16_FLOPS = 2.5e15      # MI355X dense bf16 MFMA
PEAK_HBM_BYTES = 8.0e12       # MI355X HBM3E
PROFILES = os.path.join(ROOT, "profiles")


def parse_args():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="serve256")
    ap.add_argument("--second", default="long8",
                    help="a second workload measured the same way and reported under "
                         "its own key ('' to skip)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-graph", action="store_true",
                    help="skip the HIP-graph replay of the K steps (the headline is then "
                         "the eager loop's)")
    ap.add_argument("--cpu-budget-s", type=float, default=15.0)
    ap.add_argument("--no-cold", action="store_true",
                    help="skip the steps timed after a cache flush")
    ap.add_argument("--no-loop", action="store_true",
                    help="skip the whole-decode loop runs on the synthetic model")
    ap.add_argument("--plan-overlap", action="store_true",
                    help="run the eager loop's steps, too, with the attention's plan "
                         "(fb_attention_plan) on a second stream beside the window KV write, "
                         "then fb_wavefront_attention_planned, as the graph's steps are by "
                         "default (eager it measured equal or slower: the cross-stream events "
                         "cost more than the plan)")
    ap.add_argument("--graph-one-call", action="store_true",
                    help="capture the graph's steps with the one-call attention instead of "
                         "the plan beside the window KV write")
    ap.add_argument("--no-lmhead", action="store_true",
                    help="skip the LM head with the fused vocabulary reduction")
    ap.add_argument("--lmhead-dim", type=int, default=2048,
                    help="hidden size D of the LM-head measurement")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only run a plain 1 GiB device copy (counter calibration)")
    return ap.parse_args()


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def workload_work(wl, host):
    """Live rows, attention flops over the visible keys, and algorithmic bytes."""
    st = host["state"]
    n_live = 0
    flops = 0.0
    kv_bytes = 0.0
    elt = 2 if wl.dtype == "bf16" else 4
    for b in range(wl.B):
        if not st["active"][b]:
            continue
        w = int(st["R"][b] - st["L"][b])
        o = int(st["gen_start"][b] + st["L"][b] * wl.bl)
        n_live += w * wl.bl
        for s in range(w):
            flops += 4.0 * wl.bl * wl.Hq * wl.d * (o + (s + 1) * wl.bl)
        if w:
            kv_bytes += 2.0 * wl.Hkv * wl.d * elt * (o + w * wl.bl)
    qo_bytes = 2.0 * n_live * wl.Hq * wl.d * elt
    return n_live, flops, kv_bytes + qo_bytes


def src_sha(name):
    path = os.path.join(ROOT, "paper_2607_17652_amd", "csrc", name)
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def measured_traffic(kernel, workload, src_file):
    """HBM bytes per launch from the committed counter summary, if it was taken
    on the current kernel source; else None."""
    path = os.path.join(PROFILES, f"{kernel}_{workload}_traffic.txt")
    if not os.path.exists(path):
        return None
    try:
        with open(path) as f:
            txt = f.read()
        rec = json.loads(txt[txt.index("{"): txt.rindex("}") + 1])
    except (ValueError, OSError):
        return None
    if rec.get("src_sha") != src_sha(src_file):
        return None
    return rec.get("hbm_bytes_per_launch")


def copy_probe():
    import torch
    n = 1 << 30
    src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": n, "launches": 5}), flush=True)


def gather_kv(k_cache, v_cache, pt_row, T, ps):
    import torch
    pos = torch.arange(T, device=k_cache.device)
    pages = pt_row[pos // ps].long()
    K = k_cache[pages, :, pos % ps, :]
    V = v_cache[pages, :, :, pos % ps]
    return K.double().cpu().numpy(), V.double().cpu().numpy()


def cpu_baseline(wl, host, t, budget_s, seed):
    """Time the fp64 oracle's whole step (as it stands) on whole requests, one
    at a time, until the budget is spent; only the oracle's own computation is
    timed (inputs are copied to host memory before the clock starts)."""
    import numpy as np
    import torch
    from oracle import pack as opack
    from oracle import step as ostep
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        blas_threads = 1
    st = host["state"]
    full = opack.pack_wavefronts(st, wl.W_max, wl.bl, wl.layout)
    order = np.random.default_rng(seed + 99).permutation(wl.B)
    spent, rows_done, reqs_done = 0.0, 0, 0
    params = wl.params()
    for b in order:
        if not st["active"][b] or st["R"][b] == st["L"][b]:
            continue
        sub = {k: np.asarray(v)[[b]].copy() for k, v in st.items()}
        sp = opack.pack_wavefronts(sub, wl.W_max, wl.bl, opack.RAGGED)
        rf = np.flatnonzero(full["row_req"] == b)
        rf = rf[np.argsort(full["row_pos"][rf])]
        rs = np.flatnonzero(sp["row_req"] == 0)
        rs = rs[np.argsort(sp["row_pos"][rs])]
        idx = torch.from_numpy(rf).cuda()
        cap = sp["cap"]
        q = np.zeros((cap, wl.Hq, wl.d))
        kn = np.zeros((cap, wl.Hkv, wl.d))
        vn = np.zeros((cap, wl.Hkv, wl.d))
        q[rs] = t["q"][idx].double().cpu().numpy()
        kn[rs] = t["k_new"][idx].double().cpu().numpy()
        vn[rs] = t["v_new"][idx].double().cpu().numpy()
        z = np.zeros((cap, wl.V))
        z[rs] = t["logits"][idx].double().cpu().numpy()
        o = int(st["gen_start"][b] + st["L"][b] * wl.bl)
        T = o + int(st["R"][b] - st["L"][b]) * wl.bl
        K, V = gather_kv(t["k_cache"], t["v_cache"], torch.from_numpy(
            host["page_table"][b]).cuda(), T, wl.page_size)
        tok = host["tokens"][[b]].copy()
        pe, fin = host["pe"][[b]].copy(), host["fin"][[b]].copy()
        t0 = time.perf_counter()
        ostep.wavefront_step(sub, tok, pe, fin, q, kn, vn, [K], [V], z, params,
                             wl.W_max, wl.bl, opack.RAGGED, wl.Hq, wl.Hkv)
        spent += time.perf_counter() - t0
        rows_done += len(rs)
        reqs_done += 1
        if spent >= budget_s:
            break
    return {"value": rows_done / spent if spent > 0 else None, "unit": "tokens/s",
            "cores": int(blas_threads), "kind": "oracle",
            "sample": f"{reqs_done} of {wl.B} requests ({rows_done} live tokens) of "
                      f"{wl.name}: the oracle's whole step (pack, KV write, attention, "
                      f"vocab reduction, update) in fp64 numpy; {spent:.1f} s; matmuls "
                      f"on {blas_threads} BLAS threads, the rest on one"}


def cold_steps(torch, one_step, step, K, nph, flush_bytes=1 << 30):
    """Each of K steps timed alone (HIP events on the launch stream) right
    after 1 GiB has been written, which evicts the 256 MB last-level cache
    and the L2s: the step's inputs come from HBM.  Every step starts from a
    fresh copy of the pristine request state.  Median and mean."""
    flush = torch.empty(flush_bytes, dtype=torch.uint8, device="cuda")
    pristine = (step.st, step.tokens, step.pe, step.fin)
    times = []
    for i in range(K):
        state = tuple(x.clone() for x in pristine)
        flush.fill_(i & 255)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(nph + 1)]
        one_step(i, ev, state)
        torch.cuda.synchronize()
        times.append(ev[0].elapsed_time(ev[nph]))
    del flush
    import numpy as np
    return {"ms_per_step_median": float(np.median(times)), "ms_per_step_mean": float(np.mean(times)),
            "steps": K, "flush_bytes": flush_bytes}


def hbm_probe(torch, fb, nbytes=2 << 30, reps=5, logits=None):
    """Measured device-memory ceilings beside the 8 TB/s vendor figure, from
    the library's probes: a read-only stream with the vocabulary pass's load
    form (bytes read per second) and a plain copy (bytes read + written per
    second), each the best of `reps` launches timed with HIP events on the
    launch stream.  The read probe's XOR result is checked against the
    buffer's known contents.  With `logits` (the live rows, contiguous) the
    read probe also streams exactly the bytes the vocabulary pass reads."""
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda").fill_(0x5a)
    dst = torch.empty_like(src)
    out = torch.empty(fb.FB_PROBE_BLOCKS, dtype=torch.int32, device="cuda")

    def best(fn):
        fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) * 1e-3)
        return min(ts)

    t_read = best(lambda: fb.fb_hbm_read_probe(src, out))
    # every word is 0x5a5a5a5a and the buffer holds an even number of words,
    # so the XOR of everything read is 0
    xr = 0
    for v in out.cpu().numpy().view("u4").tolist():
        xr ^= v
    t_copy = best(lambda: fb.fb_hbm_copy_probe(src, dst))
    del src, dst
    res = {"read_GBps": nbytes / t_read / 1e9, "copy_GBps": 2 * nbytes / t_copy / 1e9,
           "read_xor_ok": xr == 0, "bytes": nbytes,
           "note": "library probes (fb_hbm_read_probe, fb_hbm_copy_probe), best of 5; "
                   "copy counts bytes read + written"}
    if logits is not None:
        lb = logits.numel() * logits.element_size()
        t_log = best(lambda: fb.fb_hbm_read_probe(logits, out))
        res["read_GBps_live_logits"] = lb / t_log / 1e9
        res["live_logit_bytes"] = lb
    return res


def graph_replay(torch, fb, step, one_step, copies, K, W, split=True):
    """The same K steps captured once in a HIP graph and replayed.

    Each captured step works on its own pristine copy of the request state,
    as in the eager loop.  With `split` the attention runs in its two-call
    form, its plan on a second stream beside the window KV write (a fork and
    join inside the graph, with no event cost at replay).  A warm-up replay runs first, the copies are
    restored outside the graph, then one timed replay between two
    synchronizations (wall clock, as the eager loop; the HIP-event interval
    of the replay is reported beside it).  Its outputs (last step's attention
    output, confidences, argmax, stats and updated state) must equal the eager
    ones bit for bit, else the figure is withheld."""
    ref = [x.clone() for x in copies[K]] + [step.out.clone(), step.conf.clone(),
                                           step.argmax.clone(), step.stats.clone()]
    pristine = (step.st, step.tokens, step.pe, step.fin)
    gcopies = [tuple(x.clone() for x in pristine) for _ in range(K)]
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for i in range(K):
            one_step(0, None, gcopies[i], overlap=split)

    def restore():
        for c in gcopies:
            for dst, src in zip(c, pristine):
                dst.copy_(src)
        torch.cuda.synchronize()

    g.replay()
    restore()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record()
    g.replay()
    e1.record()
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t0) * 1e3 / K
    ms = e0.elapsed_time(e1) / K
    got = list(gcopies[0]) + [step.out, step.conf, step.argmax, step.stats]
    same = all(torch.equal(a, b) for a, b in zip(got, ref)) and \
        all(torch.equal(a, b) for a, b in zip(gcopies[K - 1], ref[:4]))
    return {"ms_per_step": wall_ms if same else None,
            "ms_per_step_events": ms if same else None, "matches_eager": bool(same),
            "steps_per_replay": K, "plan_beside_kv_write": bool(split)}


def prologue_bench(torch, fb, step, t, reps=20):
    """The window prologue (RoPE on the live rows' Q and K at absolute
    positions + the Eq. 6 write) against the plain window KV write it
    replaces, on the step's own inputs (it rewrites the window part of the
    caches, which the step rewrites anyway)."""
    q_out = torch.empty_like(t["q"])
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    for _ in range(2):
        fb.fb_window_prologue(t["q"], q_out, t["k_new"], t["v_new"], t["k_cache"],
                              t["v_cache"], step.page_table, step.pack, step.shape)
    torch.cuda.synchronize()
    ev[0].record()
    for _ in range(reps):
        fb.fb_window_prologue(t["q"], q_out, t["k_new"], t["v_new"], t["k_cache"],
                              t["v_cache"], step.page_table, step.pack, step.shape)
    ev[1].record()
    for _ in range(reps):
        fb.fb_write_window_kv(t["k_new"], t["v_new"], t["k_cache"], t["v_cache"],
                              step.page_table, step.pack, step.shape)
    ev[2].record()
    torch.cuda.synchronize()
    return {"kernel": "rope_kv_kernel", "rope_base": 10000.0,
            "ms": ev[0].elapsed_time(ev[1]) / reps,
            "kv_write_only_ms": ev[1].elapsed_time(ev[2]) / reps}


def lmhead_bench(torch, fb, synth, wl, step, logits, n_live, D, reps=5):
    """The LM head Z = H W^T of the workload's live rows with the vocabulary
    reduction as its epilogue (fb_lmhead_reduce), against the unfused path:
    the library GEMM of torch (hipBLASLt) writing bf16 logits, then
    fb_vocab_reduce reading them."""
    hid, weight = synth.make_lmhead_tensors(wl, D, seed=1)
    lm_ws = torch.empty(fb.fb_lmhead_workspace_bytes(step.pack, wl.V, D), dtype=torch.uint8,
                        device="cuda")
    flops = 2.0 * n_live * wl.V * D
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    for _ in range(2):
        fb.fb_lmhead_reduce(hid, weight, step.pack, lm_ws, step.upd_ws)
    torch.cuda.synchronize()
    ev[0].record()
    for _ in range(reps):
        fb.fb_lmhead_reduce(hid, weight, step.pack, lm_ws, step.upd_ws)
    ev[1].record()
    torch.cuda.synchronize()
    fused_ms = ev[0].elapsed_time(ev[1]) / reps
    rows = hid[:n_live] if wl.layout == "ragged" else hid
    out = logits[:rows.shape[0]]
    for _ in range(2):
        torch.matmul(rows, weight.t(), out=out)
    torch.cuda.synchronize()
    ev[0].record()
    for _ in range(reps):
        torch.matmul(rows, weight.t(), out=out)
    ev[1].record()
    for _ in range(reps):
        fb.fb_vocab_reduce(logits, step.pack, step.upd_ws)
    ev[2].record()
    torch.cuda.synchronize()
    gemm_ms = ev[0].elapsed_time(ev[1]) / reps
    vp_ms = ev[1].elapsed_time(ev[2]) / reps
    achieved = flops / (fused_ms * 1e-3)
    return {"kernel": "lmhead_kernel + lm_merge_kernel", "D": D, "V": wl.V, "rows": n_live,
            "flops": flops, "ms": fused_ms,
            "roofline": {"bound": "mfma", "achieved": achieved / 1e12,
                         "peak": PEAK_BF16_FLOPS / 1e12, "unit": "TFLOP/s",
                         "frac": achieved / PEAK_BF16_FLOPS},
            "unfused": {"gemm_ms": gemm_ms, "gemm_tflops": flops / (gemm_ms * 1e-3) / 1e12,
                        "vocab_reduce_ms": vp_ms, "total_ms": gemm_ms + vp_ms,
                        "logit_bytes_written_and_read": 2.0 * n_live * wl.V * 2},
            "fused_over_unfused": (gemm_ms + vp_ms) / fused_ms}


LOOP_WORKLOAD = dict(name="loop64", B=64, prompt=(256, 1024), n_blocks=16, bl=32,
                     W_max=4, V=157184, Hq=32, Hkv=8, d=128, seed=0)


def loop_bench(torch, fb, synth, DecodeLoop):
    """Whole decodes (Alg. 1's outer loop on the device) of 64 requests on the
    synthetic model: serial (W = 1), HWP (W = 4) and the batch-synchronous
    window (W = 4), each timed around one fb_decode_loop call (steps replayed
    as a HIP graph, one flag read per 16 steps).  Every step runs the full
    path: pack, synthetic embeddings, window KV write, attention, synthetic
    logits over the whole vocabulary, vocab reduction and update."""
    import numpy as np
    c = LOOP_WORKLOAD
    rng = np.random.default_rng(c["seed"])
    prompts = rng.integers(c["prompt"][0], c["prompt"][1] + 1, size=c["B"])
    host0 = synth.make_loop_host_state(c["B"], prompts, c["n_blocks"], c["bl"], c["V"],
                                       page_size=c["bl"], seed=c["seed"])
    P = host0["num_pages"]
    gen = torch.Generator(device="cuda")
    gen.manual_seed(c["seed"] + 17)
    k_cache = (torch.randn((P, c["Hkv"], c["bl"], c["d"]), generator=gen, device="cuda")
               * 0.1).to(torch.bfloat16)
    v_cache = (torch.randn((P, c["Hkv"], c["d"], c["bl"]), generator=gen, device="cuda")
               * 0.1).to(torch.bfloat16)
    levels = synth.loop_levels(c["V"])
    gen_tokens = c["B"] * c["n_blocks"] * c["bl"]
    runs = {}
    for name, W, sync in (("serial", 1, False), ("hwp", 4, False), ("sync", 4, True)):
        prm = dict(tau_mask=0.9, tau_edit=0.8, theta=0.5, mask_id=c["V"] - 1, eos_id=-1,
                   S_pe=2, W=W, edit_masked=False, force_progress=False, sync_window=sync)
        attn = dict(Hq=c["Hq"], Hkv=c["Hkv"], d=c["d"], dtype="bf16", page_size=c["bl"],
                    k_cache=k_cache, v_cache=v_cache, embed_seed=c["seed"] + 5)
        loop = DecodeLoop(host0, c["bl"], c["W_max"], c["V"], prm, c["seed"] + 99, levels,
                          attn=attn)
        stream = torch.cuda.Stream()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        enq, done = loop.run(max_steps=4096, check_every=16, use_graph=True, stream=stream)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        if not done:
            raise RuntimeError(f"loop {name} did not finish in 4096 steps")
        r = loop.results()
        fw = r["forwards"].astype(np.float64)
        runs[name] = {"W": W, "sync_window": sync, "steps": r["steps"],
                      "steps_enqueued": enq, "ms": dt * 1e3,
                      "ms_per_step": dt * 1e3 / max(enq, 1),
                      "tokens_per_s": gen_tokens / dt,
                      "tpf_mean": float(np.mean(c["n_blocks"] * c["bl"] / fw))}
        print(f"[bench] loop {name}: {r['steps']} steps, {dt * 1e3:.1f} ms",
              file=sys.stderr, flush=True)
        del loop
    return {"workload": {k: v for k, v in c.items()}, "generated_tokens": gen_tokens,
            "runs": runs,
            "hwp_over_serial": runs["hwp"]["tokens_per_s"] / runs["serial"]["tokens_per_s"],
            "hwp_over_sync": runs["hwp"]["tokens_per_s"] / runs["sync"]["tokens_per_s"]}


def measure_step(torch, fb, synth, WavefrontStep, name, seed, K, W, graph=True,
                 cold=True, plan_overlap=False, graph_split=True):
    """K timed steps of one workload (after W warm-up steps), each on its own
    copy of the pristine request state.  Returns (result dict, context for the
    sections that reuse the step's buffers)."""
    import numpy as np
    wl = synth.workload(name)
    host = synth.make_host_state(wl, seed)
    t = synth.make_device_tensors(wl, host, seed, device="cuda")
    step = WavefrontStep(wl, host, t)
    n_live, flops, attn_bytes = workload_work(wl, host)
    copies = [(step.st.clone(), step.tokens.clone(), step.pe.clone(), step.fin.clone())
              for _ in range(K + W)]
    torch.cuda.synchronize()
    print(f"[bench] workload={wl.name} B={wl.B} live_tokens={n_live} "
          f"steps={K} warmup={W}", file=sys.stderr, flush=True)

    nph = 5
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(nph + 1)]
              for _ in range(K)]

    # with plan_overlap the attention's plan (it reads only the pack) runs on a
    # second stream beside the window KV write, and the attention waits for both
    main = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    packed, planned = torch.cuda.Event(), torch.cuda.Event()

    def one_step(i, ev, state=None, overlap=None):
        split = plan_overlap if overlap is None else overlap
        st, tok, pe, fin = copies[i] if state is None else state
        if ev is not None:
            ev[0].record()
        fb.fb_pack_wavefronts(st, tok, step.n_max, step.T_max, step.pack)
        if ev is not None:
            ev[1].record()
        if split:
            packed.record(main)
            side.wait_event(packed)
            fb.fb_attention_plan(step.pack, step.shape, step.attn_ws, side)
            planned.record(side)
        fb.fb_write_window_kv(t["k_new"], t["v_new"], t["k_cache"], t["v_cache"],
                              step.page_table, step.pack, step.shape)
        if ev is not None:
            ev[2].record()
        if split:
            main.wait_event(planned)
            fb.fb_wavefront_attention_planned(t["q"], t["k_cache"], t["v_cache"],
                                              step.page_table, step.pack, step.shape,
                                              step.out, step.attn_ws)
        else:
            fb.fb_wavefront_attention(t["q"], t["k_cache"], t["v_cache"],
                                      step.page_table, step.pack, step.shape,
                                      step.out, step.attn_ws)
        if ev is not None:
            ev[3].record()
        fb.fb_vocab_reduce(t["logits"], step.pack, step.upd_ws)
        if ev is not None:
            ev[4].record()
        fb.fb_denoise_apply(wl.V, tok, step.conf, step.argmax, st, pe, fin,
                            step.pack, step.params, step.stats, step.upd_ws)
        if ev is not None:
            ev[5].record()

    for i in range(W):
        one_step(K + i, None)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(K):
        one_step(i, events[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    status = fb.fb_pack_read_status(step.pack)
    if status["code"] != 0:
        raise RuntimeError(f"device status {status}")
    names = ["pack", "kv_write", "attention", "vocab_reduce", "update_apply"]
    ph = {n: float(np.mean([events[i][j].elapsed_time(events[i][j + 1])
                            for i in range(K)])) for j, n in enumerate(names)}
    ms_step = wall * 1e3 / K
    step_ms = [events[i][0].elapsed_time(events[i][nph]) for i in range(K)]
    gr = None
    if graph:
        try:
            gr = graph_replay(torch, fb, step, one_step, copies, K, W, graph_split)
        except Exception as exc:   # capture unavailable: the eager loop is the headline
            try:
                torch.cuda.synchronize()
            except Exception:
                pass
            print(f"[bench] graph replay skipped: {exc!r}", file=sys.stderr, flush=True)
            gr = {"ms_per_step": None, "matches_eager": False, "error": repr(exc)}
    cd = cold_steps(torch, one_step, step, K, nph) if cold else None
    t_attn = ph["attention"] * 1e-3
    t_voc = ph["vocab_reduce"] * 1e-3
    t_upd = (ph["vocab_reduce"] + ph["update_apply"]) * 1e-3
    elt = 2 if wl.dtype == "bf16" else 4
    nsplit = fb.fb_update_workspace_bytes(step.pack, wl.V) // (wl.row_cap * 16)
    voc_bytes = n_live * wl.V * elt + n_live * nsplit * 16
    upd_bytes = n_live * wl.V * elt + 16 * n_live
    attn_frac = flops / t_attn / PEAK_BF16_FLOPS
    voc_ach = voc_bytes / t_voc
    voc_traffic = measured_traffic("vocab_pass", wl.name, "denoise.hip")
    attn_traffic = measured_traffic("attn_bf16", wl.name, "attention.hip")
    roof_voc = {"kernel": "vocab_pass_kernel", "bound": "hbm",
                "achieved": voc_ach / 1e9, "peak": PEAK_HBM_BYTES / 1e9,
                "unit": "GB/s", "frac": voc_ach / PEAK_HBM_BYTES,
                "traffic": voc_traffic, "algorithmic_bytes": voc_bytes}
    roof_attn = {"kernel": ("fb_wavefront_attention_planned (attn_bf16+combine; the plan runs "
                            "beside the KV write)" if plan_overlap else
                            "fb_wavefront_attention (plan+attn_bf16+combine)"),
                 "bound": "mfma", "achieved": flops / t_attn / 1e12,
                 "peak": PEAK_BF16_FLOPS / 1e12, "unit": "TFLOP/s",
                 "frac": attn_frac, "traffic": attn_traffic,
                 "algorithmic_flops": flops, "algorithmic_bytes": attn_bytes,
                 "hbm_GBps_if_read_once": attn_bytes / t_attn / 1e9}
    dominant, other = (roof_voc, roof_attn) if t_voc >= t_attn else (roof_attn, roof_voc)
    # The headline is the K steps replayed from one HIP graph (how a serving
    # loop runs the step: no host launch work between kernels) when the
    # replay reproduced the eager outputs bit for bit; the eager loop's
    # figures stay beside it, and are the headline otherwise.
    eager = {"value": n_live / (ms_step * 1e-3), "ms_per_step": ms_step,
             "ms_per_step_median_events": float(np.median(step_ms))}
    use_graph = gr is not None and gr["ms_per_step"] is not None
    ms_head = gr["ms_per_step"] if use_graph else ms_step
    res = {
        "value": n_live / (ms_head * 1e-3),
        "ms_per_step": ms_head,
        "execution": "hip_graph" if use_graph else "eager",
        "eager": eager,
        "config": {"workload": wl.name, "B": wl.B, "Hq": wl.Hq, "Hkv": wl.Hkv,
                   "head_dim": wl.d, "bl": wl.bl, "W_max": wl.W_max,
                   "layout": wl.layout, "page_size": wl.page_size, "V": wl.V,
                   "live_tokens": n_live, "seed": seed,
                   "execution": "hip_graph" if use_graph else "eager"},
        "attn_pct_mfma_peak": 100.0 * attn_frac,
        "update_hbm_gbps": upd_bytes / t_upd / 1e9,
        "update_pct_hbm_peak": 100.0 * upd_bytes / t_upd / PEAK_HBM_BYTES,
        "phases_ms": ph,
        "roofline": dominant,
        "roofline_other": other,
    }
    if gr is not None:
        res["graph"] = gr
    if cd is not None:
        res["cold"] = cd
    del copies
    ctx = dict(wl=wl, host=host, t=t, step=step, n_live=n_live)
    return res, ctx


def main():
    args = parse_args()
    if args.gpus != 1:
        print(f"bench.py: the library runs one GPU per process; --gpus {args.gpus} is not "
              f"supported here (requests are independent: each GPU would run this step on "
              f"its own share of them)", file=sys.stderr)
        sys.exit(2)
    if args.copy_probe:
        copy_probe()
        return
    import torch
    from paper_2607_17652_amd import binding as fb
    from paper_2607_17652_amd import synth
    from paper_2607_17652_amd.runner import DecodeLoop, WavefrontStep

    torch.cuda.set_device(0)
    K, W = args.steps, args.warmup
    overlap = args.plan_overlap
    head, ctx = measure_step(torch, fb, synth, WavefrontStep, args.workload, args.seed,
                             K, W, graph=not args.no_graph, cold=not args.no_cold,
                             plan_overlap=overlap, graph_split=not args.graph_one_call)
    wl, host, t, step, n_live = (ctx[k] for k in ("wl", "host", "t", "step", "n_live"))
    out = {
        "metric": METRIC,
        "value": head["value"],
        "unit": "tokens/s",
        "n_gpus": 1, "steps": K, "warmup": W, "ms_per_step": head["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": wl.dtype, "data": "synthetic",
        "plan_overlap": overlap,
    }
    out.update({k: v for k, v in head.items() if k not in ("value", "ms_per_step")})
    live_logits = t["logits"][:n_live] if wl.layout == "ragged" else None
    out["hbm_probe"] = hbm_probe(torch, fb, logits=live_logits)
    if live_logits is not None:
        # the vocabulary pass against the same probe over the same bytes
        out["vocab_pct_of_read_probe"] = (100.0 * head["roofline"]["achieved"] * 1e9
                                          / (out["hbm_probe"]["read_GBps_live_logits"] * 1e9)
                                          if head["roofline"]["kernel"] == "vocab_pass_kernel"
                                          else None)
    if not args.no_cpu_baseline:
        cb = cpu_baseline(wl, host, t, args.cpu_budget_s, args.seed)
        cb["host_cpus"] = os.cpu_count()
        cb["cpu_model"] = cpu_model()
        out["cpu_baseline"] = cb
    # the sections below reuse the step's buffers (the LM head overwrites its
    # logits), so they run after everything that reads the step's inputs
    out["prologue"] = prologue_bench(torch, fb, step, t)
    if not args.no_lmhead:
        out["lmhead"] = lmhead_bench(torch, fb, synth, wl, step, t["logits"], n_live,
                                     args.lmhead_dim)
    del ctx, step, t, host
    torch.cuda.empty_cache()
    if args.second and args.second != args.workload:
        sec, sctx = measure_step(torch, fb, synth, WavefrontStep, args.second, args.seed,
                                 K, W, graph=not args.no_graph, cold=not args.no_cold,
                                 plan_overlap=overlap,
                                 graph_split=not args.graph_one_call)
        out[args.second] = sec
        del sctx
        torch.cuda.empty_cache()
    if not args.no_loop:
        out["loop"] = loop_bench(torch, fb, synth, DecodeLoop)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
