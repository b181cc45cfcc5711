"""GPU parity of the HIP wavefront step against the fp64 oracle, through the
C ABI.  Bit-exact: packing, token ids, argmax, per-block pe/fin, request
state and statistics (requests holding a confidence within 1e-5 of a
threshold are counted and reported instead).  Attention within max-abs 1e-2
(bf16) / 1e-5 (fp32); confidences within 5e-6 relative of the fp64 value.
The oracle side of every comparison is its whole step (pack, window KV
write, attention, vocab reduction, update) on the same inputs."""
import numpy as np
import pytest
import torch

from harness import (OracleCase, compare_case, compare_pack, gpu_results, log,
                     setup)
from paper_2607_17652_amd import binding as fb
from paper_2607_17652_amd import synth

pytestmark = pytest.mark.gpu


def run_and_compare(name, reqs=None, seed=0, host_edit=None, kv_split=0,
                    check_pack=True, **overrides):
    wl, host, t, step = setup(name, seed, host_edit=host_edit, kv_split=kv_split,
                              **overrides)
    if reqs is None:
        reqs = list(range(wl.B))
    log(f"[parity] workload={name} seed={seed} overrides={overrides} "
        f"B={wl.B} rows={wl.row_cap} reqs={len(reqs)}")
    case = OracleCase(wl, host, t, reqs, step.page_table)
    step.run()
    torch.cuda.synchronize()
    g = gpu_results(step)
    if check_pack:
        compare_pack(wl, host, g, host["tokens"])
    case.run(wl.params())
    summary = compare_case(wl, case, g, step)
    log(f"[parity] {name}: rows={summary['rows']} attn_max_err="
        f"{summary['attn_max_err']:.3e} conf_max_rel={summary['conf_max_rel']:.3e} "
        f"band_requests={summary['band_requests']}")
    return wl, host, step, g, case, summary


def test_tiny_fp32_full():
    run_and_compare("tiny")


def test_single_request_bf16_full():
    run_and_compare("single")


def test_hetero64_padded_full():
    run_and_compare("hetero64")


def test_long8_every_request():
    """Long prefixes (16K-32K keys) exercise split-KV and the combine; every
    one of the 8 requests is compared."""
    run_and_compare("long8")


def test_longest_prefix_hits_the_split_cap():
    """One request with a 64K-key prefix and two live blocks: the split size
    is raised until no unit has more than 64 pieces (the most the merge of
    partial results takes), here 62-63 pieces of 33 key tiles per unit."""
    run_and_compare("single", prefix=("fixed", 65536), window=("fixed", 2), W_max=2)


def test_more_tiles_than_the_plan_keeps_in_registers():
    """1280 live tiles (320 requests x 4 blocks): the plan reads the fields
    of the tiles beyond its register cache (1024) again from memory."""
    run_and_compare("serve256", reqs=[0, 97, 191, 255, 256, 319], B=320,
                    prefix=("loguniform", 64, 1024), window=("fixed", 4))


@pytest.mark.parametrize("quarter", [0, 1, 2, 3])
def test_serve256_every_request(quarter):
    """The serving workload at full size in the bench's launch configuration;
    the four cases together compare all 256 requests (64 each, so that each
    case's oracle work stays well under a minute)."""
    run_and_compare("serve256", reqs=list(range(64 * quarter, 64 * quarter + 64)),
                    check_pack=quarter == 0)


@pytest.mark.parametrize("overrides", [
    dict(prefix_jitter=37),                         # unaligned prefixes: partial key tiles
    dict(page_size=16),
    dict(page_size=64),
    dict(d=64, Hq=8, Hkv=8),                        # no GQA
    dict(d=32, Hq=16, Hkv=2),                       # group of 8
    dict(d=64, Hq=8, Hkv=8, page_size=16),          # d = 64 with pages smaller than a key tile
    dict(d=32, Hq=16, Hkv=2, page_size=8, prefix_jitter=11),   # d = 32, pages of 8
    dict(bl=16, page_size=16, W_max=5, window=("fixed", 5)),
    dict(bl=64, page_size=64, W_max=4, window=("uniform", 1, 4)),   # Table 2 lengths
    dict(bl=96, page_size=32, W_max=3, window=("fixed", 3)),        # bl not a power of 2
    dict(bl=128, page_size=128, W_max=5, window=("fixed", 5), prefix_jitter=40),
    dict(bl=1, page_size=8, W_max=3, window=("fixed", 3), prefix_jitter=3),   # one-token blocks
    dict(bl=8, page_size=8, W_max=6, window=("uniform", 1, 6)),             # pages of 8, W = 6
    dict(V=1001, prefix_jitter=5),                  # unaligned logit rows
    dict(B=5, layout="padded", window=("uniform", 1, 3)),
])
def test_shape_variants(overrides):
    run_and_compare("single", **overrides)


def test_fp32_bigger_shapes():
    run_and_compare("single", dtype="f32", B=3, prefix=("uniform", 40, 300),
                    window=("uniform", 1, 3), V=5003, prefix_jitter=9)


@pytest.mark.parametrize("kv_split,ps", [(32, 32), (64, 32), (96, 32), (128, 32), (160, 32),
                                         (64, 16), (128, 16)])
def test_short_items_take_every_ring_tail(kv_split, ps):
    """A fixed split of kv_split keys makes items of one to five key tiles, so
    the d = 128 ring runs every short schedule: a lone tile, a last step only,
    near-end steps with and without a K refill, and a full step before them;
    jittered prefixes leave the last tile partial, and pages of 16 keys take
    the per-lane page path."""
    run_and_compare("single", kv_split=kv_split, B=3, page_size=ps, V=5003,
                    prefix=("uniform", 20, 400), window=("uniform", 1, 3), prefix_jitter=13)


@pytest.mark.parametrize("layout,B,W_max", [("ragged", 256, 4), ("ragged", 257, 4),
                                            ("padded", 512, 2), ("padded", 513, 2),
                                            ("ragged", 1100, 4)])
def test_pack_row_maps_in_the_workgroup_and_beyond(layout, B, W_max):
    """The pack writes the row maps itself up to 4096 rows (B*W_max*bl, bl = 4
    here) and leaves them to a per-row kernel beyond; both sides of the bound,
    in both layouts, equal the oracle's Eq. 4 pack."""
    wl, host, t, step = setup("tiny", B=B, W_max=W_max, layout=layout, V=64,
                              prefix=("uniform", 8, 64), window=("uniform", 1, W_max),
                              n_blocks=24)
    log(f"[parity] pack only: layout={layout} B={B} W_max={W_max}")
    step.pack_step()
    torch.cuda.synchronize()
    compare_pack(wl, host, gpu_results(step), host["tokens"])


@pytest.mark.parametrize("name,seed,stride", [("long8", 1, 1), ("hetero64", 2, 3),
                                             ("serve256", 1, 9), ("single", 4, 1)])
def test_other_seeds(name, seed, stride):
    """Other draws of the same workloads (request mixes, prefix lengths and
    so item lengths, page permutations, logits), every stride-th request
    compared."""
    wl = synth.workload(name)
    run_and_compare(name, reqs=list(range(seed % stride, wl.B, stride)), seed=seed)


def test_explicit_kv_split_matches_oracle():
    run_and_compare("hetero64", reqs=list(range(0, 64, 7)), kv_split=256)


def test_repeat_is_bit_identical():
    wl, host, t, step = setup("hetero64", seed=3)
    log("[parity] repeat hetero64 seed=3")
    snap = {k: v.clone() for k, v in dict(st=step.st, tokens=step.tokens,
                                          pe=step.pe, fin=step.fin).items()}
    step.run()
    torch.cuda.synchronize()
    out1, conf1, tok1 = step.out.clone(), step.conf.clone(), step.tokens.clone()
    for k, v in snap.items():
        getattr(step, k).copy_(v)
    step.run()
    torch.cuda.synchronize()
    assert torch.equal(out1, step.out)
    assert torch.equal(conf1, step.conf)
    assert torch.equal(tok1, step.tokens)


@pytest.mark.parametrize("name,seed", [("long8", 5), ("hetero64", 6), ("tiny", 7)])
def test_plan_beside_the_kv_write_equals_the_one_call_attention(name, seed):
    """fb_attention_plan on a second stream while fb_write_window_kv runs, then
    fb_wavefront_attention_planned: the same output, bit for bit, as
    fb_wavefront_attention after the KV write (long8 splits every unit, so the
    combine runs on the plan's split list; tiny is the fp32 path, which has no
    plan)."""
    wl, host, t, step = setup(name, seed)
    log(f"[parity] plan beside the KV write: {name} seed={seed}")
    step.pack_step()
    step.kv_step()
    step.attention_step()
    torch.cuda.synchronize()
    ref = step.out.clone()
    step.out.zero_()
    step.attn_ws.fill_(0xA5)       # no plan left over from the one-call run
    main = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    packed = torch.cuda.Event()
    planned = torch.cuda.Event()
    step.pack_step()
    packed.record(main)
    side.wait_event(packed)
    fb.fb_attention_plan(step.pack, step.shape, step.attn_ws, side)
    planned.record(side)
    step.kv_step()
    main.wait_event(planned)
    fb.fb_wavefront_attention_planned(t["q"], t["k_cache"], t["v_cache"], step.page_table,
                                      step.pack, step.shape, step.out, step.attn_ws)
    torch.cuda.synchronize()
    assert torch.equal(step.out, ref)
    assert fb.fb_pack_read_status(step.pack)["code"] == 0


def test_planned_attention_without_a_plan_is_reported():
    """fb_wavefront_attention_planned on a workspace that holds no plan (every
    byte 0x7F: each count is a large positive number and every record field
    lies outside the pack's capacities) reads no record outside its bounds:
    every record is skipped, FB_DERR_PLAN is recorded, and a real plan
    afterwards gives the one-call output again."""
    wl, host, t, step = setup("long8", seed=8)
    log("[parity] planned attention without a plan: long8 seed=8")
    step.pack_step()
    step.kv_step()
    step.attention_step()
    torch.cuda.synchronize()
    ref = step.out.clone()
    step.attn_ws.fill_(0x7F)
    fb.fb_wavefront_attention_planned(t["q"], t["k_cache"], t["v_cache"], step.page_table,
                                      step.pack, step.shape, step.out, step.attn_ws)
    torch.cuda.synchronize()
    s = fb.fb_pack_read_status(step.pack)
    assert s["code"] == fb.FB_DERR_PLAN and s["request"] == 0
    step.pack_step()                       # a fresh pack clears the status word
    fb.fb_attention_plan(step.pack, step.shape, step.attn_ws)
    fb.fb_wavefront_attention_planned(t["q"], t["k_cache"], t["v_cache"], step.page_table,
                                      step.pack, step.shape, step.out, step.attn_ws)
    torch.cuda.synchronize()
    assert fb.fb_pack_read_status(step.pack)["code"] == fb.FB_DERR_NONE
    assert torch.equal(step.out, ref)


def test_ragged_and_padded_agree_bitwise():
    """The same per-position inputs packed ragged and padded give bit-identical
    per-position outputs and identical request state."""
    from oracle import pack as opack      # row placement of the inputs only
    from paper_2607_17652_amd import synth
    from paper_2607_17652_amd.runner import WavefrontStep
    wl, host, t, step = setup("hetero64", seed=4)          # padded
    wl_r = synth.workload("hetero64", layout="ragged")
    log("[parity] ragged vs padded hetero64 seed=4")
    pp = opack.pack_wavefronts(host["state"], wl.W_max, wl.bl, "padded")
    pr = opack.pack_wavefronts(host["state"], wl.W_max, wl.bl, "ragged")
    key_r = {(b, p): r for r, (b, p) in enumerate(zip(pr["row_req"], pr["row_pos"]))
             if b >= 0}
    rows_p = [r for r in range(pp["cap"]) if pp["row_req"][r] >= 0]
    rows_r = [key_r[(pp["row_req"][r], pp["row_pos"][r])] for r in rows_p]
    ip = torch.tensor(rows_p, device="cuda")
    ir = torch.tensor(rows_r, device="cuda")
    t2 = dict(t)
    for k in ("q", "k_new", "v_new", "logits"):
        t2[k] = torch.zeros_like(t[k])
        t2[k][ir] = t[k][ip]
    step2 = WavefrontStep(wl_r, host, t2)
    step.run()
    step2.run()
    torch.cuda.synchronize()
    assert torch.equal(step.out[ip], step2.out[ir])
    assert torch.equal(step.conf[ip], step2.conf[ir])
    assert torch.equal(step.argmax[ip], step2.argmax[ir])
    for k in ("tokens", "st", "pe", "fin"):
        assert torch.equal(getattr(step, k), getattr(step2, k)), k


def test_later_blocks_do_not_change_earlier_outputs():
    """Sec. 4.1: perturbing the fresh K/V of window slots > s leaves every
    output of slot s bit-identical."""
    wl, host, t, step = setup("long8", seed=1, prefix=("uniform", 1000, 3000))
    log("[parity] perturbation long8-short")
    snap = {k: v.clone() for k, v in dict(k_cache=t["k_cache"],
                                          v_cache=t["v_cache"]).items()}
    step.pack_step()
    step.kv_step()
    step.attention_step()
    torch.cuda.synchronize()
    base = step.out.clone()
    view = step.pack.view()
    tiles = view["tiles"].cpu().numpy()
    n_tiles = int(view["header"][1])
    for k, v in snap.items():
        t[k].copy_(v)
    for i in range(n_tiles):
        b, s, row0 = tiles[i, 0], tiles[i, 1], tiles[i, 3]
        if s >= 1:
            t["k_new"][row0:row0 + wl.bl] += 3.0
            t["v_new"][row0:row0 + wl.bl] -= 2.0
    step.pack_step()
    step.kv_step()
    step.attention_step()
    torch.cuda.synchronize()
    for i in range(n_tiles):
        if tiles[i, 1] == 0:
            row0 = tiles[i, 3]
            assert torch.equal(base[row0:row0 + wl.bl], step.out[row0:row0 + wl.bl])


def test_packed_equals_each_request_alone():
    """Sec. 4.2: packed execution equals per-request execution, bit for bit
    (fixed split size so the key partitions are the same)."""
    wl, host, t, step = setup("hetero64", seed=5, kv_split=512, B=6,
                              layout="ragged")
    log("[parity] packed vs alone")
    step.run()
    torch.cuda.synchronize()
    g = gpu_results(step)
    from paper_2607_17652_amd import synth
    from paper_2607_17652_amd.runner import WavefrontStep
    for b in range(wl.B):
        wl1 = synth.workload("hetero64", B=1, layout="ragged")
        h1 = {k: (v[b:b + 1].copy() if isinstance(v, np.ndarray) and v.ndim >= 1
                  and v.shape[0] == wl.B else v) for k, v in host.items()}
        h1["state"] = {k: v[b:b + 1].copy() for k, v in host["state"].items()}
        rows = np.flatnonzero(g["row_req"] == b)
        t1 = {k: t[k] for k in ("k_cache", "v_cache")}
        cap1 = wl1.row_cap
        for k in ("q", "k_new", "v_new", "logits"):
            arr = torch.zeros((cap1,) + tuple(t[k].shape[1:]), dtype=t[k].dtype,
                              device="cuda")
            arr[:len(rows)] = t[k][torch.from_numpy(rows).cuda()]
            t1[k] = arr
        s1 = WavefrontStep(wl1, h1, t1, kv_split=512)
        s1.run()
        torch.cuda.synchronize()
        assert torch.equal(s1.out[:len(rows)], step.out[torch.from_numpy(rows).cuda()])
        assert torch.equal(s1.tokens[0], step.tokens[b])
        assert torch.equal(s1.st[0], step.st[b])


def test_all_inactive_is_a_noop():
    def edit(wl, host):
        host["state"]["active"][:] = 0
    wl, host, t, step = setup("hetero64", seed=2, host_edit=edit)
    log("[parity] all inactive")
    before = step.tokens.clone()
    st_before = step.st.clone()
    step.run()
    torch.cuda.synchronize()
    s = fb.fb_pack_read_status(step.pack)
    assert s["n_rows"] == 0 and s["n_tiles"] == 0 and s["code"] == 0
    assert torch.equal(before, step.tokens)
    assert torch.equal(st_before, step.st)


def test_ill_formed_state_is_reported_and_skipped():
    def edit(wl, host):
        host["state"]["R"][3] = host["state"]["L"][3] + wl.W_max + 1
    wl, host, t, step = setup("hetero64", seed=6, host_edit=edit)
    log("[parity] ill-formed request 3")
    st_before = step.st.clone()
    step.run()
    torch.cuda.synchronize()
    s = fb.fb_pack_read_status(step.pack)
    assert s["code"] == fb.FB_DERR_STATE and s["request"] == 3
    assert torch.equal(st_before[3], step.st[3])
    stats = fb.stats_to_numpy(step.stats, wl.B)
    assert stats["valid"][3] == 0 and stats["valid"][2] == 1


def test_bad_page_id_is_reported_without_fault():
    def edit(wl, host):
        host["page_table"][2, 1] = host["num_pages"] + 1000
        host["page_table"][4, 0] = -5
    wl, host, t, step = setup("hetero64", seed=6, host_edit=edit)
    log("[parity] bad page ids in requests 2 and 4")
    step.run()
    torch.cuda.synchronize()
    s = fb.fb_pack_read_status(step.pack)
    assert s["code"] == fb.FB_DERR_PAGE and s["request"] == 2


@pytest.mark.parametrize("flags", [dict(edit_masked=True),
                                   dict(force_progress=True),
                                   dict(edit_masked=True, force_progress=True, S_pe=0),
                                   dict(eos=True)])
def test_update_flags(flags):
    """Each flag, and EDIT_MASKED with FORCE_PROGRESS at S_pe = 0 (masked rows
    revealed by Delta count as the block's progress and once each, so a block
    still holding a mask is not finished)."""
    flags = dict(flags)
    eos = flags.pop("eos", False)
    extra = {"S_pe": flags.pop("S_pe")} if "S_pe" in flags else {}
    eos_id = 7

    def edit(wl, host):
        if eos:
            # plant the EOS id in a fifth of the revealed window tokens so that
            # retiring blocks hold it
            rng = np.random.default_rng(0)
            st = host["state"]
            for b in range(wl.B):
                o = int(host["o"][b])
                for p in range(o, o + int(st["R"][b] - st["L"][b]) * wl.bl):
                    if host["tokens"][b, p] != wl.mask_id and rng.uniform() < 0.2:
                        host["tokens"][b, p] = eos_id
    wl, host, t, step = setup("hetero64", seed=8, host_edit=edit,
                              eos_id=eos_id if eos else -1, **extra)
    log(f"[parity] flags {flags} eos={eos}")
    p = dict(wl.params(), **flags)
    step.set_params(flags=(fb.FB_EDIT_MASKED if p["edit_masked"] else 0) |
                    (fb.FB_FORCE_PROGRESS if p["force_progress"] else 0))
    case = OracleCase(wl, host, t, list(range(wl.B)), step.page_table)
    step.run()
    torch.cuda.synchronize()
    g = gpu_results(step)
    case.run(p, attention=False)
    compare_case(wl, case, g, step, check_attention=False, check_kv=False)


def _plant_neg_inf(logits, V):
    """-inf runs by row index mod 6: the first half of the row; all but the
    last 37 ids; the first 4 of every 8 ids; ids 0..10 (the unaligned head
    of a row when V is odd); all but one id in the middle (p = 1); none."""
    rows = logits.shape[0]
    ninf = float("-inf")
    low_half_of_8 = torch.arange(V, device=logits.device) % 8 < 4
    for r in range(rows):
        kind = r % 6
        if kind == 0:
            logits[r, :V // 2] = ninf
        elif kind == 1:
            logits[r, :V - 37] = ninf
        elif kind == 2:
            logits[r, low_half_of_8] = ninf
        elif kind == 3:
            logits[r, :11] = ninf
        elif kind == 4:
            keep = logits[r, V // 3].clone()
            logits[r] = ninf
            logits[r, V // 3] = keep


@pytest.mark.parametrize("V", [157184, 1001, 40009])
def test_neg_inf_logits(V):
    """-inf logits weigh exp(-inf) = 0 (Eq. 1's softmax): runs of them at the
    start of a workgroup's pieces, over every piece of some workgroups,
    inside every 16-byte group and at an unaligned row head give the oracle's
    argmax and confidence, and the same update (V = 40009: odd rows of three
    32 KB pieces, one per workgroup)."""
    wl, host, t, step = setup("single", seed=13, V=V)
    log(f"[parity] -inf logits V={V} rows={wl.row_cap}")
    _plant_neg_inf(t["logits"], V)
    case = OracleCase(wl, host, t, list(range(wl.B)), step.page_table)
    step.run()
    torch.cuda.synchronize()
    g = gpu_results(step)
    case.run(wl.params(), attention=False)
    compare_case(wl, case, g, step, check_attention=False, check_kv=False)
    assert np.all(np.isfinite(g["conf"][: wl.row_cap][g["row_req"] >= 0]))


def _plant_ties(logits, V, seed):
    """Exact ties at the row maximum, by row index mod 8: ids {0, V-1};
    {V-2, V-1}; four random ids; two adjacent ids; two ids 4096 apart; a
    constant row; no change; {x, V//2, V-1}.  Returns the lowest planted id
    per row (-1 where nothing was planted)."""
    rows = logits.shape[0]
    rng = np.random.default_rng(seed)
    m = logits.amax(dim=1).float()
    tie = (m + torch.clamp(m.abs() / 16, min=1.0)).to(logits.dtype)
    lowest = np.full(rows, -1, dtype=np.int64)
    rr, ii, const = [], [], []
    for r in range(rows):
        kind = r % 8
        if kind == 0:
            ids = [0, V - 1]
        elif kind == 1:
            ids = [V - 2, V - 1]
        elif kind == 2:
            ids = rng.choice(V, size=4, replace=False).tolist()
        elif kind == 3:
            x = int(rng.integers(0, V - 1))
            ids = [x, x + 1]
        elif kind == 4:
            x = int(rng.integers(0, V - 4096))
            ids = [x, x + 4096]
        elif kind == 5:
            const.append(r)
            lowest[r] = 0
            continue
        elif kind == 6:
            continue
        else:
            ids = [int(rng.integers(0, V // 2)), V // 2, V - 1]
        rr += [r] * len(ids)
        ii += ids
        lowest[r] = min(ids)
    rr = torch.tensor(rr, device=logits.device)
    logits[rr, torch.tensor(ii, device=logits.device)] = tie[rr]
    logits[torch.tensor(const, device=logits.device)] = 0.25
    return lowest


@pytest.mark.parametrize("V", [157184, 5003, 40009])
def test_argmax_ties_take_the_lowest_id(V):
    """Exact ties at the maximum of a row (Eq. 1 takes the argmax; the
    lowest id wins a tie) planted across the vocabulary partitions, inside
    one 16-byte vector, a thread stride apart and over whole constant rows:
    the GPU argmax equals the oracle's, which is the lowest planted id."""
    wl, host, t, step = setup("hetero64", seed=12, V=V)
    log(f"[parity] argmax ties V={V} rows={wl.row_cap}")
    lowest = _plant_ties(t["logits"], V, seed=12)
    case = OracleCase(wl, host, t, list(range(wl.B)), step.page_table)
    step.run()
    torch.cuda.synchronize()
    g = gpu_results(step)
    case.run(wl.params(), attention=False)
    compare_case(wl, case, g, step, check_attention=False, check_kv=False)
    n_planted = 0
    for rf, rs in case.map_rows:
        sel = lowest[rf] >= 0
        assert np.array_equal(case.xhat[rs][sel], lowest[rf][sel])
        assert np.array_equal(g["argmax"][rf][sel], lowest[rf][sel])
        n_planted += int(sel.sum())
    assert n_planted > 100
    # a constant row has p = 1/V
    const = [r for rf, _ in case.map_rows for r in rf if r % 8 == 5]
    assert const and np.allclose(g["conf"][const], 1.0 / V, rtol=1e-6)


@pytest.mark.parametrize("name", ["tiny", "single", "hetero64"])
def test_multi_step_matches_oracle(name):
    """Four consecutive steps with fresh inputs each step: the GPU state and
    the oracle state evolve identically (the oracle from its own results)."""
    from oracle import attention as oatt, pack as opack, update as oupd
    from paper_2607_17652_amd import synth
    wl, host, t, step = setup(name, seed=9)
    ost = {k: v.copy() for k, v in host["state"].items()}
    otok, ope, ofin = host["tokens"].copy(), host["pe"].copy(), host["fin"].copy()
    excluded = set()
    for it in range(4):
        log(f"[parity] multi-step {name} step {it}")
        gen = torch.Generator(device="cuda")
        gen.manual_seed(1000 + it)
        t["logits"] = synth.make_logits(wl, wl.row_cap, gen, "cuda")
        step.t = t
        packed = opack.pack_wavefronts(ost, wl.W_max, wl.bl, wl.layout)
        live = np.flatnonzero(packed["row_req"] >= 0)
        xhat = np.full(packed["cap"], -1)
        p64 = np.zeros(packed["cap"])
        for c0 in range(0, len(live), 128):
            r = live[c0:c0 + 128]
            z = t["logits"][torch.from_numpy(r).cuda()].double().cpu().numpy()
            xhat[r], p64[r] = oupd.vocab_reduce(z)
        res = oupd.denoise_update(xhat, p64, otok, ost, ope, ofin, packed,
                                  wl.params())
        step.run()
        torch.cuda.synchronize()
        g = gpu_results(step)
        assert np.array_equal(g["row_req"], packed["row_req"])
        excluded |= set(res["band_reqs"])
        for b in range(wl.B):
            if b in excluded:
                continue
            assert np.array_equal(g["tokens"][b], res["tokens"][b]), (it, b)
            for k in ("L", "R", "active"):
                assert g["st"][k][b] == res["state"][k][b], (it, b, k)
            assert np.array_equal(g["fin"][b], res["fin"][b]), (it, b)
            assert np.array_equal(g["pe"][b], res["pe"][b]), (it, b)
        ost, otok, ope, ofin = res["state"], res["tokens"], res["pe"], res["fin"]
        if excluded:
            log(f"[parity] band-excluded requests: {sorted(excluded)}")


@pytest.mark.parametrize("name", ["tiny", "single", "hetero64"])
def test_graph_replay_matches_eager(name):
    """One whole step captured in a HIP graph: every replay (with eager work
    and state restores between replays) reproduces the eager step bit for
    bit.  No kernel of the step clears memory with a memset."""
    wl, host, t, step = setup(name)
    log(f"[graph] workload={name}")
    state = [step.st, step.tokens, step.pe, step.fin]
    pristine = [x.clone() for x in state]

    def restore():
        for dst, src in zip(state, pristine):
            dst.copy_(src)

    def outputs():
        return [x.clone() for x in state] + [step.out.clone(), step.conf.clone(),
                                             step.argmax.clone(), step.stats.clone()]

    step.run()
    torch.cuda.synchronize()
    ref = outputs()
    restore()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step.run()
    for r in range(3):
        restore()
        scratch = torch.randn(1 << 20, device="cuda").sum()   # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = outputs()
        for i, (a, b) in enumerate(zip(got, ref)):
            assert torch.equal(a, b), f"replay {r}: output {i} differs from the eager step"
        del scratch


def test_hbm_probes_read_and_copy_every_byte():
    """The read probe's per-workgroup XORs combine to the XOR of every 32-bit
    word of the buffer (computed on the host), including a size that does not
    divide evenly among the workgroups; the copy probe copies exactly."""
    for nbytes in (64 << 20, (64 << 20) + 48 * 1024 + 16):
        log(f"[probe] bytes={nbytes}")
        g = torch.Generator(device="cuda")
        g.manual_seed(nbytes & 0xffff)
        src = torch.randint(-2**31, 2**31 - 1, (nbytes // 4,), dtype=torch.int32,
                            device="cuda", generator=g)
        out = torch.zeros(fb.FB_PROBE_BLOCKS, dtype=torch.int32, device="cuda")
        fb.fb_hbm_read_probe(src, out)
        dst = torch.zeros_like(src)
        fb.fb_hbm_copy_probe(src, dst)
        torch.cuda.synchronize()
        want = np.bitwise_xor.reduce(src.cpu().numpy().view(np.uint32))
        got = np.bitwise_xor.reduce(out.cpu().numpy().view(np.uint32))
        assert got == want
        assert torch.equal(src, dst)
