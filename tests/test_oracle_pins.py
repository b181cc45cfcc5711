"""Pins of the oracle against facts fixed by the paper and by mathematics:
closed forms, library routines, an independent dense-mask brute force on the
paper's own physical layout, an independent serial decoder, and invariants the
paper states.  CPU only."""
import math
import os

import numpy as np
import pytest
import scipy.special

from oracle import attention, bruteforce, pack, serial, step, update

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ----------------------------------------------------------------- helpers --
def make_case(rng, B=3, Hq=4, Hkv=2, d=8, bl=3, W_max=3, o_max=10, gen=None):
    """A small random multi-request case: states with random prefixes and
    windows, logical prefix K/V, packed q / k_new / v_new."""
    o = rng.integers(0, o_max + 1, size=B)
    w = rng.integers(1, W_max + 1, size=B)
    n = w + rng.integers(0, 3, size=B)
    state = dict(gen_start=o.copy(), prompt_len=o.copy(), n_blocks=n,
                 L=np.zeros(B, dtype=np.int64), R=w.copy(),
                 active=np.ones(B, dtype=np.int64),
                 eos_hit=np.zeros(B, dtype=np.int64))
    T = int((o + n * bl).max())
    K = [rng.normal(size=(T, Hkv, d)) for _ in range(B)]
    V = [rng.normal(size=(T, Hkv, d)) for _ in range(B)]
    cap = B * W_max * bl
    q = rng.normal(size=(cap, Hq, d))
    k_new = rng.normal(size=(cap, Hkv, d))
    v_new = rng.normal(size=(cap, Hkv, d))
    return dict(o=o, w=w, state=state, K=K, V=V, q=q, k_new=k_new,
                v_new=v_new, Hq=Hq, Hkv=Hkv, d=d, bl=bl, W_max=W_max, B=B)


def run_oracle_attention(c, layout=pack.RAGGED):
    packed = pack.pack_wavefronts(c["state"], c["W_max"], c["bl"], layout)
    K, V = attention.write_window_kv(c["K"], c["V"], c["k_new"], c["v_new"],
                                     packed)
    out = attention.window_attention(c["q"], K, V, packed, c["Hq"], c["Hkv"])
    return packed, K, V, out


def rows_of(packed, b):
    """Packed rows of request b in position order."""
    r = np.flatnonzero(packed["row_req"] == b)
    return r[np.argsort(packed["row_pos"][r])]


# ---------------------------------------------------------- golden numbers --
def read_golden(name):
    out = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                parts = line.split()
                out[parts[0]] = [int(x) for x in parts[1:]]
    return out


def test_paper_worked_window_rows():
    """Sec. 4.2 Discussion: W*bl = 64 query positions at W=2, bl=32; the
    padded packed batch gives each request exactly that many rows (Eq. 4)."""
    g = read_golden("paper_worked_numbers.txt")
    W, bl, expect = g["window_rows"]
    state = dict(gen_start=np.array([0, 96]), prompt_len=np.array([0, 96]),
                 n_blocks=np.array([64, 64]), L=np.array([3, 0]),
                 R=np.array([5, 1]), active=np.array([1, 1]),
                 eos_hit=np.array([0, 0]))
    packed = pack.pack_wavefronts(state, W, bl, pack.PADDED)
    assert packed["cap"] // 2 == expect
    # request 0: slots 0, 1 live at positions 96..159 in rows 0..63
    assert list(packed["row_pos"][:expect]) == list(range(96, 96 + expect))
    gen_len, bl2, blocks = g["blocks_per_request"]
    assert gen_len // bl2 == blocks


def test_pack_ragged_and_padded_hold_the_same_rows():
    rng = np.random.default_rng(1)
    c = make_case(rng, B=5)
    pr = pack.pack_wavefronts(c["state"], c["W_max"], c["bl"], pack.RAGGED)
    pp = pack.pack_wavefronts(c["state"], c["W_max"], c["bl"], pack.PADDED)
    assert pr["n_rows"] == pp["n_rows"] == int(c["w"].sum()) * c["bl"]
    for b in range(c["B"]):
        a, z = rows_of(pr, b), rows_of(pp, b)
        assert list(pr["row_pos"][a]) == list(pp["row_pos"][z])
        # Eq. 4: pos[b] = o_b + [0..w_b*bl)
        assert list(pr["row_pos"][a]) == list(range(c["o"][b],
                                                   c["o"][b] + c["w"][b] * c["bl"]))
    # ragged rows are dense from 0
    assert np.all(pr["row_req"][:pr["n_rows"]] >= 0)
    assert np.all(pr["row_req"][pr["n_rows"]:] == -1)


def test_pack_rejects_ill_formed_wavefront():
    state = dict(gen_start=np.array([0]), prompt_len=np.array([0]),
                 n_blocks=np.array([4]), L=np.array([0]), R=np.array([3]),
                 active=np.array([1]), eos_hit=np.array([0]))
    with pytest.raises(ValueError):
        pack.pack_wavefronts(state, 2, 4, pack.RAGGED)


# ------------------------------------------------------- vocab reduction ---
@pytest.mark.parametrize("a,expect", [
    (4.0, 0.9317384593585715), (3.0, 0.8339252302011539),
    (2.0, 0.6487856442839393), (0.0, 0.2)])
def test_two_level_confidence_closed_form(a, expect):
    """z = a*e_k over V=5 gives p = e^a / (e^a + 4)."""
    z = np.zeros((1, 5))
    z[0, 3] = a
    xhat, p = update.vocab_reduce(z)
    assert abs(p[0] - expect) < 1e-15
    assert abs(p[0] - math.exp(a) / (math.exp(a) + 4)) < 1e-15
    assert xhat[0] == (3 if a > 0 else 0)


def test_vocab_reduce_matches_library_softmax():
    rng = np.random.default_rng(2)
    z = rng.normal(size=(64, 1000)) * rng.uniform(1, 8, size=(64, 1))
    xhat, p = update.vocab_reduce(z)
    sm = scipy.special.softmax(z, axis=1)
    assert np.allclose(sm.sum(axis=1), 1.0, atol=1e-12)
    assert np.array_equal(xhat, np.argmax(z, axis=1))
    assert np.allclose(p, sm.max(axis=1), rtol=1e-12, atol=0)
    lse = scipy.special.logsumexp(z, axis=1)
    assert np.allclose(np.log(p), z.max(axis=1) - lse, atol=1e-12)


def test_vocab_reduce_ties_go_to_lowest_index():
    z = np.zeros((3, 7))
    z[0, [2, 5]] = 1.5
    z[1, [6, 0]] = 2.0
    z[2, :] = -3.0
    xhat, p = update.vocab_reduce(z)
    assert list(xhat) == [2, 0, 0]
    assert abs(p[2] - 1 / 7) < 1e-15
    assert abs(p[0] - math.exp(1.5) / (2 * math.exp(1.5) + 5)) < 1e-15


# -------------------------------------------------------------- attention --
@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_attention_equals_dense_mask_on_tail_layout(seed):
    """Eq. 5 literally (explicit dense mask, physical tail, junk in the stale
    middle) equals the kv_len rule of the oracle to 1e-12."""
    rng = np.random.default_rng(seed)
    c = make_case(rng, B=3, Hq=4, Hkv=2, d=8, bl=3, W_max=3, o_max=9)
    packed, _, _, out = run_oracle_attention(c)
    q_win, k_win, v_win = [], [], []
    for b in range(c["B"]):
        r = rows_of(packed, b)
        q_win.append(c["q"][r])
        k_win.append(c["k_new"][r])
        v_win.append(c["v_new"][r])
    bf = bruteforce.tail_layout_attention(q_win, c["K"], c["V"], k_win, v_win,
                                          c["o"], c["w"], c["W_max"], c["bl"],
                                          c["Hq"], c["Hkv"])
    for b in range(c["B"]):
        assert np.max(np.abs(out[rows_of(packed, b)] - bf[b])) < 1e-12


def test_window_of_one_equals_serial_block_attention():
    """W = 1: the single live block sees [0, o + bl) -- serial block-wise
    attention, computed by the independent serial module."""
    rng = np.random.default_rng(5)
    c = make_case(rng, B=2, Hq=4, Hkv=1, d=6, bl=4, W_max=1, o_max=12)
    packed, K, V, out = run_oracle_attention(c)
    for b in range(c["B"]):
        r = rows_of(packed, b)
        ref = serial.serial_block_attention(c["q"][r], K[b], V[b], int(c["o"][b]),
                                            c["bl"], c["Hq"], c["Hkv"])
        assert np.max(np.abs(out[r] - ref)) < 1e-12


def test_later_blocks_do_not_change_earlier_outputs():
    """Sec. 4.1: no query depends on blocks to its right.  Perturbing the
    window K/V of blocks > s leaves block s bit-identical."""
    rng = np.random.default_rng(6)
    c = make_case(rng, B=2, W_max=3)
    c["w"][:] = 3
    c["state"]["R"] = c["w"].copy()
    c["state"]["n_blocks"] = np.maximum(c["state"]["n_blocks"], 3)
    packed, _, _, out = run_oracle_attention(c)
    for t in packed["tiles"]:
        if t["s"] != 1:
            continue
        c2 = dict(c)
        c2["k_new"] = c["k_new"].copy()
        c2["v_new"] = c["v_new"].copy()
        for t2 in packed["tiles"]:
            if t2["b"] == t["b"] and t2["s"] > t["s"]:
                sl = slice(t2["row0"], t2["row0"] + c["bl"])
                c2["k_new"][sl] += 100.0
                c2["v_new"][sl] -= 50.0
        _, _, _, out2 = run_oracle_attention(c2)
        sl = slice(t["row0"], t["row0"] + c["bl"])
        assert np.array_equal(out[sl], out2[sl])


def test_prefix_kv_is_never_modified_by_window_write():
    """Sec. 4.2: committed KV entries are never modified by the Eq. 6 write."""
    rng = np.random.default_rng(7)
    c = make_case(rng)
    packed, K, V, _ = run_oracle_attention(c)
    for b in range(c["B"]):
        o = int(c["o"][b])
        assert np.array_equal(K[b][:o], c["K"][b][:o])
        assert np.array_equal(V[b][:o], c["V"][b][:o])
        end = o + int(c["w"][b]) * c["bl"]
        assert np.array_equal(K[b][end:], c["K"][b][end:])


def test_packed_equals_each_request_alone():
    """Sec. 4.2: packed execution is token-exact with independent per-sequence
    execution (bit-identical in the oracle)."""
    rng = np.random.default_rng(8)
    c = make_case(rng, B=4)
    packed, _, _, out = run_oracle_attention(c, pack.PADDED)
    for b in range(c["B"]):
        r = rows_of(packed, b)
        one = dict(c)
        one["B"] = 1
        one["state"] = {k: v[b:b + 1].copy() for k, v in c["state"].items()}
        one["K"], one["V"] = [c["K"][b]], [c["V"][b]]
        cap1 = c["W_max"] * c["bl"]
        for key, H in (("q", c["Hq"]), ("k_new", c["Hkv"]), ("v_new", c["Hkv"])):
            arr = np.zeros((cap1, H, c["d"]))
            arr[:len(r)] = c[key][r]
            one[key] = arr
        p1, _, _, out1 = run_oracle_attention(one)
        assert np.array_equal(out1[rows_of(p1, 0)], out[r])


def test_attention_closed_forms():
    """kv_len = 1 gives O = v_0; q = 0 gives the mean of the visible values;
    the weights of any query sum to 1."""
    rng = np.random.default_rng(9)
    d, Hkv = 5, 1
    state = dict(gen_start=np.array([0]), prompt_len=np.array([0]),
                 n_blocks=np.array([2]), L=np.array([0]), R=np.array([2]),
                 active=np.array([1]), eos_hit=np.array([0]))
    K = [rng.normal(size=(4, Hkv, d))]
    V = [rng.normal(size=(4, Hkv, d))]
    q = rng.normal(size=(2, 1, d))
    k_new = rng.normal(size=(2, Hkv, d))
    v_new = rng.normal(size=(2, Hkv, d))
    packed = pack.pack_wavefronts(state, 2, 1, pack.RAGGED)
    K2, V2 = attention.write_window_kv(K, V, k_new, v_new, packed)
    out = attention.window_attention(q, K2, V2, packed, 1, 1)
    assert np.allclose(out[0, 0], v_new[0, 0], atol=1e-15)   # only key 0
    q0 = np.zeros_like(q)
    out0 = attention.window_attention(q0, K2, V2, packed, 1, 1)
    assert np.allclose(out0[1, 0], v_new[:2, 0].mean(axis=0), atol=1e-15)
    wts = attention.attention_weights(q[1, 0], K2[0][:2, 0], 1 / math.sqrt(d))
    assert abs(wts.sum() - 1.0) < 1e-15


# ------------------------------------------------------------ whole step ---
@pytest.mark.parametrize("seed,layout", [(10, pack.RAGGED), (11, pack.PADDED)])
def test_whole_step_attention_is_eq5_over_the_written_window(seed, layout):
    """One whole step: the attention it returns is Eq. 5 applied literally on
    the physical tail layout whose tail holds this step's fresh window K/V
    (so the window's own keys must be visible, from the Eq. 6 write, not the
    stale cache entries at those positions); the caches it returns hold the
    window at o_b + delta and the old values everywhere else."""
    rng = np.random.default_rng(seed)
    c = make_case(rng, B=3, Hq=4, Hkv=2, d=8, bl=3, W_max=3, o_max=9)
    Vv = 11
    cap = c["B"] * c["W_max"] * c["bl"]
    logits = rng.normal(size=(cap, Vv)) * 3
    tokens = np.full((c["B"], int((c["o"] + c["state"]["n_blocks"] * c["bl"]).max())),
                     Vv - 1, dtype=np.int64)
    n_max = int(c["state"]["n_blocks"].max())
    pe = np.zeros((c["B"], n_max), dtype=np.int64)
    prm = dict(tau_mask=0.9, tau_edit=0.8, theta=0.5, mask_id=Vv - 1, eos_id=-1,
               S_pe=2, W=c["W_max"])
    res = step.wavefront_step(c["state"], tokens, pe, pe.copy(), c["q"], c["k_new"],
                              c["v_new"], c["K"], c["V"], logits, prm, c["W_max"],
                              c["bl"], layout, c["Hq"], c["Hkv"])
    packed = res["packed"]
    q_win, k_win, v_win = [], [], []
    for b in range(c["B"]):
        r = rows_of(packed, b)
        q_win.append(c["q"][r])
        k_win.append(c["k_new"][r])
        v_win.append(c["v_new"][r])
    bf = bruteforce.tail_layout_attention(q_win, c["K"], c["V"], k_win, v_win,
                                          c["o"], c["w"], c["W_max"], c["bl"],
                                          c["Hq"], c["Hkv"])
    for b in range(c["B"]):
        r = rows_of(packed, b)
        assert np.max(np.abs(res["out"][r] - bf[b])) < 1e-12
        o, n = int(c["o"][b]), int(c["w"][b]) * c["bl"]
        assert np.array_equal(res["K"][b][o:o + n], k_win[b])
        assert np.array_equal(res["V"][b][o:o + n], v_win[b])
        assert np.array_equal(res["K"][b][:o], c["K"][b][:o])
        assert np.array_equal(res["V"][b][o + n:], c["V"][b][o + n:])
        # every live row's prediction is its own row's argmax
        assert np.array_equal(res["xhat"][r], np.argmax(logits[r], axis=1))
    # fetching rows through a callable gives the same step
    res2 = step.wavefront_step(c["state"], tokens, pe, pe.copy(), c["q"], c["k_new"],
                               c["v_new"], c["K"], c["V"], lambda rows: logits[rows],
                               prm, c["W_max"], c["bl"], layout, c["Hq"], c["Hkv"])
    assert np.array_equal(res2["out"], res["out"])
    assert np.array_equal(res2["update"]["tokens"], res["update"]["tokens"])


def test_whole_step_update_follows_the_first_hand_traced_step():
    """Step 1 of the hand trace T1 (V = 5, bl = 2, W = 2; [M] = 4): logits
    (4,1) at position 0 and (2,2) at position 1 reveal position 0 only
    (p = .9317 > tau_mask; .6488 is not), rho(B0) = 1/2 >= theta admits B1.
    Run as a whole step, with the logits given in the packed row layout."""
    M_, bl, d = 4, 2, 2
    state = dict(gen_start=np.array([0]), prompt_len=np.array([0]),
                 n_blocks=np.array([3]), L=np.array([0]), R=np.array([1]),
                 active=np.array([1]), eos_hit=np.array([0]))
    tokens = np.full((1, 6), M_, dtype=np.int64)
    pe = np.zeros((1, 3), dtype=np.int64)
    cap = 2 * bl
    logits = np.zeros((cap, 5))
    logits[0, 1] = 4.0
    logits[1, 2] = 2.0
    logits[2:] = np.nan          # rows that are not live are never read
    zq = np.zeros((cap, 1, d))
    Kp = [np.zeros((6, 1, d))]
    prm = dict(tau_mask=0.9, tau_edit=0.8, theta=0.5, mask_id=M_, eos_id=-1,
               S_pe=1, W=2)
    res = step.wavefront_step(state, tokens, pe, pe.copy(), zq, zq, zq, Kp, Kp,
                              logits, prm, 2, bl, pack.RAGGED, 1, 1)
    up = res["update"]
    assert list(up["tokens"][0]) == [1, M_, M_, M_, M_, M_]
    assert list(res["xhat"][:2]) == [1, 2]
    assert abs(res["p64"][0] - 0.9317384593585715) < 1e-15
    assert abs(res["p64"][1] - 0.6487856442839393) < 1e-15
    assert (int(up["state"]["L"][0]), int(up["state"]["R"][0])) == (0, 2)
    assert up["stats"][0]["m2t"] == 1 and up["stats"][0]["spawned"] == 1
    assert up["stats"][0]["rho"] == 0.5


# ------------------------------------------------------------ loop level ---
def toy_model(V, bl_salt=0):
    """A deterministic stand-in for f_theta over a tiny vocabulary: the peak
    height of position p grows with the number of revealed tokens it can see,
    and the predicted id depends on the visible tokens, so drafts get edited
    as context fills in.  The first masked position of a block is always
    confident, so every forward reveals at least one token."""
    def model(x, lo, hi, gen_start=0):
        M = V - 1
        vis = x[:hi]
        revealed = int(np.sum(vis != M))
        ctx = int(np.sum(np.where(vis != M, vis, 0))) + bl_salt
        z = np.zeros((hi - lo, V))
        masked = [p for p in range(lo, hi) if x[p] == M]
        for i, p in enumerate(range(lo, hi)):
            k = (3 * p + (ctx // 7)) % (V - 1)
            a = 0.8 + 0.35 * revealed / (1 + (p % 3)) + 0.1 * (p % 5)
            if masked and p == masked[0]:
                a = max(a, 3.5)      # guarantees progress every forward
            z[i] = -0.2 * ((np.arange(V) + p) % 3)
            z[i, k] = a
        return z
    return model


@pytest.mark.parametrize("S_pe", [0, 1, 2])
def test_gwd_with_window_one_equals_serial_decoding(S_pe):
    """Alg. 1 with W = 1 reproduces serial block-wise decoding exactly: same
    final tokens and the same number of forwards."""
    V, bl, n, prompt = 7, 3, 5, 4
    prm = dict(tau_mask=0.55, tau_edit=0.5, theta=0.5, mask_id=V - 1,
               eos_id=-1, S_pe=S_pe, W=1)
    x0 = np.full(prompt + n * bl, V - 1, dtype=np.int64)
    x0[:prompt] = [1, 2, 3, 4]
    model = toy_model(V)
    ser, fwd, committed = serial.serial_decode(model, x0, prompt, prompt, n, bl,
                                               prm)
    state = dict(gen_start=np.array([prompt]), prompt_len=np.array([prompt]),
                 n_blocks=np.array([n]), L=np.array([0]), R=np.array([1]),
                 active=np.array([1]), eos_hit=np.array([0]))
    res = step.gwd_loop(
        model, state, x0[None, :], np.zeros((1, n), dtype=np.int64),
        np.zeros((1, n), dtype=np.int64), prm, 1, bl, pack.RAGGED)
    assert np.array_equal(res["tokens"][0], ser)
    assert res["forwards"][0] == fwd
    assert committed == n and res["state"]["L"][0] == n


def test_gwd_batch_equals_each_request_alone():
    """Sec. 4.2: per-request wavefronts are independent -- stepping B requests
    together gives each the tokens it gets alone."""
    V, bl, n = 7, 3, 4
    prm = dict(tau_mask=0.55, tau_edit=0.5, theta=0.4, mask_id=V - 1,
               eos_id=-1, S_pe=1, W=2)
    rng = np.random.default_rng(11)
    B = 3
    prompts = [2, 5, 3]
    T = max(prompts) + n * bl
    x0 = np.full((B, T), V - 1, dtype=np.int64)
    for b in range(B):
        x0[b, :prompts[b]] = rng.integers(0, V - 1, size=prompts[b])
    state = dict(gen_start=np.array(prompts), prompt_len=np.array(prompts),
                 n_blocks=np.full(B, n), L=np.zeros(B, dtype=np.int64),
                 R=np.ones(B, dtype=np.int64), active=np.ones(B, dtype=np.int64),
                 eos_hit=np.zeros(B, dtype=np.int64))
    z = np.zeros((B, n), dtype=np.int64)
    model = toy_model(V)
    res = step.gwd_loop(model, state, x0, z, z, prm, 2, bl, pack.PADDED)
    for b in range(B):
        s1 = {k: v[b:b + 1].copy() for k, v in state.items()}
        r1 = step.gwd_loop(model, s1, x0[b:b + 1], z[:1], z[:1], prm, 2, bl,
                           pack.RAGGED)
        assert np.array_equal(r1["tokens"][0], res["tokens"][b])
        assert r1["forwards"][0] == res["forwards"][b]


def test_wavefront_is_no_slower_than_serial_in_forwards():
    """With W = 2 and a gate the loop overlaps blocks, so it needs at most as
    many forwards as serial decoding on the toy model (the TPF claim of
    Sec. 5.2 in miniature)."""
    V, bl, n, prompt = 7, 3, 6, 2
    prm = dict(tau_mask=0.55, tau_edit=0.5, theta=0.3, mask_id=V - 1,
               eos_id=-1, S_pe=1, W=2)
    x0 = np.full(prompt + n * bl, V - 1, dtype=np.int64)
    x0[:prompt] = [0, 1]
    model = toy_model(V)
    _, fwd_serial, _ = serial.serial_decode(model, x0, prompt, prompt, n, bl,
                                            dict(prm, W=1))
    state = dict(gen_start=np.array([prompt]), prompt_len=np.array([prompt]),
                 n_blocks=np.array([n]), L=np.array([0]), R=np.array([1]),
                 active=np.array([1]), eos_hit=np.array([0]))
    z = np.zeros((1, n), dtype=np.int64)
    res = step.gwd_loop(model, state, x0[None], z, z, prm, 2, bl, pack.RAGGED)
    assert res["state"]["L"][0] == n
    assert res["forwards"][0] <= fwd_serial
