"""Pins of the multi-step pieces of the oracle: the synthetic model that
stands in for f_theta (SplitMix64 hash model), the decode loop of Alg. 1 on
it, and the batch-synchronous window of the Sec. 5 ablation.  CPU only."""
import math
import os

import numpy as np
import pytest

from oracle import pack, serial, step, synth_model as sm, update

HERE = os.path.dirname(os.path.abspath(__file__))
V = 1000
M = V - 1
# peak heights: p = e^a / (e^a + V - 1) -> 0.288, 0.848, 0.957, 0.994
LEVELS = (6.0, 8.625, 10.0, 12.0)


def golden_splitmix():
    with open(os.path.join(HERE, "golden", "splitmix64_seed1234567.txt")) as f:
        return [int(l) for l in f if l.strip() and not l.startswith("#")]


def test_splitmix64_matches_published_outputs():
    gold = golden_splitmix()
    assert sm.splitmix64_stream(1234567, len(gold)) == gold
    # the counter form used by the model is the same sequence
    assert [sm.H(1234567, n) for n in range(len(gold))] == gold


def _state(gen_start, n, L, R, prompt_len=None):
    B = len(gen_start)
    pl = gen_start if prompt_len is None else prompt_len
    return dict(gen_start=np.array(gen_start), prompt_len=np.array(pl),
                n_blocks=np.full(B, n), L=np.array(L), R=np.array(R),
                active=np.ones(B, dtype=np.int64), eos_hit=np.zeros(B, dtype=np.int64))


def test_model_sees_only_its_visible_prefix():
    """Sec. 4.1: block [lo, hi) depends on tokens [0, hi) only."""
    rng = np.random.default_rng(0)
    x = rng.integers(0, V - 1, size=64)
    x[30:40] = M
    model = sm.make_model(7, LEVELS, V)
    z = model(x, 24, 32, gen_start=16)
    y = x.copy()
    y[32:] = rng.integers(0, V, size=32)
    assert np.array_equal(model(y, 24, 32, gen_start=16), z)
    y = x.copy()
    y[5] = (y[5] + 1) % (V - 1)          # a visible prompt token changes the context
    assert not np.array_equal(model(y, 24, 32, gen_start=16), z)
    y = x.copy()
    y[26] = (y[26] + 1) % (V - 1)        # so does a token of the block itself
    assert not np.array_equal(model(y, 24, 32, gen_start=16), z)


def test_model_rows_are_two_level_with_closed_form_confidence():
    rng = np.random.default_rng(1)
    x = rng.integers(0, V - 1, size=48)
    x[[33, 35, 40]] = M
    model = sm.make_model(3, LEVELS, V)
    z = model(x, 32, 48, gen_start=16)
    xhat, p = update.vocab_reduce(z)
    for i in range(16):
        nz = np.flatnonzero(z[i])
        assert len(nz) == 1 and nz[0] == xhat[i] and xhat[i] != M
        a = z[i, nz[0]]
        assert a in LEVELS
        assert abs(p[i] - math.exp(a) / (math.exp(a) + V - 1)) < 1e-15
    assert z[1, xhat[1]] == LEVELS[3]      # position 33: the block's first mask


def test_model_predicts_true_tokens_when_upstream_is_complete():
    rng = np.random.default_rng(2)
    x = rng.integers(0, V - 1, size=40)
    x[32:40] = M
    preds = sm.block_predictions(5, x, 32, 40, 8, V)
    assert [k for k, _ in preds] == [sm.true_token(5, p, V) for p in range(32, 40)]
    x[20] = M                          # one upstream mask: some drafts go stale
    preds = sm.block_predictions(5, x, 32, 40, 8, V)
    assert any(k != sm.true_token(5, p, V) for p, (k, _) in zip(range(32, 40), preds))


def loop_params(**kw):
    p = dict(tau_mask=0.9, tau_edit=0.8, theta=0.5, mask_id=M, eos_id=-1,
             S_pe=2, W=2, edit_masked=False, force_progress=False)
    p.update(kw)
    return p


def fresh(prompts, n, bl, seed=0):
    rng = np.random.default_rng(seed)
    B = len(prompts)
    T = max(prompts) + n * bl
    x = np.full((B, T), M, dtype=np.int64)
    for b, pl in enumerate(prompts):
        x[b, :pl] = rng.integers(0, V - 1, size=pl)
    st = _state(list(prompts), n, [0] * B, [1] * B)
    z = np.zeros((B, n), dtype=np.int64)
    return st, x, z


@pytest.mark.parametrize("S_pe", [1, 2])
def test_serial_decoding_of_the_model_reaches_the_true_tokens(S_pe):
    """With W = 1 no block is drafted on stale context, so every revealed token
    is the true one and no edit happens: the serial decoder and the loop both
    end on the true sequence, in the same number of forwards."""
    bl, n, prompt = 8, 4, 5
    st, x, z = fresh([prompt], n, bl)
    model = sm.make_model(11, LEVELS, V)
    prm = loop_params(W=1, S_pe=S_pe)
    ser, fwd, committed = serial.serial_decode(model, x[0], prompt, prompt, n, bl, prm)
    truth = [sm.true_token(11, p, V) for p in range(prompt, prompt + n * bl)]
    assert list(ser[prompt:]) == truth and committed == n
    res = step.gwd_loop(model, st, x, z, z, prm, 1, bl, pack.RAGGED)
    assert np.array_equal(res["tokens"][0], ser)
    assert res["forwards"][0] == fwd


def test_wavefront_drafts_early_and_edits_on_the_model():
    """W = 3 with a permissive gate: blocks are admitted over masked upstream
    blocks, some drafts are stale and get edited (T2T), and the loop needs
    fewer forwards than serial decoding."""
    bl, n, prompt = 8, 6, 4
    st, x, z = fresh([prompt], n, bl, seed=3)
    model = sm.make_model(21, LEVELS, V)
    prm = loop_params(W=3, theta=0.25)
    _, fwd_serial, _ = serial.serial_decode(model, x[0], prompt, prompt, n, bl,
                                            dict(prm, W=1))
    res = step.gwd_loop(model, st, x, z, z, prm, 3, bl, pack.RAGGED)
    assert res["state"]["L"][0] == n and not res["state"]["active"][0]
    assert res["forwards"][0] < fwd_serial


@pytest.mark.parametrize("W,theta,seed", [(1, 0.5, 0), (2, 0.5, 1), (3, 0.25, 2),
                                          (4, 0.0, 3)])
def test_synchronous_window_with_one_request_equals_hwp(W, theta, seed):
    """Sec. 5 ablation: with B = 1 the synchronous wavefront and HWP are the
    same schedule."""
    bl, n = 8, 5
    st, x, z = fresh([6], n, bl, seed)
    model = sm.make_model(seed + 100, LEVELS, V)
    prm = loop_params(W=W, theta=theta)
    a = step.gwd_loop(model, st, x, z, z, prm, W, bl, pack.RAGGED)
    b = step.gwd_loop(model, st, x, z, z, dict(prm, sync_window=True), W, bl,
                      pack.RAGGED)
    assert np.array_equal(a["tokens"], b["tokens"])
    assert a["steps"] == b["steps"]
    assert np.array_equal(a["forwards"], b["forwards"])


def test_synchronous_batch_keeps_one_window_and_hwp_batch_equals_alone():
    bl, n, W = 8, 5, 3
    prompts = [3, 9, 6]
    st, x, z = fresh(prompts, n, bl, seed=5)
    model = sm.make_model(77, LEVELS, V)
    prm = loop_params(W=W, theta=0.25)
    hwp = step.gwd_loop(model, st, x, z, z, prm, W, bl, pack.PADDED)
    for b in range(3):
        s1 = {k: v[b:b + 1].copy() for k, v in st.items()}
        r1 = step.gwd_loop(model, s1, x[b:b + 1], z[:1], z[:1], prm, W, bl,
                           pack.RAGGED)
        assert np.array_equal(r1["tokens"][0], hwp["tokens"][b])
        assert r1["forwards"][0] == hwp["forwards"][b]
    # the synchronous loop raises if the windows ever diverge; every request
    # is stepped in every forward until all are done
    syn = step.gwd_loop(model, st, x, z, z, dict(prm, sync_window=True), W, bl,
                        pack.RAGGED)
    assert np.all(syn["state"]["L"] == n)
    assert np.all(syn["forwards"] == syn["steps"])
    assert syn["steps"] >= max(hwp["forwards"])


# ---- hand trace of the synchronous gate ------------------------------------
# V = 5, [M] = 4, bl = 2, n = 3, W = 2; "(a, k)" is a row with a at index k and
# 0 elsewhere, p = e^a / (e^a + 4): a=4 -> 0.932, a=2 -> 0.649.
V5, M5 = 5, 4


def _row(a, k):
    z = np.zeros(V5)
    z[k] = a
    return z


def _one_step(state, tokens, pe, fin, logits_by_req_pos, prm):
    packed = pack.pack_wavefronts(state, 2, 2, pack.RAGGED)
    xhat = np.full(packed["cap"], -1)
    p64 = np.zeros(packed["cap"])
    for r in range(packed["cap"]):
        b = packed["row_req"][r]
        if b >= 0:
            xh, p = update.vocab_reduce(_row(*logits_by_req_pos[b][packed["row_pos"][r]])[None])
            xhat[r], p64[r] = xh[0], p[0]
    return update.denoise_update(xhat, p64, tokens, state, pe, fin, packed, prm)


def _two_requests():
    st = dict(gen_start=np.array([0, 0]), prompt_len=np.array([0, 0]),
              n_blocks=np.array([3, 3]), L=np.array([0, 0]), R=np.array([2, 2]),
              active=np.array([1, 1]), eos_hit=np.array([0, 0]))
    tokens = np.array([[1, 2, M5, M5, M5, M5],
                       [1, M5, M5, M5, M5, M5]], dtype=np.int64)
    z = np.zeros((2, 3), dtype=np.int64)
    return st, tokens, z


def test_synchronous_retire_waits_for_every_request():
    """Request 0 finishes B0 (a post-edit step with no change) and would retire
    and admit on its own; request 1's B0 still has a mask, so the shared window
    does not move."""
    prm = dict(tau_mask=0.9, tau_edit=0.8, theta=0.5, mask_id=M5, eos_id=-1,
               S_pe=1, W=2)
    logits = [{0: (4, 1), 1: (4, 2), 2: (4, 1), 3: (4, 2)},
              {0: (4, 1), 1: (2, 3), 2: (4, 0), 3: (2, 1)}]
    st, tok, z = _two_requests()
    hwp = _one_step(st, tok, z, z, logits, prm)
    assert (hwp["state"]["L"][0], hwp["state"]["R"][0]) == (1, 3)   # retire + admit
    assert (hwp["state"]["L"][1], hwp["state"]["R"][1]) == (0, 2)
    syn = _one_step(st, tok, z, z, logits, dict(prm, sync_window=True))
    assert list(syn["state"]["L"]) == [0, 0] and list(syn["state"]["R"]) == [2, 2]
    assert syn["fin"][0, 0] == 1 and syn["fin"][1, 0] == 0
    # the tokens are the same either way: only retire/admit differ
    assert np.array_equal(hwp["tokens"], syn["tokens"])


@pytest.mark.parametrize("theta,admitted", [(0.5, True), (0.6, False)])
def test_synchronous_admission_uses_the_minimum_readiness(theta, admitted):
    """Both requests finish B0 and retire it together; the gate then sees
    rho(B1) = 1 for request 0 and 1/2 for request 1: the batch admits B2 only if
    the smaller one passes theta (HWP would admit request 0 at theta = 0.6)."""
    prm = dict(tau_mask=0.9, tau_edit=0.8, theta=theta, mask_id=M5, eos_id=-1,
               S_pe=1, W=2)
    st, tok, z = _two_requests()
    tok[1, 1] = 3
    logits = [{0: (4, 1), 1: (4, 2), 2: (4, 1), 3: (4, 2)},
              {0: (4, 1), 1: (4, 3), 2: (4, 0), 3: (2, 1)}]
    syn = _one_step(st, tok, z, z, logits, dict(prm, sync_window=True))
    assert list(syn["state"]["L"]) == [1, 1]
    assert list(syn["state"]["R"]) == ([3, 3] if admitted else [2, 2])
    hwp = _one_step(st, tok, z, z, logits, prm)
    assert hwp["state"]["R"][0] == 3
    assert hwp["state"]["R"][1] == (3 if admitted else 2)


# ---- LM head with the fused vocabulary reduction ---------------------------
def test_lmhead_reduce_is_the_reduction_of_the_product():
    from oracle import lmhead
    rng = np.random.default_rng(4)
    H = rng.standard_normal((5, 16))
    Wt = rng.standard_normal((37, 16))
    xh, p = lmhead.lmhead_reduce(H, Wt)
    Z = np.array([[sum(H[r, i] * Wt[v, i] for i in range(16)) for v in range(37)]
                  for r in range(5)])                  # the product, written out
    for r in range(5):
        assert xh[r] == int(np.argmax(Z[r]))
        assert abs(p[r] - 1.0 / math.fsum(math.exp(z - Z[r].max()) for z in Z[r])) < 1e-14


def test_lmhead_identity_weight_reduces_the_hidden_rows():
    """W = I (V = D): the logits are the hidden rows themselves."""
    from oracle import lmhead
    rng = np.random.default_rng(5)
    H = rng.standard_normal((4, 12))
    xh, p = lmhead.lmhead_reduce(H, np.eye(12))
    x2, p2 = update.vocab_reduce(H)
    assert np.array_equal(xh, x2) and np.allclose(p, p2, rtol=0, atol=1e-15)


def test_lmhead_two_level_closed_form():
    """One hidden direction picked out by one weight row: z = a at k, 0
    elsewhere, p = e^a / (e^a + V - 1); a weight of a non-square shape
    catches a transposed operand."""
    from oracle import lmhead
    V, D, k, a = 50, 8, 17, 3.0
    H = np.zeros((1, D))
    H[0, 2] = a
    Wt = np.zeros((V, D))
    Wt[k, 2] = 1.0
    xh, p = lmhead.lmhead_reduce(H, Wt)
    assert xh[0] == k
    assert abs(p[0] - math.exp(a) / (math.exp(a) + V - 1)) < 1e-15


def test_lmhead_accumulation_bound_covers_float32_products():
    from oracle import lmhead
    rng = np.random.default_rng(6)
    H = rng.standard_normal((6, 512)).astype(np.float32)
    Wt = rng.standard_normal((40, 512)).astype(np.float32)
    exact = lmhead.lm_logits(H, Wt)
    f32 = np.zeros((6, 40), dtype=np.float32)
    for i in range(512):                       # sequential float32 accumulation
        f32 = (f32 + np.outer(H[:, i], Wt[:, i]).astype(np.float32)).astype(np.float32)
    bound = lmhead.accumulation_bound(H, Wt)
    assert np.all(np.abs(f32 - exact).max(axis=1) <= bound)


# ---- RoPE and the window prologue ------------------------------------------
def test_rope_position_zero_is_identity_and_norms_are_kept():
    from oracle import rope
    rng = np.random.default_rng(8)
    x = rng.standard_normal((5, 3, 16))
    assert np.allclose(rope.rope(x, np.zeros(5), 10000.0), x, atol=1e-15)
    y = rope.rope(x, rng.integers(0, 50000, size=5), 10000.0)
    # each (j, j + d/2) pair keeps its length
    pn = lambda z: z[..., :8] ** 2 + z[..., 8:] ** 2
    assert np.allclose(pn(y), pn(x), rtol=1e-12)


def test_rope_scores_depend_on_relative_position_only():
    """<rope(q, m), rope(k, n)> is a function of m - n: the property RoPE is
    built for (RoFormer, Sec. 3.4)."""
    from oracle import rope
    rng = np.random.default_rng(9)
    q = rng.standard_normal((1, 1, 32))
    k = rng.standard_normal((1, 1, 32))
    dot = lambda m, n: float(np.sum(rope.rope(q, [m], 500.0) * rope.rope(k, [n], 500.0)))
    assert abs(dot(7, 3) - dot(1007, 1003)) < 1e-10
    assert abs(dot(3, 7) - dot(40, 44)) < 1e-10
    assert abs(dot(7, 3) - dot(3, 7)) > 1e-6          # but not symmetric in general


def test_rope_matches_the_complex_rotation():
    """Pair j as the complex number x_j + i x_{j+d/2} is multiplied by
    e^(i p theta_j), theta_j = base^(-2j/d)."""
    from oracle import rope
    rng = np.random.default_rng(10)
    x = rng.standard_normal((1, 1, 8))
    p, base = 123, 10000.0
    y = rope.rope(x, [p], base)[0, 0]
    for j in range(4):
        z = complex(x[0, 0, j], x[0, 0, j + 4]) * np.exp(1j * p * base ** (-2 * j / 8))
        assert abs(y[j] - z.real) < 1e-12 and abs(y[j + 4] - z.imag) < 1e-12


def test_window_prologue_rotates_live_rows_and_writes_only_the_window():
    from oracle import rope
    from oracle import pack as opack
    st = _state([4, 9], 3, [0, 1], [2, 3])
    packed = opack.pack_wavefronts(st, 2, 4, opack.PADDED)
    rng = np.random.default_rng(11)
    cap = packed["cap"]
    q = rng.standard_normal((cap, 2, 8))
    kn = rng.standard_normal((cap, 1, 8))
    vn = rng.standard_normal((cap, 1, 8))
    K = [rng.standard_normal((30, 1, 8)) for _ in range(2)]
    V = [rng.standard_normal((30, 1, 8)) for _ in range(2)]
    q2, K2, V2 = rope.window_prologue(q, kn, vn, K, V, packed, 10000.0)
    dead = packed["row_req"] < 0
    assert np.array_equal(q2[dead], q[dead])
    for r in np.flatnonzero(~dead):
        b, p = packed["row_req"][r], packed["row_pos"][r]
        assert np.allclose(q2[r], rope.rope(q[r][None], [p], 10000.0)[0], atol=1e-15)
        assert np.allclose(K2[b][p], rope.rope(kn[r][None], [p], 10000.0)[0], atol=1e-15)
        assert np.array_equal(V2[b][p], vn[r])
    o0 = 4 + 0 * 4
    assert np.array_equal(K2[0][:o0], K[0][:o0])          # frozen prefix untouched
