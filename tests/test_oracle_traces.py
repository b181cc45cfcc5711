"""Hand-worked traces of the update rules, pinning the oracle's Eq. 1 / Eq. 2 /
Eq. 3 / Sec. 3.1 / Alg. 1 logic step by step.

Shared setting: V = 5, mask id 4 ([M]), bl = 2, n = 3 blocks (B0 = positions
0-1, B1 = 2-3, B2 = 4-5), W = 2, tau_mask = 0.9, tau_edit = 0.8, theta = 0.5,
S_pe = 1, no EOS, no prompt.  A row's logits "(a, k)" are a at index k and 0
elsewhere, so its confidence is e^a / (e^a + 4):
  a=4 -> 0.9317 (> tau_mask), a=3 -> 0.8339 (between the thresholds),
  a=2 -> 0.6488, a=0 -> 0.2 with the argmax tie going to index 0.
Every expected value below was derived by hand from the paper's rules, not by
running the oracle.
"""
import numpy as np
import pytest

from oracle import pack, update

M = 4
V = 5


def params(**kw):
    p = dict(tau_mask=0.9, tau_edit=0.8, theta=0.5, mask_id=M, eos_id=-1,
             S_pe=1, W=2, edit_masked=False, force_progress=False)
    p.update(kw)
    return p


def init(tokens, L=0, R=1, n=3, prompt_len=0, bl=2):
    state = dict(gen_start=np.array([0]), prompt_len=np.array([prompt_len]),
                 n_blocks=np.array([n]), L=np.array([L]), R=np.array([R]),
                 active=np.array([1]), eos_hit=np.array([0]))
    return dict(state=state, tokens=np.array([tokens], dtype=np.int64),
                pe=np.zeros((1, n), dtype=np.int64),
                fin=np.zeros((1, n), dtype=np.int64), bl=bl)


def row(a, k):
    z = np.zeros(V)
    z[k] = a
    return z


def step(sim, logits_by_pos, prm, W_max=2):
    packed = pack.pack_wavefronts(sim["state"], W_max, sim["bl"], pack.RAGGED)
    rows = np.zeros((packed["cap"], V))
    for r in range(packed["cap"]):
        if packed["row_req"][r] >= 0:
            rows[r] = row(*logits_by_pos[int(packed["row_pos"][r])])
    live = packed["row_req"] >= 0
    xhat = np.full(packed["cap"], -1)
    p64 = np.zeros(packed["cap"])
    xhat[live], p64[live] = update.vocab_reduce(rows[live])
    res = update.denoise_update(xhat, p64, sim["tokens"], sim["state"],
                                sim["pe"], sim["fin"], packed, prm)
    sim.update(state=res["state"], tokens=res["tokens"], pe=res["pe"],
               fin=res["fin"])
    return res


def LR(sim):
    return int(sim["state"]["L"][0]), int(sim["state"]["R"][0])


T1_LOGITS = [
    {0: (4, 1), 1: (2, 2)},
    {0: (4, 1), 1: (4, 2), 2: (4, 3), 3: (3, 0)},
    {0: (4, 1), 1: (4, 2), 2: (3, 0), 3: (4, 1)},
    {2: (0, 0), 3: (4, 1), 4: (4, 0), 5: (4, 4)},
    {4: (4, 0), 5: (4, 3)},
    {4: (4, 0), 5: (4, 3)},
]


def test_trace_T1_full_decode():
    sim = init([M] * 6)
    prm = params()
    # Step 1: pos0 (4,1) is M2T; pos1 (2,2) stays masked.  B0: 1 of 2 masks
    # decodable -> rho = 0.5 >= theta, window not full -> admit B1.
    r = step(sim, T1_LOGITS[0], prm)
    assert list(sim["tokens"][0]) == [1, M, M, M, M, M]
    assert LR(sim) == (0, 2)
    assert r["stats"][0]["m2t"] == 1 and r["stats"][0]["spawned"] == 1
    assert r["stats"][0]["rho"] == 0.5
    # Step 2: pos1, pos2 M2T; pos3 (3,0) is between the thresholds and masked:
    # no M2T, and T2T does not apply to a masked position.  B0 lost its last
    # mask but S_pe = 1 > 0, so it is not finished; window full.
    step(sim, T1_LOGITS[1], prm)
    assert list(sim["tokens"][0]) == [1, 2, 3, M, M, M]
    assert LR(sim) == (0, 2)
    assert list(sim["fin"][0]) == [0, 0, 0]
    # Step 3: B0 unchanged in a post-edit step -> finished, retired.  pos2 is a
    # T2T edit 3 -> 0 (p = 0.834 > 0.8); pos3 M2T -> 1.  B1 rho = 1/1 -> admit B2.
    r = step(sim, T1_LOGITS[2], prm)
    assert list(sim["tokens"][0]) == [1, 2, 0, 1, M, M]
    assert LR(sim) == (1, 3)
    assert r["stats"][0]["t2t"] == 1 and r["stats"][0]["m2t"] == 1
    assert r["stats"][0]["committed"] == 1 and r["stats"][0]["spawned"] == 1
    # Step 4: pos2 all-zero logits -> argmax tie to 0 (= current), p = 0.2.
    # B1 unchanged post-edit -> finished, retired.  pos4 M2T -> 0; pos5 predicts
    # [M] itself: no write, but it still counts as decodable for rho.
    r = step(sim, T1_LOGITS[3], prm)
    assert list(sim["tokens"][0]) == [1, 2, 0, 1, 0, M]
    assert LR(sim) == (2, 3)
    assert r["stats"][0]["rho"] == 1.0
    assert r["argmax"][0] == 0  # row 0 holds pos2 in the ragged layout
    # Step 5: pos5 M2T -> 3.  B2 not finished yet (S_pe = 1).
    step(sim, T1_LOGITS[4], prm)
    assert list(sim["tokens"][0]) == [1, 2, 0, 1, 0, 3]
    assert LR(sim) == (2, 3)
    assert sim["state"]["active"][0] == 1
    # Step 6: unchanged post-edit step -> finished -> retired -> L = n -> done.
    r = step(sim, T1_LOGITS[5], prm)
    assert LR(sim) == (3, 3)
    assert sim["state"]["active"][0] == 0
    assert r["stats"][0]["done"] == 1 and r["stats"][0]["eos"] == 0


def test_trace_T1_edit_masked_reading():
    """The literal Eq. 1 reading: Delta also covers a masked position, so in
    step 2 pos3 (3,0) becomes 0 although it is below tau_mask."""
    sim = init([M] * 6)
    prm = params(edit_masked=True)
    step(sim, T1_LOGITS[0], prm)
    r = step(sim, T1_LOGITS[1], prm)
    assert list(sim["tokens"][0]) == [1, 2, 3, 0, M, M]
    # counted as M2T (a masked position was written)
    assert r["stats"][0]["m2t"] == 3 and r["stats"][0]["t2t"] == 0


def test_trace_T2_eos_stops_at_commit():
    """T1 with eos_id = 2: B0 = [1, 2] commits in step 3 and holds EOS, so the
    request deactivates; the step's own edits still happened; no admission."""
    sim = init([M] * 6)
    prm = params(eos_id=2)
    for k in range(2):
        step(sim, T1_LOGITS[k], prm)
        assert sim["state"]["active"][0] == 1   # EOS checked at commit only
    r = step(sim, T1_LOGITS[2], prm)
    assert list(sim["tokens"][0]) == [1, 2, 0, 1, M, M]
    assert LR(sim) == (1, 2)
    assert sim["state"]["active"][0] == 0 and sim["state"]["eos_hit"][0] == 1
    assert r["stats"][0]["eos"] == 1 and r["stats"][0]["spawned"] == 0


def test_trace_T3_prompt_positions_are_never_edited():
    """prompt_len = 1 with pos0 preset to 3: a confident different prediction
    at pos0 would be a T2T edit, but i in P excludes it (Eq. 1, Delta)."""
    sim = init([3, M, M, M, M, M], prompt_len=1)
    r = step(sim, {0: (4, 1), 1: (2, 2)}, params())
    assert list(sim["tokens"][0]) == [3, M, M, M, M, M]
    # B0 masks: {pos1}; p = 0.649 < 0.9 -> rho = 0 -> no admission
    assert r["stats"][0]["rho"] == 0.0
    assert LR(sim) == (0, 1)


def test_trace_T4_window_of_one_is_serial():
    """W = 1: no admission while B0 is live, even though rho(B0) = 0.5; the
    next block enters in the step that retires B0."""
    sim = init([M] * 6)
    prm = params(W=1)
    step(sim, {0: (4, 1), 1: (2, 2)}, prm, W_max=1)
    assert LR(sim) == (0, 1)
    step(sim, {0: (4, 1), 1: (4, 2)}, prm, W_max=1)
    assert LR(sim) == (0, 1)
    assert list(sim["tokens"][0][:2]) == [1, 2]
    r = step(sim, {0: (4, 1), 1: (4, 2)}, prm, W_max=1)
    assert LR(sim) == (1, 2)
    assert r["stats"][0]["committed"] == 1 and r["stats"][0]["spawned"] == 1


def test_trace_T5_post_edit_cap_and_early_stop():
    """S_pe = 2, one mask-free block [1, 2].  A post-edit step with a change
    gives pe = 1 (not finished); a second with a change reaches the cap."""
    prm = params(S_pe=2)
    sim = init([1, 2], n=1)
    step(sim, {0: (3, 0), 1: (4, 2)}, prm)        # T2T 1 -> 0
    assert list(sim["tokens"][0]) == [0, 2]
    assert sim["pe"][0, 0] == 1 and sim["fin"][0, 0] == 0
    step(sim, {0: (4, 1), 1: (4, 2)}, prm)        # T2T 0 -> 1, pe = 2 = S_pe
    assert list(sim["tokens"][0]) == [1, 2]
    assert sim["pe"][0, 0] == 2
    assert sim["state"]["active"][0] == 0         # finished, retired, L = n
    # Early stop: a post-edit step without change finishes at pe = 1.
    sim = init([1, 2], n=1)
    step(sim, {0: (4, 1), 1: (4, 2)}, prm)
    assert sim["pe"][0, 0] == 1 and sim["state"]["active"][0] == 0


def test_threshold_strictness():
    """Eq. 1 is strict (p > tau) while Eq. 2 is not (p >= tau).  With tau_mask
    set exactly to a row's float32 confidence, the row is decodable for rho
    but is not unmasked."""
    p = np.float32(np.exp(4) / (np.exp(4) + 4))
    prm = params(tau_mask=float(p))
    sim = init([M] * 6)
    r = step(sim, {0: (4, 1), 1: (4, 2)}, prm)
    assert list(sim["tokens"][0][:2]) == [M, M]
    assert r["stats"][0]["rho"] == 1.0


def test_m2t_only_when_tau_edit_above_one():
    """tau_edit > 1 switches T2T off (LLaDA-2.0-style decoding, Sec. 5.1):
    step 3 of T1 no longer edits pos2."""
    sim = init([M] * 6)
    prm = params(tau_edit=1.5)
    for k in range(3):
        step(sim, T1_LOGITS[k], prm)
    assert list(sim["tokens"][0][:4]) == [1, 2, 3, 1]


def test_identity_when_both_thresholds_above_one():
    sim = init([M, 3, M, M, M, M], R=2)
    prm = params(tau_mask=1.5, tau_edit=1.5)
    before = sim["tokens"].copy()
    step(sim, {0: (9, 1), 1: (9, 0), 2: (9, 2), 3: (9, 3)}, prm)
    assert np.array_equal(before, sim["tokens"])


def test_force_progress_flag():
    """With FORCE_PROGRESS, a block whose masks all stay below tau_mask still
    unmasks its most confident masked row (ties to the lowest position)."""
    sim = init([M] * 6)
    step(sim, {0: (2, 1), 1: (3, 2)}, params(force_progress=True))
    assert list(sim["tokens"][0][:2]) == [M, 2]
    sim = init([M] * 6)
    step(sim, {0: (2, 1), 1: (2, 3)}, params(force_progress=True))
    assert list(sim["tokens"][0][:2]) == [1, M]


def test_force_progress_with_edit_masked_counts_each_row_once():
    """With EDIT_MASKED and FORCE_PROGRESS, a masked row revealed by Delta
    (tau_edit < p <= tau_mask) is this step's progress: nothing is forced.
    pos0 (3,2): p = .834 > tau_edit, so Delta writes 2 (counted once, as
    M2T, since the row was masked); pos1 (2,1): p = .649, stays [M].  With
    S_pe = 0 the block still holds a mask, so it is not finished."""
    sim = init([M] * 6)
    prm = params(force_progress=True, edit_masked=True, S_pe=0)
    r = step(sim, {0: (3, 2), 1: (2, 1)}, prm)
    assert list(sim["tokens"][0][:2]) == [2, M]
    assert r["stats"][0]["m2t"] == 1 and r["stats"][0]["t2t"] == 0
    assert sim["fin"][0, 0] == 0
    assert LR(sim) == (0, 1)        # rho(B0) = 0/2 < theta: no admission
    # the same logits without EDIT_MASKED: no row is revealed, so the most
    # confident masked row (pos0, p = .834) is forced
    sim = init([M] * 6)
    r = step(sim, {0: (3, 2), 1: (2, 1)}, params(force_progress=True, S_pe=0))
    assert list(sim["tokens"][0][:2]) == [2, M]
    assert r["stats"][0]["m2t"] == 1


def test_multi_block_retire_in_one_step():
    """Finished blocks behind the leftmost retire together once the leftmost
    finishes (Alg. 1 inner while)."""
    sim = init([1, 2, 3, 0, M, M], L=0, R=2, n=3)
    sim["fin"][0, 1] = 1
    r = step(sim, {0: (4, 1), 1: (4, 2), 2: (4, 3), 3: (4, 0)}, params())
    assert r["stats"][0]["committed"] == 2
    assert LR(sim) == (2, 3)


def test_empty_window_admits_unconditionally():
    """An active request with an empty window admits one block regardless of
    theta (the way Alg. 1 admits B_0)."""
    sim = init([M] * 6, L=1, R=1)
    sim["fin"][0, 0] = 1
    r = step(sim, {}, params(theta=2.0))
    assert LR(sim) == (1, 2)
    assert r["stats"][0]["spawned"] == 1


@pytest.mark.parametrize("theta,expect_R", [(0.0, 3), (-1.0, 3), (0.5, 1)])
def test_admission_loop_with_nonpositive_theta(theta, expect_R):
    """A newly admitted block has rho = 0, so only theta <= 0 admits more than
    one block per step (up to W)."""
    sim = init([M] * 8, n=4)
    step(sim, {0: (2, 1), 1: (2, 2)}, params(theta=theta, W=3), W_max=3)
    assert LR(sim) == (0, expect_R)
