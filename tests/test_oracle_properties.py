"""Properties of the oracle's update (Eq. 1-3, Alg. 1) that hold for any
state, logits and thresholds, checked on random small workloads:

- the frontier only moves forward: L' >= L, R' >= R, L' <= R' <= n and the
  window never holds more than W blocks (Alg. 1);
- only rows of the window that was live at the start of the step change
  (Eq. 1 writes the live rows; admission adds masked blocks only);
- prompt positions never change (Eq. 1 excludes them) and nothing is
  remasked (reading 6), so the masked count never grows;
- fin is sticky, and an inactive request is left as it is;
- with tau_edit above 1 no revealed token changes (T2T needs p > tau_edit),
  and with both thresholds above 1 (no forced progress) no token changes.
"""
import numpy as np
from hypothesis import given, settings, strategies as st

from oracle import pack, update
from paper_2607_17652_amd import synth


def run(seed, tau_mask, tau_edit, theta, edit_masked, force, inactive):
    wl = synth.workload("tiny", V=40, B=6, n_blocks=6, W_max=3, prefix=("uniform", 0, 13),
                        window=("uniform", 1, 3), mask=synth.MASK_BLOCK_UNIFORM)
    h = synth.make_host_state(wl, seed)
    state = {k: v.copy() for k, v in h["state"].items()}
    state["active"][:] = [0 if (inactive >> b) & 1 else 1 for b in range(wl.B)]
    packed = pack.pack_wavefronts(state, wl.W_max, wl.bl, pack.RAGGED)
    rng = np.random.default_rng(seed + 17)
    cap = packed["cap"]
    sigma = rng.choice([0.5, 3.0, 9.0], size=(cap, 1))
    z = rng.normal(size=(cap, wl.V)) * sigma
    live = packed["row_req"] >= 0
    xhat = np.full(cap, -1)
    p64 = np.zeros(cap)
    xhat[live], p64[live] = update.vocab_reduce(z[live])
    prm = dict(wl.params(), tau_mask=tau_mask, tau_edit=tau_edit, theta=theta,
               edit_masked=edit_masked, force_progress=force)
    res = update.denoise_update(xhat, p64, h["tokens"], state, h["pe"], h["fin"], packed, prm)
    return wl, h, state, res, prm


PARAMS = dict(
    seed=st.integers(0, 10_000),
    tau_mask=st.floats(0.05, 0.99),
    tau_edit=st.floats(0.05, 1.5),
    theta=st.floats(-0.5, 1.0),
    edit_masked=st.booleans(),
    force=st.booleans(),
    inactive=st.integers(0, 63),
)


@settings(max_examples=80, deadline=None)
@given(**PARAMS)
def test_update_invariants(seed, tau_mask, tau_edit, theta, edit_masked, force, inactive):
    wl, h, s0, res, prm = run(seed, tau_mask, tau_edit, theta, edit_masked, force, inactive)
    s1, tok0, tok1 = res["state"], h["tokens"], res["tokens"]
    M, bl = wl.mask_id, wl.bl
    for b in range(wl.B):
        L0, R0, L1, R1 = (int(s0["L"][b]), int(s0["R"][b]), int(s1["L"][b]), int(s1["R"][b]))
        n, g = int(s0["n_blocks"][b]), int(s0["gen_start"][b])
        assert L1 >= L0 and R1 >= R0 and L1 <= R1 <= n and R1 - L1 <= prm["W"], (b, L0, R0, L1, R1)
        assert np.all(res["fin"][b] >= h["fin"][b])
        if not s0["active"][b]:
            assert (L1, R1) == (L0, R0) and np.array_equal(tok1[b], tok0[b])
            assert not s1["active"][b]
            continue
        changed = np.flatnonzero(tok1[b] != tok0[b])
        lo, hi = g + L0 * bl, g + R0 * bl
        assert np.all((changed >= lo) & (changed < hi)), (b, changed, lo, hi)
        assert np.all(changed >= int(s0["prompt_len"][b]))
        assert not np.any((tok0[b] != M) & (tok1[b] == M)), b
        if tau_edit > 1.0:
            assert np.all(tok0[b][changed] == M), b


@settings(max_examples=30, deadline=None)
@given(seed=st.integers(0, 10_000), theta=st.floats(-0.5, 1.0), edit_masked=st.booleans())
def test_no_token_changes_when_both_thresholds_exceed_one(seed, theta, edit_masked):
    wl, h, s0, res, prm = run(seed, 1.01, 1.2, theta, edit_masked, False, 0)
    assert np.array_equal(res["tokens"], h["tokens"])
