"""The seeded workload generators: shapes, determinism and the stated
distributions (CPU only)."""
import numpy as np
import pytest

from paper_2607_17652_amd import synth
from oracle import pack


@pytest.mark.parametrize("name", synth.WORKLOAD_ORDER)
def test_host_state_is_well_formed_and_seeded(name):
    wl = synth.workload(name)
    h1 = synth.make_host_state(wl, seed=0)
    h2 = synth.make_host_state(wl, seed=0)
    for k in ("tokens", "pe", "fin", "page_table"):
        assert np.array_equal(h1[k], h2[k])
    st = h1["state"]
    assert np.all(st["R"] - st["L"] >= 1) and np.all(st["R"] - st["L"] <= wl.W_max)
    assert np.all(st["R"] <= st["n_blocks"])
    o = st["gen_start"] + st["L"] * wl.bl
    assert np.array_equal(o, h1["o"])
    assert np.all(o % wl.bl == 0) and np.all(o >= wl.bl)
    # every position the step touches is covered by the request's pages
    for b in range(wl.B):
        need = -(-(int(st["gen_start"][b]) + wl.n_blocks * wl.bl) // wl.page_size)
        assert np.all(h1["page_table"][b, :need] >= 0)
    pt = h1["page_table"][h1["page_table"] >= 0]
    assert len(np.unique(pt)) == len(pt) == h1["num_pages"]
    # leftmost live block never starts finished
    for b in range(wl.B):
        assert h1["fin"][b, st["L"][b]] == 0
    pack.pack_wavefronts(st, wl.W_max, wl.bl, wl.layout)   # well formed


def test_tiny_workload_matches_its_description():
    wl = synth.workload("tiny")
    h = synth.make_host_state(wl, seed=0)
    o, w = int(h["o"][0]), int(h["w"][0])
    assert (o, w) == (8, 2)
    win = h["tokens"][0, o:o + w * wl.bl]
    assert int(np.sum(win == wl.mask_id)) == 4      # exactly half of 8 rows


def test_prefix_distributions():
    wl = synth.workload("serve256")
    o = synth.make_host_state(wl, seed=3)["o"]
    assert o.min() >= 128 and o.max() <= 8192
    # log-uniform: the median sits near the geometric mean sqrt(128*8192)=1024
    assert 600 < np.median(o) < 1700
    wl = synth.workload("long8")
    o = synth.make_host_state(wl, seed=0)["o"]
    assert o.min() >= 16384 and o.max() <= 32768


def test_cpu_tensors_and_logits():
    import torch
    wl = synth.workload("tiny")
    h = synth.make_host_state(wl, seed=0)
    t = synth.make_device_tensors(wl, h, seed=0, device="cpu")
    assert t["q"].shape == (wl.row_cap, wl.Hq, wl.d)
    assert t["v_cache"].shape == (h["num_pages"], wl.Hkv, wl.d, wl.page_size)
    assert t["logits"].dtype == torch.float32
    z = t["logits"].double().numpy()
    top2 = np.sort(z, axis=1)[:, -2:]
    planted = np.isclose(top2[:, 1] - top2[:, 0], 4.0, atol=1e-4)
    assert planted.sum() >= 1
    t2 = synth.make_device_tensors(wl, h, seed=0, device="cpu")
    assert torch.equal(t["logits"], t2["logits"])
