"""The bench's algorithmic work (the numerators of its roofline entries and
of its tokens/s) recounted from the oracle's own pack (Eq. 4): every live
row, every (row, query head, visible key) triple of Eq. 5 at 4*d flops, and
each request's K/V read once plus Q and O.  Host-side only."""
import numpy as np
import pytest

import bench
from oracle import pack as opack
from paper_2607_17652_amd import synth


def recount(wl, host):
    p = opack.pack_wavefronts(host["state"], wl.W_max, wl.bl, wl.layout)
    elt = 2 if wl.dtype == "bf16" else 4
    rows = int((p["row_req"] >= 0).sum())
    flops = 0.0
    keys_of = {}
    for t in p["tiles"]:
        # bl query positions x Hq heads, each against kv_len keys: q.k and p.v
        # are 2*d flops apiece
        flops += wl.bl * wl.Hq * t["kv_len"] * (2 * wl.d + 2 * wl.d)
        keys_of[t["b"]] = max(keys_of.get(t["b"], 0), t["kv_len"])
    kv = sum(2 * wl.Hkv * wl.d * elt * k for k in keys_of.values())
    qo = 2 * rows * wl.Hq * wl.d * elt
    return rows, flops, kv + qo


@pytest.mark.parametrize("name", ["tiny", "single", "hetero64", "long8", "serve256"])
def test_bench_work_equals_a_recount_from_the_oracle_pack(name):
    wl = synth.workload(name)
    host = synth.make_host_state(wl, 0)
    n_live, flops, nbytes = bench.workload_work(wl, host)
    rows, flops2, nbytes2 = recount(wl, host)
    assert n_live == rows
    assert flops == pytest.approx(flops2, rel=1e-12)
    assert nbytes == pytest.approx(nbytes2, rel=1e-12)


def test_serve256_live_rows_and_logit_bytes():
    """The figures the bench's headline and vocab roofline are quoted on:
    20416 live rows at seed 0, so 6.418 GB of bf16 logits per step, plus one
    16-byte partial per row and vocabulary share (two shares at this size)."""
    wl = synth.workload("serve256")
    n_live, _, _ = bench.workload_work(wl, synth.make_host_state(wl, 0))
    assert n_live == 20416
    assert n_live * wl.V * 2 == 6418137088
    assert n_live * wl.V * 2 + n_live * 2 * 16 == 6418790400


def test_inactive_requests_add_no_work():
    wl = synth.workload("hetero64")
    host = synth.make_host_state(wl, 0)
    full = bench.workload_work(wl, host)
    st = host["state"]
    st["active"] = np.array(st["active"]).copy()
    b = int(np.flatnonzero(st["active"])[0])
    st["active"][b] = 0
    less = bench.workload_work(wl, host)
    rows, flops, nbytes = recount(wl, host)
    assert less == (rows, pytest.approx(flops, rel=1e-12), pytest.approx(nbytes, rel=1e-12))
    assert less[0] < full[0] and less[1] < full[1]
