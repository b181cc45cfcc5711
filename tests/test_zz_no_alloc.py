"""fb_denoise_update_noalloc (the update for callers that cannot allocate)
gives exactly what fb_denoise_update gives on the same inputs, on two calls
in a row through the C ABI, the second with a smaller pack and vocabulary
than the first (the library's array keeps the first call's contents)."""
import numpy as np
import pytest
import torch

from harness import gpu_results, log, setup
from paper_2607_17652_amd import binding as fb

pytestmark = pytest.mark.gpu


def _outputs(step):
    g = gpu_results(step)
    return {k: g[k] for k in ("tokens", "pe", "fin", "conf", "argmax")} | {
        "st": step.st.cpu().numpy().copy(), "stats": step.stats.cpu().numpy().copy()}


def _run_both(name, seed, **overrides):
    wl, host, t, step = setup(name, seed, **overrides)
    log(f"[noalloc] workload={name} seed={seed} overrides={overrides} rows={wl.row_cap} "
        f"V={wl.V} ws={fb.fb_update_workspace_bytes(step.pack, wl.V)}")
    pristine = [x.clone() for x in (step.st, step.tokens, step.pe, step.fin)]
    step.pack_step()
    step.update_step()
    torch.cuda.synchronize()
    ref = _outputs(step)
    for dst, src in zip((step.st, step.tokens, step.pe, step.fin), pristine):
        dst.copy_(src)
    step.conf.zero_()
    step.argmax.fill_(-1)
    step.stats.zero_()
    step.pack_step()
    fb.fb_denoise_update_noalloc(t["logits"], step.tokens, step.conf, step.argmax,
                                 step.st, step.pe, step.fin, step.pack, step.params,
                                 step.stats)
    torch.cuda.synchronize()
    got = _outputs(step)
    for k in ref:
        assert np.array_equal(ref[k], got[k]), f"{name}: {k} differs"
    return wl


def test_noalloc_update_equals_the_workspace_update_twice():
    big = _run_both("serve256", 0)
    small = _run_both("single", 1, V=5003, prefix_jitter=7)
    assert small.row_cap < big.row_cap and small.V < big.V
