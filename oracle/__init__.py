"""Plain fp64 CPU oracle for the FlowBlock packed wavefront denoising step.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, calls or links
this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may use it.  It shares no code, constants
or helpers with the HIP path (``paper_2607_17652_amd``) and imports nothing
from it; both sides are fed the same arrays by the caller.

Every function states the passage of the paper (FlowBlock, arxiv 2607.17652)
it follows.  The arithmetic is written as the plain definition, in float64,
with numpy matmul / exp / max as library primitives and no blocking, fusion or
reordering beyond what the definition states:

* ``pack``       -- Eq. 4 (per-row gather into a dense [B, q] batch), plus the
                    ragged variant that drops padding slots.
* ``attention``  -- Sec. 4.1 "W-shaped block-causal attention" and Eq. 5:
                    block ``s`` of request ``b`` sees keys ``[0, o_b + (s+1) bl)``;
                    Eq. 6 window KV write-back on logical per-request arrays.
* ``bruteforce`` -- Eq. 5 applied literally on the paper's physical tail layout
                    with an explicit dense mask (an independent check of
                    ``attention``).
* ``update``     -- Eq. 1 (joint M2T/T2T update), Eq. 2 (readiness),
                    Sec. 3.1 post-edit steps, Alg. 1 retire / gated admit, Eq. 3.
* ``serial``     -- an independently written serial block-wise decoder (one
                    block at a time), the W = 1 special case of Alg. 1.
* ``step``       -- one whole wavefront step = pack, KV write, attention, update;
                    the multi-step loop of Alg. 1, per-request windows (HWP) or
                    one shared window (the synchronous variant of the Sec. 5
                    ablation).
* ``synth_model`` -- a deterministic SplitMix64 hash model standing in for
                    f_theta in the loop (no weights exist here), with the
                    block-causal visibility of Sec. 4.1.

Readings of points the paper leaves open (all shared with the HIP path by
specification, never by code) are listed in ``READINGS`` below.
"""

READINGS = {
    "delta_masked": "Delta (T2T) excludes masked positions unless the "
                    "EDIT_MASKED flag is set (literal Eq. 1).",
    "strictness": "Eq. 1 uses p > tau; Eq. 2 and Eq. 3 use >= (as printed).",
    "rho_set": "rho counts the masked set of x_t, before this step's update.",
    "rho_new_block": "A block admitted in this step has rho = 0; an empty "
                     "window after retirement admits one block unconditionally.",
    "argmax_ties": "Lowest vocabulary index wins.",
    "xhat_mask": "A prediction equal to mask_id is never written.",
    "post_edit": "A post-edit step is one that starts with no masks in the "
                 "block; fin after a post-edit step with no change or S_pe of them.",
    "fin_sticky": "fin is sticky once set.",
    "eos": "EOS is checked in a block at commit only; eos_id < 0 disables it.",
    "precision": "Confidence is rounded to float32 before the threshold "
                 "compares (the kernel's precision); rows with |p64 - tau| < 1e-5 "
                 "are flagged.",
    "scale": "Softmax scale 1/sqrt(d); query head h reads kv-head h // (Hq/Hkv).",
}

from . import pack, attention, bruteforce, update, serial, step, synth_model  # noqa: E402,F401
