"""Planted mistakes: each case copies the oracle to a temporary directory,
plants one plausible bug in the copy (a flipped comparison, a dropped term, a
wrong index, a sign error, a transposed mapping) and checks that the pin
suites fail against it.  The real oracle is never modified.  CPU only."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MUTATIONS = [
    ("update.py", "return float(conf32) > tau", "return float(conf32) >= tau",
     "Eq. 1 strict threshold made non-strict"),
    ("update.py", "and not prompt\n", "\n", "prompt positions made editable"),
    ("update.py", "in_delta = ((edit_masked or not masked)",
     "in_delta = ((True)", "T2T allowed on masked positions"),
    ("update.py", "float(dec) / float(m_before)",
     "float(dec) / float(max(m_after, 1))", "rho over the post-update masks"),
    ("update.py", "and fin[b, st[\"L\"][b]]:", "and fin[b, st[\"R\"][b] - 1]:",
     "retirement not in order"),
    ("update.py", "np.flatnonzero(z[r] == m[r])[0]",
     "np.flatnonzero(z[r] == m[r])[-1]", "argmax ties to the highest index"),
    ("update.py", "np.exp(z - m[:, None])", "np.exp(m[:, None] - z)",
     "sign error in the softmax normaliser"),
    ("update.py", "if u == 0 or pe[b, g] >= S_pe:", "if pe[b, g] >= S_pe:",
     "post-edit early stop dropped"),
    ("update.py", "if force and m_before > 0 and revealed == 0:",
     "if force and m_before > 0:",
     "forced progress also where a masked row was revealed"),
    ("step.py", "out = attention.window_attention(q, K, V, packed, Hq, Hkv, sm_scale)",
     "out = attention.window_attention(q, K_prefix, V_prefix, packed, Hq, Hkv, sm_scale)",
     "whole step attends over the caches before the window write"),
    ("step.py", "xhat[rows], p64[rows] = update.vocab_reduce(z)",
     "xhat[rows[::-1]], p64[rows[::-1]] = update.vocab_reduce(z)",
     "whole step reduces the logits of the wrong rows"),
    ("step.py", "res = update.denoise_update(xhat, p64, tokens, state, pe, fin, packed,\n                                params)\n    return dict(packed",
     "res = update.denoise_update(xhat, p64, tokens, state, pe, fin, packed,\n                                dict(params, theta=1.0))\n    return dict(packed",
     "whole step drops the caller's admission gate"),
    ("pack.py", "row0 = (next_ragged_block + s) * bl", "row0 = (b + s) * bl",
     "ragged rows overlap"),
    ("pack.py", "kv_len=o_b + (s + 1) * bl", "kv_len=o_b + s * bl",
     "block does not see itself"),
    ("attention.py", "c = h // g", "c = h % Hkv", "GQA head mapping transposed"),
    ("attention.py", "sm_scale = 1.0 / np.sqrt(d)", "sm_scale = 1.0 / d",
     "softmax scale"),
    ("attention.py", "S = S - S.max(axis=1, keepdims=True)\n    P = np.exp(S)\n    P = P / P.sum(axis=1, keepdims=True)",
     "P = np.exp(S)", "softmax not normalised"),
    ("update.py", "all(fin[b, L] for b in act)", "any(fin[b, L] for b in act)",
     "synchronous retire on any() instead of all()"),
    ("update.py", "min(_rho_of(rho_of[b], R - 1, L) for b in act)",
     "max(_rho_of(rho_of[b], R - 1, L) for b in act)",
     "synchronous gate on the largest readiness"),
    ("synth_model.py", "z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64",
     "z = ((z ^ (z >> 26)) * 0x94D049BB133111EB) & MASK64", "hash mix shift"),
    ("synth_model.py", "    for j in range(hi):\n", "    for j in range(lo):\n",
     "model context misses the block's own tokens"),
    ("synth_model.py", "for j in range(gen_start, lo) if int(x[j]) == mask_id)",
     "for j in range(gen_start, hi) if int(x[j]) == mask_id)",
     "staleness counts the block's own masks"),
    ("synth_model.py", "lvl = 3 if p == first else (h >> 32) % 4",
     "lvl = (h >> 32) % 4", "no guaranteed reveal per forward"),
    ("lmhead.py", "@ np.asarray(weight, dtype=np.float64).T",
     "@ np.asarray(weight, dtype=np.float64)[:, :hidden.shape[0]]",
     "LM head takes the wrong operand orientation"),
    ("lmhead.py", "gamma = D * u / (1.0 - D * u)", "gamma = u",
     "accumulation bound without the length factor"),
    ("rope.py", "[lo * c - hi * s, hi * c + lo * s]", "[lo * c + hi * s, hi * c - lo * s]",
     "RoPE rotates the wrong way"),
    ("rope.py", "inv = base ** (-2.0 * j / d)", "inv = base ** (-1.0 * j / d)",
     "RoPE frequency exponent"),
]


def _plant(tmp, fname, old, new):
    dst = os.path.join(tmp, "oracle")
    shutil.copytree(os.path.join(ROOT, "oracle"), dst,
                    ignore=shutil.ignore_patterns("__pycache__"))
    tdst = os.path.join(tmp, "tests")
    os.makedirs(tdst)
    for f in ("conftest.py", "test_oracle_pins.py", "test_oracle_traces.py",
              "test_oracle_loop.py"):
        shutil.copy(os.path.join(ROOT, "tests", f), tdst)
    shutil.copytree(os.path.join(ROOT, "tests", "golden"),
                    os.path.join(tdst, "golden"))
    path = os.path.join(dst, fname)
    src = open(path).read()
    assert src.count(old) == 1, f"mutation anchor not unique in {fname}: {old!r}"
    with open(path, "w") as f:
        f.write(src.replace(old, new))


@pytest.mark.parametrize("fname,old,new,what", MUTATIONS,
                         ids=[m[3] for m in MUTATIONS])
def test_pins_catch_planted_mistake(tmp_path, fname, old, new, what):
    _plant(str(tmp_path), fname, old, new)
    env = dict(os.environ, PYTHONDONTWRITEBYTECODE="1")
    proc = subprocess.run(
        [sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
         "tests/test_oracle_pins.py", "tests/test_oracle_traces.py",
         "tests/test_oracle_loop.py"],
        cwd=str(tmp_path), env=env, capture_output=True, text=True, timeout=300)
    assert proc.returncode != 0, f"pins did not catch: {what}\n{proc.stdout[-2000:]}"
    assert "failed" in proc.stdout or "error" in proc.stdout.lower()
