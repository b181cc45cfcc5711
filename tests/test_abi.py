"""The C ABI library loads, exports every function include/*.h declares, and rejects bad host-visible arguments before touching a GPU.
CPU only: nothing here launches a kernel."""
import ctypes
import glob
import os
import re
import subprocess

import pytest

from paper_2607_17652_amd import binding as fb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = sorted(glob.glob(os.path.join(ROOT, "include", "*.h")))


def declared_functions():
    names = set()
    for h in HEADERS:
        src = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"^[A-Za-z_][\w\s\*]*?\b(fb_\w+)\s*\(", src, re.M))
    return sorted(names)


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(fb.LIB_PATH):
        from paper_2607_17652_amd import build
        build.build()
    return fb.lib()


def test_header_declares_the_bound_functions():
    assert declared_functions() == sorted(fb.EXPORTS)


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", fb.LIB_PATH],
                         capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r"\b(fb_\w+)\b", out))
    assert set(declared_functions()) <= exported
    # no other unmangled (C-linkage) function leaks out of the library: the
    # internal helpers of the C-ABI file are static
    plain = {ln.split()[-1] for ln in out.splitlines()
             if len(ln.split()) == 3 and ln.split()[1] in "TW" and not ln.split()[-1].startswith("_")}
    assert plain == set(declared_functions()), sorted(plain ^ set(declared_functions()))


def test_version_and_sizes(lib):
    assert fb.fb_version().startswith("flowblock")
    assert fb.fb_pack_bytes(0, 1, 1) == 0
    off = fb.fb_pack_get_offsets(3, 2, 4)
    assert off["header"] == 0 and off["tiles"] == 64
    assert off["req_w"] == 64 + 6 * 8 * 4
    assert off["row_tok"] + 3 * 2 * 4 * 4 == off["total"] == fb.fb_pack_bytes(3, 2, 4)


def test_struct_sizes_match_header():
    assert ctypes.sizeof(fb.fb_pack) == 32
    assert ctypes.sizeof(fb.fb_attn_shape) == 48
    assert ctypes.sizeof(fb.fb_update_params) == 56
    assert fb.REQ_STATE_DTYPE.itemsize == 32
    assert fb.REQ_STATS_DTYPE.itemsize == 40
    assert ctypes.sizeof(fb.fb_synth_model) == 24


def test_ctypes_layouts_match_the_c_compiler(tmp_path):
    """Every struct the binding mirrors has the size and field offsets the C
    compiler gives the header's declaration."""
    structs = [fb.fb_pack, fb.fb_pack_offsets, fb.fb_attn_shape,
               fb.fb_update_params, fb.fb_synth_model, fb.fb_loop_args]
    lines = ["#include <stdio.h>", "#include <stddef.h>",
             '#include "flowblock_loop.h"', "int main(void) {"]
    for S in structs:
        n = S.__name__
        lines.append(f'printf("{n} %zu\\n", sizeof({n}));')
        for f, _ in S._fields_:
            lines.append(f'printf("{n}.{f} %zu\\n", offsetof({n}, {f}));')
    lines += ["return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", "-I", os.path.join(ROOT, "include"), str(src),
                    "-o", str(exe)], check=True)
    got = dict(l.rsplit(" ", 1) for l in
               subprocess.run([str(exe)], capture_output=True, text=True,
                              check=True).stdout.split("\n") if l)
    for S in structs:
        n = S.__name__
        assert int(got[n]) == ctypes.sizeof(S), n
        for f, _ in S._fields_:
            assert int(got[f"{n}.{f}"]) == getattr(S, f).offset, (n, f)


def _init(lib, buf, nbytes, B, W, bl, layout):
    h = fb.fb_pack()
    rc = lib.fb_pack_init(ctypes.byref(h), buf, nbytes, B, W, bl, layout)
    return rc, h


def test_pack_init_validation(lib):
    fake = ctypes.c_void_p(0x10000)     # never dereferenced by fb_pack_init
    need = fb.fb_pack_bytes(4, 2, 8)
    assert _init(lib, fake, need, 4, 2, 8, fb.FB_RAGGED)[0] == fb.FB_OK
    assert _init(lib, None, need, 4, 2, 8, fb.FB_RAGGED)[0] == fb.FB_E_INVAL
    assert _init(lib, fake, need - 1, 4, 2, 8, fb.FB_RAGGED)[0] == fb.FB_E_WORKSPACE
    assert _init(lib, fake, need, 0, 2, 8, fb.FB_RAGGED)[0] == fb.FB_E_INVAL
    assert _init(lib, fake, need, 4, 2, 8, 7)[0] == fb.FB_E_INVAL
    assert _init(lib, ctypes.c_void_p(0x10004), need, 4, 2, 8, 0)[0] == fb.FB_E_INVAL
    assert _init(lib, fake, 10**12, 4, 65, 8, 0)[0] == fb.FB_E_UNSUPPORTED
    assert "W_max" in fb.fb_last_error()


def test_calls_reject_bad_arguments_before_launch(lib):
    fake = ctypes.c_void_p(0x10000)
    rc, h = _init(lib, fake, fb.fb_pack_bytes(2, 2, 32), 2, 2, 32, fb.FB_RAGGED)
    assert rc == fb.FB_OK
    sh = fb.make_shape(8, 3, 128, fb.FB_BF16, 32, 4, 8)         # 8 % 3 != 0
    rc = lib.fb_wavefront_attention(fake, fake, fake, fake, ctypes.byref(h),
                                    ctypes.byref(sh), fake, fake, 1 << 30, None)
    assert rc == fb.FB_E_INVAL
    rc = lib.fb_wavefront_attention_planned(fake, fake, fake, fake, ctypes.byref(h),
                                            ctypes.byref(sh), fake, fake, 1 << 30, None)
    assert rc == fb.FB_E_INVAL
    assert lib.fb_attention_plan(ctypes.byref(h), ctypes.byref(sh), fake, 1 << 30,
                                 None) == fb.FB_E_INVAL
    # the split calls check the workspace like the one-call form
    sh = fb.make_shape(8, 4, 128, fb.FB_BF16, 32, 4, 8)
    need = lib.fb_attention_workspace_bytes(ctypes.byref(h), ctypes.byref(sh))
    assert need > 0
    assert lib.fb_attention_plan(ctypes.byref(h), ctypes.byref(sh), fake, need - 1,
                                 None) == fb.FB_E_WORKSPACE
    assert lib.fb_wavefront_attention_planned(fake, fake, fake, fake, ctypes.byref(h),
                                              ctypes.byref(sh), fake, fake, need - 1,
                                              None) == fb.FB_E_WORKSPACE
    assert lib.fb_wavefront_attention_planned(None, fake, fake, fake, ctypes.byref(h),
                                              ctypes.byref(sh), fake, fake, need,
                                              None) == fb.FB_E_INVAL
    sh = fb.make_shape(8, 4, 96, fb.FB_BF16, 32, 4, 8)          # head_dim 96
    rc = lib.fb_write_window_kv(fake, fake, fake, fake, fake, ctypes.byref(h),
                                ctypes.byref(sh), None)
    assert rc == fb.FB_E_UNSUPPORTED
    sh = fb.make_shape(8, 4, 128, fb.FB_BF16, 24, 4, 8)         # page 24
    rc = lib.fb_write_window_kv(fake, fake, fake, fake, fake, ctypes.byref(h),
                                ctypes.byref(sh), None)
    assert rc == fb.FB_E_INVAL
    sh = fb.make_shape(8, 4, 128, fb.FB_BF16, 4, 4, 8)          # bf16 page 4
    rc = lib.fb_write_window_kv(fake, fake, fake, fake, fake, ctypes.byref(h),
                                ctypes.byref(sh), None)
    assert rc == fb.FB_E_UNSUPPORTED
    sh = fb.make_shape(8, 4, 128, fb.FB_BF16, 32, 4, 8, kv_split=100)
    rc = lib.fb_write_window_kv(fake, fake, fake, fake, fake, ctypes.byref(h),
                                ctypes.byref(sh), None)
    assert rc == fb.FB_E_INVAL
    rc = lib.fb_write_window_kv(None, fake, fake, fake, fake, ctypes.byref(h),
                                ctypes.byref(fb.make_shape(8, 4, 128, fb.FB_BF16, 32,
                                                           4, 8)), None)
    assert rc == fb.FB_E_INVAL
    prm = fb.make_params(0.9, 0.8, 0.5, 99, -1, 2, 3)            # W > W_max
    rc = lib.fb_denoise_update(fake, 100, fb.FB_BF16, fake, 64, fake, fake, fake,
                               fake, fake, 4, ctypes.byref(h), ctypes.byref(prm),
                               None, fake, 1 << 30, None)
    assert rc == fb.FB_E_INVAL
    prm = fb.make_params(0.9, 0.8, 0.5, 100, -1, 2, 2)           # mask_id == V
    rc = lib.fb_denoise_update(fake, 100, fb.FB_BF16, fake, 64, fake, fake, fake,
                               fake, fake, 4, ctypes.byref(h), ctypes.byref(prm),
                               None, fake, 1 << 30, None)
    assert rc == fb.FB_E_INVAL
    for S_pe in (-1, 256):                                     # pe is a uint8 count
        prm = fb.make_params(0.9, 0.8, 0.5, 99, -1, S_pe, 2)
        rc = lib.fb_denoise_update(fake, 100, fb.FB_BF16, fake, 64, fake, fake, fake,
                                   fake, fake, 4, ctypes.byref(h), ctypes.byref(prm),
                                   None, fake, 1 << 30, None)
        assert rc == fb.FB_E_INVAL, S_pe
        assert "S_pe" in fb.fb_last_error()
        rc = lib.fb_denoise_apply(100, fake, 64, fake, fake, fake, fake, fake, 4,
                                  ctypes.byref(h), ctypes.byref(prm), None, fake,
                                  1 << 30, None)
        assert rc == fb.FB_E_INVAL, S_pe
    prm = fb.make_params(0.9, 0.8, 0.5, 99, -1, 2, 2)
    prm.flags = 0x80
    rc = lib.fb_denoise_update(fake, 100, fb.FB_BF16, fake, 64, fake, fake, fake,
                               fake, fake, 4, ctypes.byref(h), ctypes.byref(prm),
                               None, fake, 1 << 30, None)
    assert rc == fb.FB_E_INVAL
    rc = lib.fb_pack_wavefronts(None, None, 4, 64, ctypes.byref(h), None)
    assert rc == fb.FB_E_INVAL
    bad = fb.fb_pack()
    rc = lib.fb_pack_wavefronts(fake, None, 4, 64, ctypes.byref(bad), None)
    assert rc == fb.FB_E_INVAL


def test_loop_and_lmhead_calls_reject_bad_arguments_before_launch(lib):
    fake = ctypes.c_void_p(0x10000)
    odd = ctypes.c_void_p(0x10004)
    rc, h = _init(lib, fake, fb.fb_pack_bytes(2, 2, 32), 2, 2, 32, fb.FB_RAGGED)
    assert rc == fb.FB_OK
    P = ctypes.byref(h)
    # LM head: D a multiple of 64, sizes, pointers, alignment, workspaces
    assert lib.fb_lmhead_workspace_bytes(P, 1000, 100) == 0
    assert lib.fb_lmhead_workspace_bytes(P, 1000, 128) > 0
    big = 1 << 30
    assert lib.fb_lmhead_reduce(fake, fake, 100, 1000, P, fake, big, fake, big,
                                None) == fb.FB_E_UNSUPPORTED
    assert lib.fb_lmhead_reduce(fake, fake, 1 << 14, 1 << 17, P, fake, big, fake, big,
                                None) == fb.FB_E_UNSUPPORTED
    assert lib.fb_lmhead_reduce(None, fake, 128, 1000, P, fake, big, fake, big,
                                None) == fb.FB_E_INVAL
    assert lib.fb_lmhead_reduce(odd, fake, 128, 1000, P, fake, big, fake, big,
                                None) == fb.FB_E_INVAL
    assert lib.fb_lmhead_reduce(fake, fake, 128, 1000, P, fake, 16, fake, big,
                                None) == fb.FB_E_WORKSPACE
    assert lib.fb_lmhead_reduce(fake, fake, 128, 1000, P, fake, big, fake, 16,
                                None) == fb.FB_E_WORKSPACE
    # synthetic model: levels positive, finite and exact in the logits dtype
    st = fake
    m = fb.make_model(1, (6.0, 8.625, 10.0, 11.5))
    assert lib.fb_synth_logits(st, fake, 64, P, ctypes.byref(m), 1000, fb.FB_BF16,
                               odd, fake, None) == fb.FB_E_INVAL          # pred alignment
    assert lib.fb_synth_logits(st, fake, 64, P, ctypes.byref(m), 1, fb.FB_BF16,
                               fake, fake, None) == fb.FB_E_INVAL         # V < 2
    m2 = fb.make_model(1, (6.0, 8.6, 10.0, 11.5))                       # 8.6 not bf16
    assert lib.fb_synth_logits(st, fake, 64, P, ctypes.byref(m2), 1000, fb.FB_BF16,
                               fake, fake, None) == fb.FB_E_INVAL
    assert "bf16" in fb.fb_last_error()
    m3 = fb.make_model(1, (0.0, 8.625, 10.0, 11.5))
    assert lib.fb_synth_logits(st, fake, 64, P, ctypes.byref(m3), 1000, fb.FB_F32,
                               fake, fake, None) == fb.FB_E_INVAL
    sh = fb.make_shape(8, 4, 96, fb.FB_BF16, 32, 4, 8)
    assert lib.fb_synth_embed(P, ctypes.byref(sh), 1, fake, fake, fake,
                              None) == fb.FB_E_UNSUPPORTED
    # decode loop
    prm = fb.make_params(0.9, 0.8, 0.5, 999, -1, 2, 2)
    a = fb.fb_loop_args()
    a.st = a.tokens = a.pe = a.fin = a.logits = a.pred = a.conf = a.argmax = 0x10000
    a.T_max, a.n_max, a.V, a.logit_dtype = 64, 4, 1000, fb.FB_BF16
    a.pack = ctypes.pointer(h)
    a.prm = ctypes.pointer(prm)
    a.model = ctypes.pointer(m)
    a.upd_ws, a.upd_ws_bytes = 0x10000, big
    a.counters = a.forwards = 0x10000
    steps, done = ctypes.c_int(-1), ctypes.c_int(-1)
    call = lambda *x: lib.fb_decode_loop(ctypes.byref(a), *x, ctypes.byref(steps),
                                         ctypes.byref(done), None)
    assert call(10, 0, 0) == fb.FB_E_INVAL                      # check_every 0
    assert call(10, 4, 1) == fb.FB_E_INVAL                      # graph on the null stream
    prm.mask_id = 5
    assert call(10, 4, 0) == fb.FB_E_INVAL                      # mask_id != V - 1
    prm.mask_id = 999
    a.counters = 0
    assert call(10, 4, 0) == fb.FB_E_INVAL
    a.counters = 0x10000
    a.upd_ws_bytes = 16
    assert call(10, 4, 0) == fb.FB_E_WORKSPACE
    assert steps.value == -1 and done.value == -1               # nothing ran


def test_probes_reject_bad_arguments_before_launch(lib):
    fake = ctypes.c_void_p(0x10000)
    other = ctypes.c_void_p(0x90000)
    assert lib.fb_hbm_read_probe(None, 64, fake, None) == fb.FB_E_INVAL
    assert lib.fb_hbm_read_probe(fake, 0, fake, None) == fb.FB_E_INVAL
    assert lib.fb_hbm_read_probe(fake, 40, fake, None) == fb.FB_E_INVAL
    assert lib.fb_hbm_read_probe(ctypes.c_void_p(0x10008), 64, fake, None) == fb.FB_E_INVAL
    assert lib.fb_hbm_copy_probe(fake, ctypes.c_void_p(0x10010), 64, None) == fb.FB_E_INVAL
    assert "overlap" in fb.fb_last_error()
    assert lib.fb_hbm_copy_probe(fake, other, 24, None) == fb.FB_E_INVAL


def test_noalloc_update_rejects_a_pack_above_its_array(lib):
    """fb_denoise_update_noalloc: a pack whose update workspace exceeds the
    library's array is refused before anything is enqueued."""
    fake = ctypes.c_void_p(0x10000)
    B, W, bl = 8192, 4, 32                       # 2^20 rows of 16-byte partials
    rc, h = _init(lib, fake, fb.fb_pack_bytes(B, W, bl), B, W, bl, fb.FB_RAGGED)
    assert rc == fb.FB_OK
    assert lib.fb_update_workspace_bytes(ctypes.byref(h), 157184) > fb.FB_NOALLOC_SCRATCH_BYTES
    prm = fb.make_params(0.9, 0.8, 0.5, 157183, -1, 2, 4)
    rc = lib.fb_denoise_update_noalloc(fake, 157184, fb.FB_BF16, fake, 4096, fake, fake,
                                       fake, fake, fake, 64, ctypes.byref(h),
                                       ctypes.byref(prm), None, None)
    assert rc == fb.FB_E_UNSUPPORTED
    assert "noalloc" in fb.fb_last_error()
    prm.S_pe = 300                               # argument errors come first
    rc = lib.fb_denoise_update_noalloc(fake, 157184, fb.FB_BF16, fake, 4096, fake, fake,
                                       fake, fake, fake, 64, ctypes.byref(h),
                                       ctypes.byref(prm), None, None)
    assert rc == fb.FB_E_INVAL
