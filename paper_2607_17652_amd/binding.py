"""ctypes binding of libflowblock.so -- argument marshalling only.

Each function has the name of the C entry point it calls and takes torch
tensors where the C call takes device pointers; every step of the work runs
in the library's HIP kernels.  A non-zero status raises ``FlowBlockError``
with the library's message.  Loading fails loudly if the library is not built:
there is no fallback path.
"""
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libflowblock.so")

FB_OK = 0
FB_E_INVAL = -1
FB_E_UNSUPPORTED = -2
FB_E_WORKSPACE = -3
FB_E_HIP = -4

FB_DERR_NONE = 0
FB_DERR_STATE = 1
FB_DERR_PAGE = 2
FB_DERR_PLAN = 3

FB_F32 = 0
FB_BF16 = 1
FB_RAGGED = 0
FB_PADDED = 1
FB_EDIT_MASKED = 1
FB_FORCE_PROGRESS = 2
FB_SYNC_WINDOW = 4

LAYOUTS = {"ragged": FB_RAGGED, "padded": FB_PADDED}

# Every symbol include/*.h declares.
EXPORTS = [
    "fb_version", "fb_last_error", "fb_pack_bytes", "fb_pack_get_offsets",
    "fb_pack_init", "fb_pack_wavefronts", "fb_pack_read_status",
    "fb_write_window_kv", "fb_attention_workspace_bytes",
    "fb_wavefront_attention", "fb_attention_plan", "fb_wavefront_attention_planned",
    "fb_update_workspace_bytes", "fb_denoise_update",
    "fb_vocab_reduce", "fb_denoise_apply",
    "fb_synth_embed", "fb_synth_logits", "fb_decode_loop",
    "fb_lmhead_workspace_bytes", "fb_lmhead_reduce", "fb_window_prologue",
    "fb_hbm_read_probe", "fb_hbm_copy_probe", "fb_denoise_update_noalloc",
]
FB_NOALLOC_SCRATCH_BYTES = 4 << 20
FB_PROBE_BLOCKS = 2048


class FlowBlockError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"flowblock status {code}: {msg}")
        self.code = code


class fb_pack(ctypes.Structure):
    _fields_ = [("buf", ctypes.c_void_p), ("B", ctypes.c_int32),
                ("W_max", ctypes.c_int32), ("bl", ctypes.c_int32),
                ("layout", ctypes.c_int32), ("row_cap", ctypes.c_int32),
                ("tile_cap", ctypes.c_int32)]


class fb_pack_offsets(ctypes.Structure):
    _fields_ = [(n, ctypes.c_size_t) for n in
                ("header", "tiles", "req_w", "req_row0", "row_req", "row_pos",
                 "row_tok", "total")]


class fb_attn_shape(ctypes.Structure):
    _fields_ = [("Hq", ctypes.c_int32), ("Hkv", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("max_pages", ctypes.c_int32),
                ("num_pages", ctypes.c_int32), ("kv_split", ctypes.c_int32),
                ("sm_scale", ctypes.c_float), ("reserved", ctypes.c_int32 * 3)]


class fb_update_params(ctypes.Structure):
    _fields_ = [("tau_mask", ctypes.c_double), ("tau_edit", ctypes.c_double),
                ("theta_spawn", ctypes.c_double), ("mask_id", ctypes.c_int32),
                ("eos_id", ctypes.c_int32), ("S_pe", ctypes.c_int32),
                ("W", ctypes.c_int32), ("flags", ctypes.c_uint32),
                ("reserved", ctypes.c_int32 * 3)]


class fb_synth_model(ctypes.Structure):
    _fields_ = [("seed", ctypes.c_uint64), ("levels", ctypes.c_float * 4)]


class fb_loop_args(ctypes.Structure):
    vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    _fields_ = [
        ("st", vp), ("tokens", vp), ("T_max", i32), ("n_max", i32), ("pe", vp),
        ("fin", vp), ("pack", ctypes.POINTER(fb_pack)),
        ("prm", ctypes.POINTER(fb_update_params)),
        ("model", ctypes.POINTER(fb_synth_model)), ("logits", vp), ("V", i32),
        ("logit_dtype", i32), ("pred", vp), ("conf", vp), ("argmax", vp),
        ("stats", vp), ("upd_ws", vp), ("upd_ws_bytes", sz),
        ("shape", ctypes.POINTER(fb_attn_shape)), ("q", vp), ("k_new", vp),
        ("v_new", vp), ("k_cache", vp), ("v_cache", vp), ("page_table", vp),
        ("attn_out", vp), ("attn_ws", vp), ("attn_ws_bytes", sz),
        ("embed_seed", ctypes.c_uint64), ("counters", vp), ("forwards", vp)]


# numpy views of the device records
REQ_STATE_DTYPE = np.dtype([(n, "<i4") for n in
                            ("gen_start", "prompt_len", "n_blocks", "L", "R",
                             "active", "eos_hit", "reserved")])
REQ_STATS_DTYPE = np.dtype([("m2t", "<i4"), ("t2t", "<i4"), ("committed", "<i4"),
                            ("spawned", "<i4"), ("eos", "<i4"), ("done", "<i4"),
                            ("valid", "<i4"), ("reserved", "<i4"),
                            ("rho_frontier", "<f8")])
assert REQ_STATE_DTYPE.itemsize == 32 and REQ_STATS_DTYPE.itemsize == 40

_lib = None


def lib():
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is not built; run `python -m paper_2607_17652_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
        P = ctypes.POINTER
        sig = {
            "fb_version": (ctypes.c_char_p, []),
            "fb_last_error": (ctypes.c_char_p, []),
            "fb_pack_bytes": (sz, [i32, i32, i32]),
            "fb_pack_get_offsets": (i32, [i32, i32, i32, P(fb_pack_offsets)]),
            "fb_pack_init": (i32, [P(fb_pack), vp, sz, i32, i32, i32, i32]),
            "fb_pack_wavefronts": (i32, [vp, vp, i32, i32, P(fb_pack), vp]),
            "fb_pack_read_status": (i32, [P(fb_pack), P(i32), P(i32), P(i32),
                                          P(i32), vp]),
            "fb_write_window_kv": (i32, [vp, vp, vp, vp, vp, P(fb_pack),
                                         P(fb_attn_shape), vp]),
            "fb_attention_workspace_bytes": (sz, [P(fb_pack), P(fb_attn_shape)]),
            "fb_wavefront_attention": (i32, [vp, vp, vp, vp, P(fb_pack),
                                             P(fb_attn_shape), vp, vp, sz, vp]),
            "fb_attention_plan": (i32, [P(fb_pack), P(fb_attn_shape), vp, sz, vp]),
            "fb_wavefront_attention_planned": (i32, [vp, vp, vp, vp, P(fb_pack),
                                                     P(fb_attn_shape), vp, vp, sz, vp]),
            "fb_update_workspace_bytes": (sz, [P(fb_pack), i32]),
            "fb_denoise_update": (i32, [vp, i32, i32, vp, i32, vp, vp, vp, vp, vp,
                                        i32, P(fb_pack), P(fb_update_params), vp,
                                        vp, sz, vp]),
            "fb_vocab_reduce": (i32, [vp, i32, i32, P(fb_pack), vp, sz, vp]),
            "fb_denoise_apply": (i32, [i32, vp, i32, vp, vp, vp, vp, vp, i32,
                                       P(fb_pack), P(fb_update_params), vp, vp, sz,
                                       vp]),
            "fb_window_prologue": (i32, [vp, vp, vp, vp, vp, vp, vp, P(fb_pack),
                                         P(fb_attn_shape), ctypes.c_double, vp]),
            "fb_lmhead_workspace_bytes": (sz, [P(fb_pack), i32, i32]),
            "fb_lmhead_reduce": (i32, [vp, vp, i32, i32, P(fb_pack), vp, sz, vp, sz, vp]),
            "fb_synth_embed": (i32, [P(fb_pack), P(fb_attn_shape), ctypes.c_uint64,
                                     vp, vp, vp, vp]),
            "fb_synth_logits": (i32, [vp, vp, i32, P(fb_pack), P(fb_synth_model),
                                      i32, i32, vp, vp, vp]),
            "fb_decode_loop": (i32, [P(fb_loop_args), i32, i32, i32, P(i32), P(i32),
                                     vp]),
            "fb_hbm_read_probe": (i32, [vp, sz, vp, vp]),
            "fb_denoise_update_noalloc": (i32, [vp, i32, i32, vp, i32, vp, vp, vp, vp,
                                                vp, i32, P(fb_pack), P(fb_update_params),
                                                vp, vp]),
            "fb_hbm_copy_probe": (i32, [vp, vp, sz, vp]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _check(rc):
    if rc != FB_OK:
        raise FlowBlockError(rc, lib().fb_last_error().decode())


def _ptr(t):
    if t is None:
        return None
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _dtype_code(t):
    import torch
    if t.dtype == torch.bfloat16:
        return FB_BF16
    if t.dtype == torch.float32:
        return FB_F32
    raise FlowBlockError(FB_E_UNSUPPORTED, f"dtype {t.dtype}")


# ------------------------------------------------------------------ library
def fb_version():
    return lib().fb_version().decode()


def fb_last_error():
    return lib().fb_last_error().decode()


# ------------------------------------------------------------------ packing
def fb_pack_bytes(B, W_max, bl):
    return int(lib().fb_pack_bytes(B, W_max, bl))


def fb_pack_get_offsets(B, W_max, bl):
    off = fb_pack_offsets()
    _check(lib().fb_pack_get_offsets(B, W_max, bl, ctypes.byref(off)))
    return {n: int(getattr(off, n)) for n, _ in fb_pack_offsets._fields_}


class Pack:
    """A host fb_pack handle plus the device buffer it points into."""

    def __init__(self, handle, buf):
        self.handle = handle
        self.buf = buf

    @property
    def row_cap(self):
        return self.handle.row_cap

    @property
    def tile_cap(self):
        return self.handle.tile_cap

    def ref(self):
        return ctypes.byref(self.handle)

    def view(self):
        """int32 device views of the packed batch (header, tiles, row maps)."""
        h = self.handle
        off = fb_pack_get_offsets(h.B, h.W_max, h.bl)
        b32 = self.buf.view(dtype=__import__("torch").int32)

        def sl(a, n):
            return b32[off[a] // 4: off[a] // 4 + n]
        return dict(header=sl("header", 16),
                    tiles=sl("tiles", h.tile_cap * 8).view(h.tile_cap, 8),
                    req_w=sl("req_w", h.B), req_row0=sl("req_row0", h.B),
                    row_req=sl("row_req", h.row_cap),
                    row_pos=sl("row_pos", h.row_cap),
                    row_tok=sl("row_tok", h.row_cap))


def fb_pack_init(buf, B, W_max, bl, layout):
    """buf: a uint8 CUDA tensor of at least fb_pack_bytes(B, W_max, bl) bytes."""
    if isinstance(layout, str):
        layout = LAYOUTS[layout]
    h = fb_pack()
    _check(lib().fb_pack_init(ctypes.byref(h), _ptr(buf),
                              buf.numel() * buf.element_size(), B, W_max, bl,
                              layout))
    return Pack(h, buf)


def fb_pack_wavefronts(st, tokens, n_max, T_max, pack, stream=None):
    _check(lib().fb_pack_wavefronts(_ptr(st), _ptr(tokens), n_max, T_max,
                                    pack.ref(), _stream(stream)))


def fb_pack_read_status(pack, stream=None):
    code, req, rows, tiles = (ctypes.c_int(), ctypes.c_int(), ctypes.c_int(),
                              ctypes.c_int())
    _check(lib().fb_pack_read_status(pack.ref(), ctypes.byref(code),
                                     ctypes.byref(req), ctypes.byref(rows),
                                     ctypes.byref(tiles), _stream(stream)))
    return dict(code=code.value, request=req.value, n_rows=rows.value,
                n_tiles=tiles.value)


# ---------------------------------------------------------------- attention
def make_shape(Hq, Hkv, head_dim, dtype, page_size, max_pages, num_pages,
               kv_split=0, sm_scale=0.0):
    if not isinstance(dtype, int):
        dtype = FB_BF16 if str(dtype) in ("bf16", "torch.bfloat16") else FB_F32
    return fb_attn_shape(Hq, Hkv, head_dim, dtype, page_size, max_pages,
                         num_pages, kv_split, sm_scale)


def fb_write_window_kv(k_new, v_new, k_cache, v_cache, page_table, pack, shape,
                       stream=None):
    _check(lib().fb_write_window_kv(_ptr(k_new), _ptr(v_new), _ptr(k_cache),
                                    _ptr(v_cache), _ptr(page_table), pack.ref(),
                                    ctypes.byref(shape), _stream(stream)))


def fb_window_prologue(q_in, q_out, k_new, v_new, k_cache, v_cache, page_table, pack, shape,
                       rope_base=10000.0, stream=None):
    _check(lib().fb_window_prologue(_ptr(q_in), _ptr(q_out), _ptr(k_new), _ptr(v_new),
                                    _ptr(k_cache), _ptr(v_cache), _ptr(page_table), pack.ref(),
                                    ctypes.byref(shape), float(rope_base), _stream(stream)))


def fb_attention_workspace_bytes(pack, shape):
    return int(lib().fb_attention_workspace_bytes(pack.ref(), ctypes.byref(shape)))


def fb_wavefront_attention(q, k_cache, v_cache, page_table, pack, shape, out,
                           ws, stream=None):
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().fb_wavefront_attention(_ptr(q), _ptr(k_cache), _ptr(v_cache),
                                        _ptr(page_table), pack.ref(),
                                        ctypes.byref(shape), _ptr(out), _ptr(ws),
                                        nbytes, _stream(stream)))


def fb_attention_plan(pack, shape, ws, stream=None):
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().fb_attention_plan(pack.ref(), ctypes.byref(shape), _ptr(ws), nbytes,
                                   _stream(stream)))


def fb_wavefront_attention_planned(q, k_cache, v_cache, page_table, pack, shape, out,
                                   ws, stream=None):
    nbytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().fb_wavefront_attention_planned(_ptr(q), _ptr(k_cache), _ptr(v_cache),
                                                _ptr(page_table), pack.ref(),
                                                ctypes.byref(shape), _ptr(out), _ptr(ws),
                                                nbytes, _stream(stream)))


# ------------------------------------------------------------------- update
def make_params(tau_mask, tau_edit, theta, mask_id, eos_id, S_pe, W,
                edit_masked=False, force_progress=False, sync_window=False):
    flags = (FB_EDIT_MASKED if edit_masked else 0) | \
        (FB_FORCE_PROGRESS if force_progress else 0) | \
        (FB_SYNC_WINDOW if sync_window else 0)
    return fb_update_params(tau_mask, tau_edit, theta, mask_id, eos_id, S_pe, W,
                            flags)


def fb_update_workspace_bytes(pack, V):
    return int(lib().fb_update_workspace_bytes(pack.ref(), V))


def fb_denoise_update(logits, tokens, conf, argmax, st, pe, fin, pack, params,
                      stats, ws, stream=None):
    """logits [row_cap, V]; tokens int32 [B, T_max]; pe/fin uint8 [B, n_max];
    st: int32 [B, 8] (fb_req_state records); stats: uint8 [B*40] or None."""
    V = logits.shape[-1]
    T_max = tokens.shape[-1]
    n_max = pe.shape[-1]
    nbytes = ws.numel() * ws.element_size()
    _check(lib().fb_denoise_update(_ptr(logits), V, _dtype_code(logits),
                                   _ptr(tokens), T_max, _ptr(conf), _ptr(argmax),
                                   _ptr(st), _ptr(pe), _ptr(fin), n_max,
                                   pack.ref(), ctypes.byref(params), _ptr(stats),
                                   _ptr(ws), nbytes, _stream(stream)))


def fb_denoise_update_noalloc(logits, tokens, conf, argmax, st, pe, fin, pack, params,
                              stats, stream=None):
    """fb_denoise_update without a workspace argument: the library's own
    per-device array serves as the workspace (nothing is allocated)."""
    _check(lib().fb_denoise_update_noalloc(_ptr(logits), logits.shape[-1],
                                           _dtype_code(logits), _ptr(tokens),
                                           tokens.shape[-1], _ptr(conf), _ptr(argmax),
                                           _ptr(st), _ptr(pe), _ptr(fin), pe.shape[-1],
                                           pack.ref(), ctypes.byref(params), _ptr(stats),
                                           _stream(stream)))


def fb_vocab_reduce(logits, pack, ws, stream=None):
    nbytes = ws.numel() * ws.element_size()
    _check(lib().fb_vocab_reduce(_ptr(logits), logits.shape[-1], _dtype_code(logits),
                                 pack.ref(), _ptr(ws), nbytes, _stream(stream)))


def fb_denoise_apply(V, tokens, conf, argmax, st, pe, fin, pack, params, stats, ws,
                     stream=None):
    nbytes = ws.numel() * ws.element_size()
    _check(lib().fb_denoise_apply(V, _ptr(tokens), tokens.shape[-1], _ptr(conf),
                                  _ptr(argmax), _ptr(st), _ptr(pe), _ptr(fin),
                                  pe.shape[-1], pack.ref(), ctypes.byref(params),
                                  _ptr(stats), _ptr(ws), nbytes, _stream(stream)))


def fb_lmhead_workspace_bytes(pack, V, D):
    return int(lib().fb_lmhead_workspace_bytes(pack.ref(), V, D))


def fb_lmhead_reduce(hidden, weight, pack, lm_ws, upd_ws, stream=None):
    """hidden bf16 [row_cap, D]; weight bf16 [V, D]; the reduction lands in
    upd_ws for fb_denoise_apply."""
    D = hidden.shape[-1]
    V = weight.shape[0]
    _check(lib().fb_lmhead_reduce(_ptr(hidden), _ptr(weight), D, V, pack.ref(), _ptr(lm_ws),
                                  lm_ws.numel() * lm_ws.element_size(), _ptr(upd_ws),
                                  upd_ws.numel() * upd_ws.element_size(), _stream(stream)))


def stats_to_numpy(stats_tensor, B):
    raw = stats_tensor.cpu().numpy().view(np.uint8)[: B * REQ_STATS_DTYPE.itemsize]
    return raw.view(REQ_STATS_DTYPE)


# ------------------------------------------------------ multi-step loop
def make_model(seed, levels):
    m = fb_synth_model()
    m.seed = seed
    for i, a in enumerate(levels):
        m.levels[i] = a
    return m


def fb_synth_embed(pack, shape, seed, q, k_new, v_new, stream=None):
    _check(lib().fb_synth_embed(pack.ref(), ctypes.byref(shape), seed, _ptr(q),
                                _ptr(k_new), _ptr(v_new), _stream(stream)))


def fb_synth_logits(st, tokens, pack, model, pred, logits, stream=None):
    """st int32 [B, 8]; tokens int32 [B, T_max]; pred int32 [row_cap, 2];
    logits [row_cap, V] (bf16 or fp32)."""
    _check(lib().fb_synth_logits(_ptr(st), _ptr(tokens), tokens.shape[-1],
                                 pack.ref(), ctypes.byref(model), logits.shape[-1],
                                 _dtype_code(logits), _ptr(pred), _ptr(logits),
                                 _stream(stream)))


def fb_decode_loop(args, max_steps, check_every, use_graph, stream=None):
    """args: an fb_loop_args (its pointer fields must stay alive for the call).
    Returns (steps enqueued, done)."""
    steps, done = ctypes.c_int(), ctypes.c_int()
    _check(lib().fb_decode_loop(ctypes.byref(args), max_steps, check_every,
                                1 if use_graph else 0, ctypes.byref(steps),
                                ctypes.byref(done), _stream(stream)))
    return steps.value, bool(done.value)


# ------------------------------------------------------------- HBM probes
def fb_hbm_read_probe(src, out, stream=None):
    """Stream `src` (a contiguous device tensor) once; out: int32 or uint32
    tensor of FB_PROBE_BLOCKS words receiving per-workgroup XORs."""
    _check(lib().fb_hbm_read_probe(_ptr(src), src.numel() * src.element_size(),
                                   _ptr(out), _stream(stream)))


def fb_hbm_copy_probe(src, dst, stream=None):
    nbytes = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() < nbytes:
        raise FlowBlockError(FB_E_INVAL, "dst smaller than src")
    _check(lib().fb_hbm_copy_probe(_ptr(src), _ptr(dst), nbytes, _stream(stream)))
