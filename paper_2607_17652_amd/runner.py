"""Device buffers and call order of one packed wavefront step, and of a whole
decode on the synthetic model.

``WavefrontStep`` owns the torch allocations a step needs (pack buffer,
workspaces, outputs) and calls the four C entry points in the order of
Alg. 1 on one stream: pack (Eq. 4), window KV write (Eq. 6), attention
(Sec. 4.1), denoise update (Eq. 1-3).  No arithmetic of the method happens
here.
"""
import ctypes

import numpy as np
import torch

from . import binding as fb
from . import synth


class WavefrontStep:
    def __init__(self, wl, host, tensors, device="cuda", kv_split=0):
        self.wl = wl
        self.host = host
        self.t = tensors
        dev = synth.host_to_device_state(host, device)
        self.st = dev["req_state"]
        self.tokens = dev["tokens"]
        self.pe = dev["pe"]
        self.fin = dev["fin"]
        self.page_table = dev["page_table"]
        self.n_max = host["n_max"]
        self.T_max = host["T_max"]
        nbytes = fb.fb_pack_bytes(wl.B, wl.W_max, wl.bl)
        self.pack_buf = torch.zeros(nbytes, dtype=torch.uint8, device=device)
        self.pack = fb.fb_pack_init(self.pack_buf, wl.B, wl.W_max, wl.bl, wl.layout)
        self.shape = fb.make_shape(wl.Hq, wl.Hkv, wl.d, wl.dtype, wl.page_size,
                                   host["max_pages"], host["num_pages"],
                                   kv_split=kv_split)
        p = wl.params()
        self.params = fb.make_params(p["tau_mask"], p["tau_edit"], p["theta"],
                                     p["mask_id"], p["eos_id"], p["S_pe"], p["W"],
                                     p["edit_masked"], p["force_progress"])
        aw = fb.fb_attention_workspace_bytes(self.pack, self.shape)
        self.attn_ws = torch.empty(max(aw, 16), dtype=torch.uint8, device=device)
        uw = fb.fb_update_workspace_bytes(self.pack, wl.V)
        self.upd_ws = torch.empty(max(uw, 16), dtype=torch.uint8, device=device)
        self.out = torch.zeros_like(tensors["q"])
        self.conf = torch.zeros(wl.row_cap, dtype=torch.float32, device=device)
        self.argmax = torch.full((wl.row_cap,), -1, dtype=torch.int32, device=device)
        self.stats = torch.zeros(wl.B * fb.REQ_STATS_DTYPE.itemsize,
                                 dtype=torch.uint8, device=device)

    def set_params(self, **kw):
        for k, v in kw.items():
            setattr(self.params, k, v)

    def pack_step(self, stream=None):
        fb.fb_pack_wavefronts(self.st, self.tokens, self.n_max, self.T_max,
                              self.pack, stream)

    def kv_step(self, stream=None):
        t = self.t
        fb.fb_write_window_kv(t["k_new"], t["v_new"], t["k_cache"], t["v_cache"],
                              self.page_table, self.pack, self.shape, stream)

    def attention_step(self, stream=None):
        t = self.t
        fb.fb_wavefront_attention(t["q"], t["k_cache"], t["v_cache"],
                                  self.page_table, self.pack, self.shape,
                                  self.out, self.attn_ws, stream)

    def update_step(self, stream=None, st=None, tokens=None, pe=None, fin=None):
        fb.fb_denoise_update(self.t["logits"],
                             self.tokens if tokens is None else tokens,
                             self.conf, self.argmax,
                             self.st if st is None else st,
                             self.pe if pe is None else pe,
                             self.fin if fin is None else fin,
                             self.pack, self.params, self.stats, self.upd_ws,
                             stream)

    def run(self, stream=None):
        self.pack_step(stream)
        self.kv_step(stream)
        self.attention_step(stream)
        self.update_step(stream)


class DecodeLoop:
    """Device buffers of a whole decode (Alg. 1's outer loop) on the synthetic
    model, and the call of fb_decode_loop that runs it.  With ``attn`` =
    dict(Hq, Hkv, d, dtype, page_size, k_cache, v_cache, embed_seed) each step
    also writes the window K/V of synthetic embeddings and runs the attention.
    Marshalling only: every step runs in the library's kernels."""

    def __init__(self, host, bl, W_max, V, params, model_seed, levels,
                 layout="ragged", logit_dtype="bf16", attn=None, device="cuda"):
        B = len(host["state"]["L"])
        self.B = B
        dev = synth.host_to_device_state(host, device)
        self.st, self.tokens = dev["req_state"], dev["tokens"]
        self.pe, self.fin = dev["pe"], dev["fin"]
        self.page_table = dev["page_table"]
        self.T_max, self.n_max = host["T_max"], host["n_max"]
        self.pack_buf = torch.zeros(fb.fb_pack_bytes(B, W_max, bl), dtype=torch.uint8,
                                    device=device)
        self.pack = fb.fb_pack_init(self.pack_buf, B, W_max, bl, layout)
        self.params = fb.make_params(**params)
        self.model = fb.make_model(model_seed, levels)
        cap = self.pack.row_cap
        ldt = torch.bfloat16 if logit_dtype == "bf16" else torch.float32
        self.logits = torch.zeros((cap, V), dtype=ldt, device=device)
        self.pred = torch.zeros((cap, 2), dtype=torch.int32, device=device)
        self.conf = torch.zeros(cap, dtype=torch.float32, device=device)
        self.argmax = torch.full((cap,), -1, dtype=torch.int32, device=device)
        self.stats = torch.zeros(B * fb.REQ_STATS_DTYPE.itemsize, dtype=torch.uint8,
                                 device=device)
        uw = fb.fb_update_workspace_bytes(self.pack, V)
        self.upd_ws = torch.empty(max(uw, 16), dtype=torch.uint8, device=device)
        self.counters = torch.zeros(4, dtype=torch.int32, device=device)
        self.forwards = torch.zeros(B, dtype=torch.int32, device=device)
        a = fb.fb_loop_args()
        a.st, a.tokens, a.T_max, a.n_max = (self.st.data_ptr(), self.tokens.data_ptr(),
                                            self.T_max, self.n_max)
        a.pe, a.fin = self.pe.data_ptr(), self.fin.data_ptr()
        a.pack = ctypes.pointer(self.pack.handle)
        a.prm = ctypes.pointer(self.params)
        a.model = ctypes.pointer(self.model)
        a.logits, a.V, a.logit_dtype = (self.logits.data_ptr(), V,
                                        fb.FB_BF16 if logit_dtype == "bf16" else fb.FB_F32)
        a.pred, a.conf, a.argmax = (self.pred.data_ptr(), self.conf.data_ptr(),
                                    self.argmax.data_ptr())
        a.stats = self.stats.data_ptr()
        a.upd_ws, a.upd_ws_bytes = self.upd_ws.data_ptr(), self.upd_ws.numel()
        a.counters, a.forwards = self.counters.data_ptr(), self.forwards.data_ptr()
        self.attn = attn
        if attn is not None:
            self.shape = fb.make_shape(attn["Hq"], attn["Hkv"], attn["d"], attn["dtype"],
                                       attn["page_size"], host["max_pages"],
                                       host["num_pages"])
            adt = torch.bfloat16 if attn["dtype"] == "bf16" else torch.float32
            self.q = torch.zeros((cap, attn["Hq"], attn["d"]), dtype=adt, device=device)
            self.k_new = torch.zeros((cap, attn["Hkv"], attn["d"]), dtype=adt, device=device)
            self.v_new = torch.zeros_like(self.k_new)
            self.out = torch.zeros_like(self.q)
            self.k_cache, self.v_cache = attn["k_cache"], attn["v_cache"]
            aw = fb.fb_attention_workspace_bytes(self.pack, self.shape)
            self.attn_ws = torch.empty(max(aw, 16), dtype=torch.uint8, device=device)
            a.shape = ctypes.pointer(self.shape)
            a.q, a.k_new, a.v_new = (self.q.data_ptr(), self.k_new.data_ptr(),
                                     self.v_new.data_ptr())
            a.k_cache, a.v_cache = self.k_cache.data_ptr(), self.v_cache.data_ptr()
            a.page_table = self.page_table.data_ptr()
            a.attn_out = self.out.data_ptr()
            a.attn_ws, a.attn_ws_bytes = self.attn_ws.data_ptr(), self.attn_ws.numel()
            a.embed_seed = attn["embed_seed"]
        self.args = a

    def run(self, max_steps=100000, check_every=8, use_graph=False, stream=None):
        """Returns (steps enqueued, done)."""
        if stream is not None:
            torch.cuda.synchronize()       # buffers were filled on another stream
        return fb.fb_decode_loop(self.args, max_steps, check_every, use_graph, stream)

    def results(self):
        return dict(tokens=self.tokens.cpu().numpy().astype(np.int64),
                    st=synth.state_from_records(self.st.cpu().numpy()),
                    pe=self.pe.cpu().numpy().astype(np.int64),
                    fin=self.fin.cpu().numpy().astype(np.int64),
                    steps=int(self.counters[0].item()),
                    forwards=self.forwards.cpu().numpy().astype(np.int64))
