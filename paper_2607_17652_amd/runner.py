"""Device buffers and call order of one packed wavefront step.

``WavefrontStep`` owns the torch allocations a step needs (pack buffer,
workspaces, outputs) and calls the four C entry points in the order of
Alg. 1 on one stream: pack (Eq. 4), window KV write (Eq. 6), attention
(Sec. 4.1), denoise update (Eq. 1-3).  No arithmetic of the method happens
here.
"""
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
