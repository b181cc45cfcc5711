// C ABI of libflowblock.so: argument validation, workspace sizing and launch.
// Every entry point validates what the host can see before enqueueing
// anything, returns an FB_* status and keeps a thread-local message for
// fb_last_error().  No exception crosses the ABI.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>

#include "internal.h"

namespace {

thread_local char g_err[512];

int fail(int code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return code;
}

int ok() {
    g_err[0] = 0;
    return FB_OK;
}

int hip_fail(hipError_t e, const char* what) {
    return fail(FB_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

bool is_pow2(int x) { return x > 0 && (x & (x - 1)) == 0; }

// Compute units of the current device, cached per device ordinal.
int cu_count() {
    static thread_local int cached_dev = -1;
    static thread_local int cached_cus = 0;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 256;
    if (dev != cached_dev) {
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
                hipSuccess || cus <= 0)
            cus = 256;
        cached_dev = dev;
        cached_cus = cus;
    }
    return cached_cus;
}

int check_pack(const fb_pack* p) {
    if (!p) return fail(FB_E_INVAL, "pack is NULL");
    if (!p->buf) return fail(FB_E_INVAL, "pack buffer is NULL (call fb_pack_init)");
    if (p->B < 1 || p->W_max < 1 || p->bl < 1)
        return fail(FB_E_INVAL, "pack capacities are not initialised");
    if (p->row_cap != p->B * p->W_max * p->bl || p->tile_cap != p->B * p->W_max)
        return fail(FB_E_INVAL, "pack capacities are inconsistent");
    return FB_OK;
}

int check_shape(const fb_pack* p, const fb_attn_shape* sh) {
    if (!sh) return fail(FB_E_INVAL, "shape is NULL");
    if (sh->Hq < 1 || sh->Hkv < 1 || sh->Hq % sh->Hkv)
        return fail(FB_E_INVAL, "need Hq >= 1, Hkv >= 1 and Hq %% Hkv == 0 (got %d, %d)",
                    sh->Hq, sh->Hkv);
    if (sh->head_dim != 32 && sh->head_dim != 64 && sh->head_dim != 128)
        return fail(FB_E_UNSUPPORTED, "head_dim %d not built (32, 64, 128)", sh->head_dim);
    if (sh->dtype != FB_BF16 && sh->dtype != FB_F32)
        return fail(FB_E_UNSUPPORTED, "dtype %d not supported", sh->dtype);
    if (!is_pow2(sh->page_size))
        return fail(FB_E_INVAL, "page_size %d is not a power of two", sh->page_size);
    if (sh->dtype == FB_BF16 && sh->page_size < 8)
        return fail(FB_E_UNSUPPORTED, "bf16 needs page_size >= 8 (got %d)", sh->page_size);
    if (sh->max_pages < 1 || sh->num_pages < 1)
        return fail(FB_E_INVAL, "max_pages and num_pages must be >= 1");
    if (sh->kv_split < 0 || sh->kv_split % 32)
        return fail(FB_E_INVAL, "kv_split %d must be 0 or a positive multiple of 32",
                    sh->kv_split);
    const size_t elt = sh->dtype == FB_BF16 ? 2 : 4;
    if ((size_t)p->bl * sh->head_dim * elt > 65536)
        return fail(FB_E_UNSUPPORTED, "bl*head_dim too large for the KV staging buffer");
    if (isnan(sh->sm_scale) || isinf(sh->sm_scale))
        return fail(FB_E_INVAL, "sm_scale is not finite");
    return FB_OK;
}

}  // namespace

extern "C" {

const char* fb_version(void) { return "flowblock 0.1.0 gfx950"; }

const char* fb_last_error(void) { return g_err; }

size_t fb_pack_bytes(int B, int W_max, int bl) {
    if (B < 1 || W_max < 1 || bl < 1) return 0;
    size_t o[8];
    fb::pack_offsets_ints(B, B * W_max, B * W_max * bl, o);
    return o[7] * sizeof(int32_t);
}

int fb_pack_get_offsets(int B, int W_max, int bl, fb_pack_offsets* off) {
    if (!off) return fail(FB_E_INVAL, "offsets is NULL");
    if (B < 1 || W_max < 1 || bl < 1) return fail(FB_E_INVAL, "B, W_max, bl must be >= 1");
    size_t o[8];
    fb::pack_offsets_ints(B, B * W_max, B * W_max * bl, o);
    off->header = o[0] * 4;
    off->tiles = o[1] * 4;
    off->req_w = o[2] * 4;
    off->req_row0 = o[3] * 4;
    off->row_req = o[4] * 4;
    off->row_pos = o[5] * 4;
    off->row_tok = o[6] * 4;
    off->total = o[7] * 4;
    return ok();
}

int fb_pack_init(fb_pack* pack, void* buf, size_t buf_bytes, int B, int W_max, int bl,
                 int layout) {
    if (!pack) return fail(FB_E_INVAL, "pack is NULL");
    if (!buf) return fail(FB_E_INVAL, "buf is NULL");
    if (B < 1 || W_max < 1 || bl < 1)
        return fail(FB_E_INVAL, "B, W_max, bl must be >= 1 (got %d, %d, %d)", B, W_max, bl);
    if ((long long)B * W_max * bl > (1LL << 30))
        return fail(FB_E_INVAL, "B*W_max*bl exceeds 2^30 rows");
    if (W_max > 64) return fail(FB_E_UNSUPPORTED, "W_max %d > 64", W_max);
    if (layout != FB_RAGGED && layout != FB_PADDED)
        return fail(FB_E_INVAL, "layout %d is neither FB_RAGGED nor FB_PADDED", layout);
    if (!aligned16(buf)) return fail(FB_E_INVAL, "pack buffer must be 16-byte aligned");
    const size_t need = fb_pack_bytes(B, W_max, bl);
    if (buf_bytes < need)
        return fail(FB_E_WORKSPACE, "pack buffer has %zu bytes, needs %zu", buf_bytes, need);
    pack->buf = buf;
    pack->B = B;
    pack->W_max = W_max;
    pack->bl = bl;
    pack->layout = layout;
    pack->row_cap = B * W_max * bl;
    pack->tile_cap = B * W_max;
    return ok();
}

int fb_pack_wavefronts(const fb_req_state* st, const int32_t* tokens, int n_max, int T_max,
                       fb_pack* pack, void* stream) {
    int rc = check_pack(pack);
    if (rc) return rc;
    if (!st) return fail(FB_E_INVAL, "state is NULL");
    if (n_max < 1 || T_max < 1) return fail(FB_E_INVAL, "n_max and T_max must be >= 1");
    hipError_t e = fb::launch_pack(st, tokens, n_max, T_max, pack, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "pack launch");
    return ok();
}

int fb_pack_read_status(const fb_pack* pack, int* code, int* request, int* n_rows,
                        int* n_tiles, void* stream) {
    int rc = check_pack(pack);
    if (rc) return rc;
    int32_t hdr[fb::kHdrInts];
    hipError_t e = hipMemcpyAsync(hdr, pack->buf, sizeof hdr, hipMemcpyDeviceToHost,
                                  (hipStream_t)stream);
    if (e == hipSuccess) e = hipStreamSynchronize((hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "reading the pack status");
    const int32_t key = hdr[fb::kHdrStatus];
    if (code) *code = key == FB_PACK_STATUS_NONE ? FB_DERR_NONE : (key & 15);
    if (request) *request = key == FB_PACK_STATUS_NONE ? -1 : (key >> 4);
    if (n_rows) *n_rows = hdr[fb::kHdrRows];
    if (n_tiles) *n_tiles = hdr[fb::kHdrTiles];
    return ok();
}

int fb_write_window_kv(const void* k_new, const void* v_new, void* k_cache, void* v_cache,
                       const int32_t* page_table, const fb_pack* pack,
                       const fb_attn_shape* sh, void* stream) {
    int rc = check_pack(pack);
    if (rc) return rc;
    rc = check_shape(pack, sh);
    if (rc) return rc;
    if (!k_new || !v_new || !k_cache || !v_cache || !page_table)
        return fail(FB_E_INVAL, "a tensor pointer is NULL");
    if (!aligned16(k_new) || !aligned16(v_new) || !aligned16(k_cache) || !aligned16(v_cache))
        return fail(FB_E_INVAL, "K/V pointers must be 16-byte aligned");
    hipError_t e = fb::launch_write_kv(k_new, v_new, k_cache, v_cache, page_table, pack, sh,
                                       (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "KV write launch");
    return ok();
}

int fb_window_prologue(const void* q_in, void* q_out, const void* k_new, const void* v_new,
                       void* k_cache, void* v_cache, const int32_t* page_table,
                       const fb_pack* pack, const fb_attn_shape* sh, double rope_base,
                       void* stream) {
    int rc = check_pack(pack);
    if (rc) return rc;
    rc = check_shape(pack, sh);
    if (rc) return rc;
    if (!q_in || !q_out || !k_new || !v_new || !k_cache || !v_cache || !page_table)
        return fail(FB_E_INVAL, "a tensor pointer is NULL");
    if (!aligned16(q_in) || !aligned16(q_out) || !aligned16(k_new) || !aligned16(v_new) ||
        !aligned16(k_cache) || !aligned16(v_cache))
        return fail(FB_E_INVAL, "q, K/V pointers must be 16-byte aligned");
    if (!(rope_base > 1.0) || isinf(rope_base))
        return fail(FB_E_INVAL, "rope_base must be finite and > 1");
    if ((size_t)pack->bl * sh->head_dim * 4 > 65536)
        return fail(FB_E_UNSUPPORTED, "bl*head_dim too large for the block's cos/sin table");
    hipError_t e = fb::launch_window_prologue(q_in, q_out, k_new, v_new, k_cache, v_cache,
                                              page_table, pack, sh, rope_base,
                                              (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "window prologue launch");
    return ok();
}

size_t fb_attention_workspace_bytes(const fb_pack* pack, const fb_attn_shape* sh) {
    if (check_pack(pack) || check_shape(pack, sh)) return 0;
    return fb::attention_sizes(pack, sh, cu_count()).total;
}

namespace {

static int check_attention_ws(const fb::AttnPlanSizes& z, const void* ws, size_t ws_bytes) {
    if (ws_bytes < z.total || (z.total > 0 && !ws))
        return fail(FB_E_WORKSPACE, "attention workspace has %zu bytes, needs %zu", ws_bytes,
                    z.total);
    if (ws && !aligned16(ws)) return fail(FB_E_INVAL, "workspace must be 16-byte aligned");
    return FB_OK;
}

static int wavefront_attention(const void* q, const void* k_cache, const void* v_cache,
                        const int32_t* page_table, const fb_pack* pack,
                        const fb_attn_shape* sh, void* out, void* ws, size_t ws_bytes,
                        void* stream, bool planned) {
    int rc = check_pack(pack);
    if (rc) return rc;
    rc = check_shape(pack, sh);
    if (rc) return rc;
    if (!q || !k_cache || !v_cache || !page_table || !out)
        return fail(FB_E_INVAL, "a tensor pointer is NULL");
    if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(out))
        return fail(FB_E_INVAL, "q, caches and out must be 16-byte aligned");
    const fb::AttnPlanSizes z = fb::attention_sizes(pack, sh, cu_count());
    rc = check_attention_ws(z, ws, ws_bytes);
    if (rc) return rc;
    hipError_t e = fb::launch_attention(q, k_cache, v_cache, page_table, pack, sh, out, ws, z,
                                        (hipStream_t)stream, planned);
    if (e != hipSuccess) return hip_fail(e, "attention launch");
    return ok();
}

}  // namespace

int fb_wavefront_attention(const void* q, const void* k_cache, const void* v_cache,
                           const int32_t* page_table, const fb_pack* pack,
                           const fb_attn_shape* sh, void* out, void* ws, size_t ws_bytes,
                           void* stream) {
    return wavefront_attention(q, k_cache, v_cache, page_table, pack, sh, out, ws, ws_bytes,
                               stream, false);
}

int fb_attention_plan(const fb_pack* pack, const fb_attn_shape* sh, void* ws, size_t ws_bytes,
                      void* stream) {
    int rc = check_pack(pack);
    if (rc) return rc;
    rc = check_shape(pack, sh);
    if (rc) return rc;
    const fb::AttnPlanSizes z = fb::attention_sizes(pack, sh, cu_count());
    rc = check_attention_ws(z, ws, ws_bytes);
    if (rc) return rc;
    hipError_t e = fb::launch_attention_plan(pack, sh, ws, z, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "attention plan launch");
    return ok();
}

int fb_wavefront_attention_planned(const void* q, const void* k_cache, const void* v_cache,
                                   const int32_t* page_table, const fb_pack* pack,
                                   const fb_attn_shape* sh, void* out, void* ws,
                                   size_t ws_bytes, void* stream) {
    return wavefront_attention(q, k_cache, v_cache, page_table, pack, sh, out, ws, ws_bytes,
                               stream, true);
}

size_t fb_update_workspace_bytes(const fb_pack* pack, int V) {
    if (check_pack(pack) || V < 1) return 0;
    return fb::update_sizes(pack, V, cu_count()).total;
}

namespace {

static int check_update_args(const fb_pack* pack, int V, const void* tokens, const void* conf,
                      const void* argmax, const void* st, const void* pe, const void* fin,
                      const fb_update_params* prm, int T_max, int n_max) {
    if (!tokens || !conf || !argmax || !st || !pe || !fin || !prm)
        return fail(FB_E_INVAL, "a required pointer is NULL");
    if (V < 1) return fail(FB_E_INVAL, "V must be >= 1");
    if (T_max < 1 || n_max < 1) return fail(FB_E_INVAL, "T_max and n_max must be >= 1");
    if (prm->W < 1 || prm->W > pack->W_max)
        return fail(FB_E_INVAL, "W %d outside [1, W_max=%d]", prm->W, pack->W_max);
    if (prm->S_pe < 0 || prm->S_pe > 255)
        return fail(FB_E_INVAL, "S_pe must be in [0, 255] (pe is a uint8 counter)");
    if (prm->mask_id < 0 || prm->mask_id >= V)
        return fail(FB_E_INVAL, "mask_id %d outside [0, V)", prm->mask_id);
    if (isnan(prm->tau_mask) || isnan(prm->tau_edit) || isnan(prm->theta_spawn))
        return fail(FB_E_INVAL, "a threshold is NaN");
    if (prm->flags & ~(FB_EDIT_MASKED | FB_FORCE_PROGRESS | FB_SYNC_WINDOW))
        return fail(FB_E_INVAL, "unknown flag bits 0x%x", prm->flags);
    return FB_OK;
}

static int check_reduce_args(const fb_pack* pack, const void* logits, int V, int dtype) {
    if (!logits) return fail(FB_E_INVAL, "logits is NULL");
    if (V < 1) return fail(FB_E_INVAL, "V must be >= 1");
    if (dtype != FB_BF16 && dtype != FB_F32)
        return fail(FB_E_UNSUPPORTED, "logit dtype %d not supported", dtype);
    if (!aligned16(logits)) return fail(FB_E_INVAL, "logits must be 16-byte aligned");
    (void)pack;
    return FB_OK;
}

static int check_ws(const void* ws, size_t ws_bytes, size_t need) {
    if (ws_bytes < need || !ws)
        return fail(FB_E_WORKSPACE, "update workspace has %zu bytes, needs %zu", ws_bytes,
                    need);
    if (!aligned16(ws)) return fail(FB_E_INVAL, "workspace must be 16-byte aligned");
    return FB_OK;
}

}  // namespace

int fb_vocab_reduce(const void* logits, int V, int dtype, const fb_pack* pack, void* ws,
                    size_t ws_bytes, void* stream) {
    int rc = check_pack(pack);
    if (rc) return rc;
    rc = check_reduce_args(pack, logits, V, dtype);
    if (rc) return rc;
    const fb::UpdateSizes z = fb::update_sizes(pack, V, cu_count());
    rc = check_ws(ws, ws_bytes, z.total);
    if (rc) return rc;
    hipError_t e = fb::launch_vocab_reduce(logits, V, dtype, pack, ws, z,
                                           (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "vocab reduction launch");
    return ok();
}

namespace {

static int check_lmhead(const fb_pack* pack, int V, int D) {
    int rc = check_pack(pack);
    if (rc) return rc;
    if (V < 1) return fail(FB_E_INVAL, "V must be >= 1");
    if (D < 64 || D % 64)
        return fail(FB_E_UNSUPPORTED, "hidden size %d must be a positive multiple of 64", D);
    if ((long long)V * D >= (1LL << 30) || (long long)pack->row_cap * D >= (1LL << 30))
        return fail(FB_E_UNSUPPORTED, "V*D and row_cap*D must be below 2^30");
    return FB_OK;
}

}  // namespace

size_t fb_lmhead_workspace_bytes(const fb_pack* pack, int V, int D) {
    if (check_lmhead(pack, V, D)) return 0;
    return fb::lm_sizes(pack, V, D, cu_count()).total;
}

int fb_lmhead_reduce(const void* hidden, const void* weight, int D, int V, const fb_pack* pack,
                     void* lm_ws, size_t lm_ws_bytes, void* upd_ws, size_t upd_ws_bytes,
                     void* stream) {
    int rc = check_lmhead(pack, V, D);
    if (rc) return rc;
    if (!hidden || !weight) return fail(FB_E_INVAL, "hidden or weight is NULL");
    if (!aligned16(hidden) || !aligned16(weight))
        return fail(FB_E_INVAL, "hidden and weight must be 16-byte aligned");
    const fb::LmSizes z = fb::lm_sizes(pack, V, D, cu_count());
    if (lm_ws_bytes < z.total || !lm_ws)
        return fail(FB_E_WORKSPACE, "LM-head workspace has %zu bytes, needs %zu", lm_ws_bytes,
                    z.total);
    if (!aligned16(lm_ws)) return fail(FB_E_INVAL, "LM-head workspace must be 16-byte aligned");
    const fb::UpdateSizes uz = fb::update_sizes(pack, V, cu_count());
    rc = check_ws(upd_ws, upd_ws_bytes, uz.total);
    if (rc) return rc;
    hipError_t e = fb::launch_lmhead(hidden, weight, D, V, pack, lm_ws, z, upd_ws, uz,
                                     (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "LM-head launch");
    return ok();
}

int fb_denoise_apply(int V, int32_t* tokens, int T_max, float* conf, int32_t* argmax,
                     fb_req_state* st, uint8_t* pe, uint8_t* fin, int n_max,
                     const fb_pack* pack, const fb_update_params* prm,
                     fb_req_stats* stats, const void* ws, size_t ws_bytes, void* stream) {
    int rc = check_pack(pack);
    if (rc) return rc;
    rc = check_update_args(pack, V, tokens, conf, argmax, st, pe, fin, prm, T_max, n_max);
    if (rc) return rc;
    const fb::UpdateSizes z = fb::update_sizes(pack, V, cu_count());
    rc = check_ws(ws, ws_bytes, z.total);
    if (rc) return rc;
    hipError_t e = fb::launch_apply(tokens, T_max, conf, argmax, st, pe, fin, n_max, pack,
                                    prm, stats, ws, z, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "update launch");
    return ok();
}

int fb_denoise_update(const void* logits, int V, int dtype, int32_t* tokens, int T_max,
                      float* conf, int32_t* argmax, fb_req_state* st, uint8_t* pe,
                      uint8_t* fin, int n_max, const fb_pack* pack,
                      const fb_update_params* prm, fb_req_stats* stats, void* ws,
                      size_t ws_bytes, void* stream) {
    int rc = check_pack(pack);
    if (rc) return rc;
    rc = check_reduce_args(pack, logits, V, dtype);
    if (rc) return rc;
    rc = check_update_args(pack, V, tokens, conf, argmax, st, pe, fin, prm, T_max, n_max);
    if (rc) return rc;
    const fb::UpdateSizes z = fb::update_sizes(pack, V, cu_count());
    rc = check_ws(ws, ws_bytes, z.total);
    if (rc) return rc;
    hipError_t e = fb::launch_vocab_reduce(logits, V, dtype, pack, ws, z,
                                           (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "vocab reduction launch");
    e = fb::launch_apply(tokens, T_max, conf, argmax, st, pe, fin, n_max, pack, prm, stats,
                         ws, z, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "update launch");
    return ok();
}

// ---- the update without a caller workspace -------------------------------
}  // extern "C"

// The update's workspace for callers that cannot allocate: one array per
// device, alive until the process ends.  Host code never passes this name to
// a kernel (on the host it is a stand-in, not a device address); it uses the
// address hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) unsigned char scratch[FB_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];   // per device ordinal, guarded by g_scratch_mu

// Device address of `scratch` on the current device, resolved once per
// device (with that device current) and kept.
int scratch_address(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices)
        return fail(FB_E_UNSUPPORTED, "device ordinal %d above %d", dev, kMaxDevices - 1);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, "resolving the update scratch array");
        if (!p) return fail(FB_E_HIP, "the update scratch array has no device address");
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return FB_OK;
}

}  // namespace

extern "C" {

int fb_denoise_update_noalloc(const void* logits, int V, int dtype, int32_t* tokens,
                              int T_max, float* conf, int32_t* argmax, fb_req_state* st,
                              uint8_t* pe, uint8_t* fin, int n_max, const fb_pack* pack,
                              const fb_update_params* prm, fb_req_stats* stats,
                              void* stream) {
    int rc = check_pack(pack);
    if (rc) return rc;
    rc = check_reduce_args(pack, logits, V, dtype);
    if (rc) return rc;
    rc = check_update_args(pack, V, tokens, conf, argmax, st, pe, fin, prm, T_max, n_max);
    if (rc) return rc;
    const fb::UpdateSizes z = fb::update_sizes(pack, V, cu_count());
    if (z.total > (size_t)FB_NOALLOC_SCRATCH_BYTES)
        return fail(FB_E_UNSUPPORTED,
                    "this pack and vocabulary need %zu bytes of update workspace, above "
                    "the %d bytes fb_denoise_update_noalloc holds; use fb_denoise_update",
                    z.total, FB_NOALLOC_SCRATCH_BYTES);
    void* ws = nullptr;
    rc = scratch_address(&ws);
    if (rc) return rc;
    hipError_t e = fb::launch_vocab_reduce(logits, V, dtype, pack, ws, z,
                                           (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "vocab reduction launch");
    e = fb::launch_apply(tokens, T_max, conf, argmax, st, pe, fin, n_max, pack, prm, stats,
                         ws, z, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "update launch");
    return ok();
}

// ---- multi-step loop on the synthetic model (flowblock_loop.h) -----------

namespace {

static bool exact_in(float a, int dtype) {
    if (dtype == FB_F32) return true;
    uint32_t u;
    memcpy(&u, &a, 4);
    return (u & 0xffffu) == 0;   // a bf16 value: the low half of the float is zero
}

static int check_model(const fb_synth_model* m, int V, int dtype) {
    if (!m) return fail(FB_E_INVAL, "model is NULL");
    if (V < 2) return fail(FB_E_INVAL, "the synthetic model needs V >= 2");
    if (dtype != FB_BF16 && dtype != FB_F32)
        return fail(FB_E_UNSUPPORTED, "logit dtype %d not supported", dtype);
    for (int l = 0; l < 4; ++l) {
        const float a = m->levels[l];
        if (!(a > 0.0f) || isinf(a))
            return fail(FB_E_INVAL, "level %d (%g) must be finite and > 0", l, (double)a);
        if (!exact_in(a, dtype))
            return fail(FB_E_INVAL, "level %d (%g) is not exact in bf16", l, (double)a);
    }
    return FB_OK;
}

static int check_embed_args(const fb_pack* pack, const fb_attn_shape* sh, const void* q,
                     const void* k_new, const void* v_new) {
    int rc = check_pack(pack);
    if (rc) return rc;
    rc = check_shape(pack, sh);
    if (rc) return rc;
    if (!q || !k_new || !v_new) return fail(FB_E_INVAL, "q, k_new or v_new is NULL");
    return FB_OK;
}

static int check_logit_args(const fb_req_state* st, const int32_t* tokens, int T_max,
                     const fb_pack* pack, const fb_synth_model* m, int V, int dtype,
                     const int32_t* pred, const void* logits) {
    int rc = check_pack(pack);
    if (rc) return rc;
    rc = check_model(m, V, dtype);
    if (rc) return rc;
    if (!st || !tokens || !pred || !logits) return fail(FB_E_INVAL, "a pointer is NULL");
    if (T_max < 1) return fail(FB_E_INVAL, "T_max must be >= 1");
    if (((uintptr_t)pred & 7u) != 0) return fail(FB_E_INVAL, "pred must be 8-byte aligned");
    if (!aligned16(logits)) return fail(FB_E_INVAL, "logits must be 16-byte aligned");
    return FB_OK;
}

// Enqueue one step of the loop (validated by the caller).
static hipError_t enqueue_step(const fb_loop_args* a, const fb::AttnPlanSizes* az,
                        const fb::UpdateSizes& uz, hipStream_t s) {
    hipError_t e = fb::launch_loop_count(a->st, a->pack->B, a->counters, a->forwards, 1, s);
    if (e != hipSuccess) return e;
    e = fb::launch_pack(a->st, a->tokens, a->n_max, a->T_max, a->pack, s);
    if (e != hipSuccess) return e;
    if (a->shape) {
        e = fb::launch_synth_embed(a->pack, a->shape, a->embed_seed, a->q, a->k_new, a->v_new,
                                   s);
        if (e != hipSuccess) return e;
        e = fb::launch_write_kv(a->k_new, a->v_new, a->k_cache, a->v_cache, a->page_table,
                                a->pack, a->shape, s);
        if (e != hipSuccess) return e;
        e = fb::launch_attention(a->q, a->k_cache, a->v_cache, a->page_table, a->pack,
                                 a->shape, a->attn_out, a->attn_ws, *az, s);
        if (e != hipSuccess) return e;
    }
    e = fb::launch_synth_logits(a->st, a->tokens, a->T_max, a->pack, a->model, a->V,
                                a->logit_dtype, a->pred, a->logits, s);
    if (e != hipSuccess) return e;
    e = fb::launch_vocab_reduce(a->logits, a->V, a->logit_dtype, a->pack, a->upd_ws, uz, s);
    if (e != hipSuccess) return e;
    return fb::launch_apply(a->tokens, a->T_max, a->conf, a->argmax, a->st, a->pe, a->fin,
                            a->n_max, a->pack, a->prm, a->stats, a->upd_ws, uz, s);
}

}  // namespace

int fb_synth_embed(const fb_pack* pack, const fb_attn_shape* sh, uint64_t seed, void* q,
                   void* k_new, void* v_new, void* stream) {
    int rc = check_embed_args(pack, sh, q, k_new, v_new);
    if (rc) return rc;
    hipError_t e = fb::launch_synth_embed(pack, sh, seed, q, k_new, v_new, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "synthetic embedding launch");
    return ok();
}

int fb_synth_logits(const fb_req_state* st, const int32_t* tokens, int T_max,
                    const fb_pack* pack, const fb_synth_model* model, int V, int dtype,
                    int32_t* pred, void* logits, void* stream) {
    int rc = check_logit_args(st, tokens, T_max, pack, model, V, dtype, pred, logits);
    if (rc) return rc;
    hipError_t e = fb::launch_synth_logits(st, tokens, T_max, pack, model, V, dtype, pred,
                                           logits, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "synthetic logits launch");
    return ok();
}

int fb_decode_loop(const fb_loop_args* a, int max_steps, int check_every, int use_graph,
                   int* steps_out, int* done_out, void* stream) {
    if (!a) return fail(FB_E_INVAL, "args is NULL");
    if (max_steps < 0 || check_every < 1)
        return fail(FB_E_INVAL, "need max_steps >= 0 and check_every >= 1");
    hipStream_t s = (hipStream_t)stream;
    if (use_graph && !s) return fail(FB_E_INVAL, "graph capture needs a non-null stream");
    int rc = check_logit_args(a->st, a->tokens, a->T_max, a->pack, a->model, a->V,
                              a->logit_dtype, a->pred, a->logits);
    if (rc) return rc;
    rc = check_update_args(a->pack, a->V, a->tokens, a->conf, a->argmax, a->st, a->pe, a->fin,
                           a->prm, a->T_max, a->n_max);
    if (rc) return rc;
    if (a->prm->mask_id != a->V - 1)
        return fail(FB_E_INVAL, "the synthetic model needs mask_id == V - 1");
    if (!a->counters || !a->forwards) return fail(FB_E_INVAL, "counters or forwards is NULL");
    const fb::UpdateSizes uz = fb::update_sizes(a->pack, a->V, cu_count());
    rc = check_ws(a->upd_ws, a->upd_ws_bytes, uz.total);
    if (rc) return rc;
    fb::AttnPlanSizes az{};
    if (a->shape) {
        rc = check_embed_args(a->pack, a->shape, a->q, a->k_new, a->v_new);
        if (rc) return rc;
        if (!a->k_cache || !a->v_cache || !a->page_table || !a->attn_out)
            return fail(FB_E_INVAL, "an attention pointer is NULL");
        if (!aligned16(a->q) || !aligned16(a->k_new) || !aligned16(a->v_new) ||
            !aligned16(a->k_cache) || !aligned16(a->v_cache) || !aligned16(a->attn_out))
            return fail(FB_E_INVAL, "attention tensors must be 16-byte aligned");
        az = fb::attention_sizes(a->pack, a->shape, cu_count());
        if (a->attn_ws_bytes < az.total || (az.total > 0 && !a->attn_ws))
            return fail(FB_E_WORKSPACE, "attention workspace has %zu bytes, needs %zu",
                        a->attn_ws_bytes, az.total);
        if (a->attn_ws && !aligned16(a->attn_ws))
            return fail(FB_E_INVAL, "attention workspace must be 16-byte aligned");
    }

    hipGraph_t graph = nullptr;
    hipGraphExec_t exec = nullptr;
    auto cleanup = [&]() {
        if (exec) (void)hipGraphExecDestroy(exec);
        if (graph) (void)hipGraphDestroy(graph);
    };
    int enq = 0, done = 0;
    hipError_t e = hipSuccess;
    for (;;) {
        if (enq >= max_steps) break;
        const int k = check_every < max_steps - enq ? check_every : max_steps - enq;
        if (use_graph && k == check_every) {
            if (!exec) {
                e = hipStreamBeginCapture(s, hipStreamCaptureModeThreadLocal);
                if (e != hipSuccess) return hip_fail(e, "begin capture");
                hipError_t ee = hipSuccess;
                for (int i = 0; i < k && ee == hipSuccess; ++i) ee = enqueue_step(a, &az, uz, s);
                e = hipStreamEndCapture(s, &graph);
                if (ee != hipSuccess) {
                    cleanup();
                    return hip_fail(ee, "step launch during capture");
                }
                if (e != hipSuccess) {
                    cleanup();
                    return hip_fail(e, "end capture");
                }
                e = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
                if (e != hipSuccess) {
                    exec = nullptr;
                    cleanup();
                    return hip_fail(e, "graph instantiate");
                }
            }
            e = hipGraphLaunch(exec, s);
            if (e != hipSuccess) {
                cleanup();
                return hip_fail(e, "graph launch");
            }
        } else {
            for (int i = 0; i < k; ++i) {
                e = enqueue_step(a, &az, uz, s);
                if (e != hipSuccess) {
                    cleanup();
                    return hip_fail(e, "step launch");
                }
            }
        }
        enq += k;
        e = fb::launch_loop_count(a->st, a->pack->B, a->counters, a->forwards, 0, s);
        int32_t flag = 1;
        if (e == hipSuccess)
            e = hipMemcpyAsync(&flag, &a->counters->any_active, sizeof flag,
                               hipMemcpyDeviceToHost, s);
        if (e == hipSuccess) e = hipStreamSynchronize(s);
        if (e != hipSuccess) {
            cleanup();
            return hip_fail(e, "reading the loop flag");
        }
        if (!flag) {
            done = 1;
            break;
        }
    }
    if (!done && enq == 0) {
        // no step asked for: report the current state
        int32_t flag = 1;
        e = fb::launch_loop_count(a->st, a->pack->B, a->counters, a->forwards, 0, s);
        if (e == hipSuccess)
            e = hipMemcpyAsync(&flag, &a->counters->any_active, sizeof flag,
                               hipMemcpyDeviceToHost, s);
        if (e == hipSuccess) e = hipStreamSynchronize(s);
        if (e != hipSuccess) {
            cleanup();
            return hip_fail(e, "reading the loop flag");
        }
        done = !flag;
    }
    cleanup();
    if (steps_out) *steps_out = enq;
    if (done_out) *done_out = done;
    return ok();
}

int fb_hbm_read_probe(const void* src, size_t bytes, uint32_t* out, void* stream) {
    if (!src || !out) return fail(FB_E_INVAL, "src and out must be device pointers");
    if (!aligned16(src) || ((uintptr_t)out & 3u))
        return fail(FB_E_INVAL, "src must be 16-byte and out 4-byte aligned");
    if (bytes == 0 || bytes % 16) return fail(FB_E_INVAL, "bytes must be a positive multiple of 16");
    hipError_t e = fb::launch_read_probe(src, bytes, out, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "read probe launch");
    return ok();
}

int fb_hbm_copy_probe(const void* src, void* dst, size_t bytes, void* stream) {
    if (!src || !dst) return fail(FB_E_INVAL, "src and dst must be device pointers");
    if (!aligned16(src) || !aligned16(dst)) return fail(FB_E_INVAL, "src and dst must be 16-byte aligned");
    if (bytes == 0 || bytes % 16) return fail(FB_E_INVAL, "bytes must be a positive multiple of 16");
    const char* a = static_cast<const char*>(src);
    const char* b = static_cast<const char*>(dst);
    if (a < b + bytes && b < a + bytes) return fail(FB_E_INVAL, "src and dst overlap");
    hipError_t e = fb::launch_copy_probe(src, dst, bytes, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "copy probe launch");
    return ok();
}

}  // extern "C"
