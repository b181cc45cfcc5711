/*
 * flowblock.h -- C ABI of libflowblock.so, the MI355X (gfx950) packed
 * wavefront denoising step of FlowBlock (Gated Wavefront Decoding with
 * Heterogeneous Wavefront Packing, arxiv 2607.17652).
 *
 * One step, enqueued on one HIP stream with no host synchronisation:
 *
 *   fb_pack_wavefronts      Eq. 4   per-request windows -> packed rows + tiles
 *   fb_write_window_kv      Eq. 6   fresh window K/V -> absolute paged slots
 *   fb_wavefront_attention  Sec. 4.1 / Eq. 5   block-causal window attention
 *   fb_denoise_update       Eq. 1-3, Sec. 3.1, Alg. 1   vocab reduction,
 *                           M2T/T2T update, in-order retire, gated admission
 *
 * Conventions shared by every call
 * --------------------------------
 * Memory   Every array argument is a device pointer to caller-owned memory
 *          (hipMalloc / torch) unless it is documented as host memory.  The
 *          library never allocates, frees or copies on these calls; scratch
 *          memory is passed in as a workspace whose size the matching
 *          *_workspace_bytes query returns.
 * Streams  `stream` is a hipStream_t (NULL = the null stream).  Calls only
 *          enqueue work; they never wait for the device.  Launch shapes depend
 *          only on capacities (B, W_max, bl, heads, V), never on device data,
 *          so a step can be captured into a HIP graph.
 * Status   Every call returns FB_OK (0) or a negative FB_E_* code.  Argument
 *          errors the host can see are reported before anything is launched;
 *          fb_last_error() then returns a message (thread-local).  Errors that
 *          depend on device data (an ill-formed request state, a page-table
 *          entry out of range) are recorded in the pack's device status word
 *          (fb_pack_read_status) and the offending request is skipped; no
 *          kernel traps.  No C++ exception crosses this ABI.
 * Threads  No global mutable state besides the thread-local error message;
 *          calls on different streams are independent.
 * Layouts  All arrays are dense row-major in the index order written below.
 *
 * Terms (the paper's notation)
 * ----------------------------
 *   b       request (sequence) index, 0 <= b < B
 *   bl      block length in tokens; block g of request b covers absolute
 *           positions gen_start_b + g*bl + [0, bl)
 *   [L, R)  request b's live window of blocks (Sec. 4.1); w_b = R - L <= W_max
 *   o_b     = gen_start_b + L_b*bl, the frozen-prefix length (start of B_L)
 *   kv_len  of window slot s: o_b + (s+1)*bl -- keys that slot's queries see
 *   packed row  one query token of a live block; a request's live rows are
 *           consecutive packed rows in position order
 */
#ifndef FLOWBLOCK_H
#define FLOWBLOCK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------ */
#define FB_OK             0
#define FB_E_INVAL       -1   /* bad argument (null pointer, size, range)     */
#define FB_E_UNSUPPORTED -2   /* valid but not built (head_dim, dtype, ...)   */
#define FB_E_WORKSPACE   -3   /* workspace smaller than the query returned    */
#define FB_E_HIP         -4   /* a HIP runtime call failed                    */

/* ---- device status codes (fb_pack_read_status) ------------------------- */
#define FB_DERR_NONE   0
#define FB_DERR_STATE  1  /* active request with !(0<=L<=R<=n<=n_max),
                             R-L > W_max, gen_start < 0 or
                             gen_start + n*bl > T_max                        */
#define FB_DERR_PAGE   2  /* a KV position past max_pages*page_size or a
                             page id outside [0, num_pages)                  */
#define FB_DERR_PLAN   3  /* fb_wavefront_attention_planned found a work
                             record the plan of this pack cannot hold (the
                             workspace had no plan); recorded for request 0,
                             the record skipped                              */

/* ---- element types and packing layouts --------------------------------- */
#define FB_F32   0
#define FB_BF16  1

#define FB_RAGGED 0   /* live blocks of all requests back to back           */
#define FB_PADDED 1   /* request b owns rows [b*W_max*bl, (b+1)*W_max*bl)    */

/* ---- fb_update_params.flags ------------------------------------------- */
#define FB_EDIT_MASKED    1u  /* literal Eq. 1: T2T may also overwrite [M]     */
#define FB_FORCE_PROGRESS 2u  /* a block with masks none of which was
                                 revealed this step (by Gamma, or by Delta
                                 under FB_EDIT_MASKED) unmasks its most
                                 confident masked row                          */
#define FB_SYNC_WINDOW    4u  /* the batch-synchronous wavefront that the
                                 Sec. 5 ablation compares HWP with: every
                                 active request shares one window [L, R);
                                 block L retires only when it is finished in
                                 all of them and admission (Eq. 3) gates on the
                                 smallest rho over them                        */

/* Per-request wavefront state (Sec. 4.2: "independent wavefront states
 * (L_b, R_b), finished flags, and in-order commit pointer").  Device array
 * of B records, read by fb_pack_wavefronts and updated in place by
 * fb_denoise_update.  32 bytes. */
typedef struct fb_req_state {
    int32_t gen_start;   /* absolute position of block 0                      */
    int32_t prompt_len;  /* positions < prompt_len are the prompt set P       */
    int32_t n_blocks;    /* n: number of blocks to generate                   */
    int32_t L;           /* leftmost live block (blocks < L are committed)    */
    int32_t R;           /* one past the rightmost admitted block             */
    int32_t active;      /* nonzero while the request is decoding             */
    int32_t eos_hit;     /* set when a committed block held eos_id            */
    int32_t reserved;
} fb_req_state;

/* Host-side handle of a packed batch.  `buf` is caller-owned device memory of
 * fb_pack_bytes(B, W_max, bl) bytes; fb_pack_init fills the capacities.  The
 * device contents are written by fb_pack_wavefronts and read by every other
 * call of the same step. */
typedef struct fb_pack {
    void*   buf;
    int32_t B, W_max, bl, layout;
    int32_t row_cap;     /* B*W_max*bl packed rows (both layouts)             */
    int32_t tile_cap;    /* B*W_max live-block tiles                          */
} fb_pack;

/* Byte offsets inside fb_pack.buf, for callers that read the packed batch.
 *   header   int32[16]: [0] live rows, [1] live tiles, [2] status word
 *            (FB_PACK_STATUS_NONE or request*16 + FB_DERR_* of the lowest
 *            offending request), [3..] reserved
 *   tiles    int32[tile_cap][8]: b, s (window slot), g (absolute block),
 *            row0 (first packed row), pos0 (its absolute position),
 *            o (= o_b), kv_len (= o_b + (s+1)*bl), w (= w_b)
 *   req_w    int32[B]: w_b, 0 if inactive, -1 if its state is ill-formed
 *   req_row0 int32[B]: first packed row of request b
 *   row_req  int32[row_cap]: request of each packed row, -1 if not live
 *   row_pos  int32[row_cap]: absolute position (the RoPE id of Eq. 4), or -1
 *   row_tok  int32[row_cap]: token x[b, pos] gathered per Eq. 4, or -1 */
typedef struct fb_pack_offsets {
    size_t header, tiles, req_w, req_row0, row_req, row_pos, row_tok, total;
} fb_pack_offsets;

#define FB_PACK_STATUS_NONE 0x7fffffff

/* Attention problem shape. */
typedef struct fb_attn_shape {
    int32_t Hq, Hkv;       /* query / KV heads; Hq % Hkv == 0; query head h
                              reads KV head h / (Hq/Hkv)                       */
    int32_t head_dim;      /* d: 32, 64 or 128                                 */
    int32_t dtype;         /* FB_BF16 or FB_F32 (q, caches, k_new/v_new, out)  */
    int32_t page_size;     /* power of two; FB_BF16 needs >= 8                 */
    int32_t max_pages;     /* columns of page_table                            */
    int32_t num_pages;     /* physical pages in each cache                     */
    int32_t kv_split;      /* keys per split-KV partition, a multiple of 32
                              (doubled on the device while the partitions
                              would overflow the workspace's item or partial
                              slots or exceed 64 per unit; a unit of at most
                              1.5 partitions stays whole); 0 chooses one
                              from the device's CU count                       */
    float   sm_scale;      /* <= 0 means 1/sqrt(head_dim)                      */
    int32_t reserved[3];
} fb_attn_shape;

/* Update parameters (Eq. 1-3; Sec. 3.1; Sec. 5.1 "model-default thresholds"). */
typedef struct fb_update_params {
    double   tau_mask;     /* M2T threshold, Eq. 1 (strict >) / Eq. 2 (>=)     */
    double   tau_edit;     /* T2T threshold, Eq. 1 (strict >)                  */
    double   theta_spawn;  /* admission gate, Eq. 3 (>=)                       */
    int32_t  mask_id;      /* the [M] token id                                 */
    int32_t  eos_id;       /* < 0 disables the EOS stop                        */
    int32_t  S_pe;         /* post-edit step cap (Sec. 3.1), 0..255 (pe is a
                              uint8 counter that saturates at 255)             */
    int32_t  W;            /* admission cap, 1 <= W <= W_max of the pack       */
    uint32_t flags;        /* FB_EDIT_MASKED | FB_FORCE_PROGRESS |
                              FB_SYNC_WINDOW                                   */
    int32_t  reserved[3];
} fb_update_params;

/* Per-request statistics of one fb_denoise_update call (device array [B]).
 * 40 bytes. */
typedef struct fb_req_stats {
    int32_t m2t;           /* masked positions written (|Gamma|, + forced)    */
    int32_t t2t;           /* revealed positions overwritten (|Delta|)        */
    int32_t committed;     /* blocks retired this step                        */
    int32_t spawned;       /* blocks admitted this step                       */
    int32_t eos;           /* 1 if a committed block held eos_id              */
    int32_t done;          /* 1 if the request became inactive this step      */
    int32_t valid;         /* 0 if the request was skipped (ill-formed state) */
    int32_t reserved;
    double  rho_frontier;  /* Eq. 2 readiness of the window's last live block
                              this step, -1 if it had no live block           */
} fb_req_stats;

/* ---- library ------------------------------------------------------------ */

/* Version string, e.g. "flowblock 0.1.0 gfx950". */
const char* fb_version(void);

/* Message for the last non-zero status returned on the calling thread, or "". */
const char* fb_last_error(void);

/* ---- Eq. 4: packing ------------------------------------------------------ */

/* Bytes of the device buffer of a packed batch with capacity (B, W_max, bl). */
size_t fb_pack_bytes(int B, int W_max, int bl);

/* Offsets of the fields of fb_pack.buf (see fb_pack_offsets above). */
int fb_pack_get_offsets(int B, int W_max, int bl, fb_pack_offsets* off);

/* Fill a host handle.  B >= 1, W_max >= 1, bl >= 1, layout FB_RAGGED or
 * FB_PADDED, buf non-null with buf_bytes >= fb_pack_bytes(B, W_max, bl).
 * Host only; touches no device memory. */
int fb_pack_init(fb_pack* pack, void* buf, size_t buf_bytes, int B, int W_max,
                 int bl, int layout);

/* Eq. 4 (Sec. 4.2, "From asynchronous states to dense tensors"): gather the
 * live window of every request into the packed batch.  Request b takes part
 * when active and well formed; its w_b live blocks (window slots
 * s = 0..w_b-1, absolute blocks L_b+s) become tiles whose rows hold positions
 * o_b + s*bl + [0, bl).  Ragged layout: request after request, no padding.
 * Padded layout: the paper's dense [B, q] batch, q = W_max*bl, with slots
 * s >= w_b left as non-live rows.  Also writes the token ids x[b, pos] of
 * every live row (row_tok) when `tokens` is non-null.
 *   st      device fb_req_state[B] (read only)
 *   tokens  device int32[B][T_max] or NULL
 *   n_max   columns of the per-block pe/fin arrays (n_blocks must be <= n_max)
 *   T_max   columns of `tokens` (gen_start + n_blocks*bl must be <= T_max)
 * Ill-formed active requests get req_w = -1 and FB_DERR_STATE. */
int fb_pack_wavefronts(const fb_req_state* st, const int32_t* tokens,
                       int n_max, int T_max, fb_pack* pack, void* stream);

/* Copy the pack's header to the host and wait for it (a synchronising call
 * meant for tests and monitoring, not for the step).  Any output may be NULL.
 *   code: FB_DERR_* of the lowest offending request (FB_DERR_NONE if none)
 *   request: that request, or -1;  n_rows / n_tiles: live rows and tiles. */
int fb_pack_read_status(const fb_pack* pack, int* code, int* request,
                        int* n_rows, int* n_tiles, void* stream);

/* ---- Eq. 6: window KV write-back ---------------------------------------- */

/* Eq. 6 (Sec. 4.2, "KV retrieval and write-back"): store the fresh K/V of
 * every live packed row at its absolute position in the paged caches:
 * position p of request b lives in page page_table[b][p / page_size], slot
 * p % page_size.  Only positions [o_b, o_b + w_b*bl) are written, so the
 * frozen prefix is never modified.
 *   k_new, v_new  [row_cap][Hkv][d] (dtype of sh)
 *   k_cache       [num_pages][Hkv][page_size][d]
 *   v_cache       [num_pages][Hkv][d][page_size]  (keys innermost)
 *   page_table    int32[B][max_pages]
 * A page id outside [0, num_pages) or a position past max_pages*page_size is
 * skipped and recorded as FB_DERR_PAGE. */
int fb_write_window_kv(const void* k_new, const void* v_new, void* k_cache,
                       void* v_cache, const int32_t* page_table,
                       const fb_pack* pack, const fb_attn_shape* sh,
                       void* stream);

/* Window prologue: rotary position embedding (RoPE, rotate-half
 * arrangement) at the rows' absolute positions -- the absolute RoPE position
 * ids of Sec. 4.2 (Fig. 2b) -- on the live rows' queries and fresh keys,
 * fused with the Eq. 6 write above: keys are rotated on their way into the
 * K cache, values written as fb_write_window_kv writes them.  Pair j of a
 * head vector, (x_j, x_{j+d/2}), turns by the angle p * rope_base^(-2j/d)
 * (angles in float64, products in float32, results rounded to the dtype).
 * Use it in place of fb_write_window_kv when the model hands over Q/K before
 * RoPE; the attention then reads q_out.
 *   q_in, q_out   [row_cap][Hq][d]; may be the same buffer (in place); rows
 *                 that are not live are not written
 *   k_new, v_new, caches, page_table  as for fb_write_window_kv
 *   rope_base     > 1 (10000 in the original RoPE)
 * Needs bl * d * 4 <= 65536 (the block's cos/sin table lives in LDS). */
int fb_window_prologue(const void* q_in, void* q_out, const void* k_new,
                       const void* v_new, void* k_cache, void* v_cache,
                       const int32_t* page_table, const fb_pack* pack,
                       const fb_attn_shape* sh, double rope_base, void* stream);

/* ---- Sec. 4.1 / Eq. 5: block-causal window attention ------------------- */

/* Workspace bytes for fb_wavefront_attention with this pack and shape. */
size_t fb_attention_workspace_bytes(const fb_pack* pack, const fb_attn_shape* sh);

/* W-shaped block-causal attention (Sec. 4.1; Eq. 5 per packed row): a query
 * of window slot s of request b, head h, attends to keys [0, o_b + (s+1)*bl)
 * of KV head h/(Hq/Hkv) -- the committed prefix plus live blocks 0..s, all of
 * its own block (bidirectional) and none to its right:
 *   out[row][h] = sum_j softmax_j(sm_scale * <q[row][h], K[j]>) V[j].
 * The mask is a per-block key count, never materialised.  Call after
 * fb_write_window_kv so the window's own keys are in the caches.
 *   q, out  [row_cap][Hq][d];  caches and page_table as above
 *   ws      device workspace of fb_attention_workspace_bytes bytes
 * Rows that are not live are not written.  Deterministic: no atomics on
 * outputs, so repeated calls give bit-identical results. */
int fb_wavefront_attention(const void* q, const void* k_cache,
                           const void* v_cache, const int32_t* page_table,
                           const fb_pack* pack, const fb_attn_shape* sh,
                           void* out, void* ws, size_t ws_bytes, void* stream);

/* fb_wavefront_attention in two calls, so that its scheduling can overlap the
 * window KV write (Sec. 4.1 / Eq. 5 as above).  fb_attention_plan writes the
 * attention's work list for this pack into ws: it reads only the pack (the
 * tiles of fb_pack_wavefronts), not q or the caches, so it may run on another
 * stream while fb_write_window_kv runs.  fb_wavefront_attention_planned then
 * runs the attention on that list, with the same arguments, results and
 * errors as fb_wavefront_attention.  The caller orders the two (planned after
 * plan, e.g. with an event) and keeps ws untouched between them; the pack
 * must not change in between.  For FB_F32 the plan is empty and the planned
 * call is the whole attention.
 *   ws  device workspace of fb_attention_workspace_bytes bytes (the same
 *       buffer in both calls)
 * Errors as fb_wavefront_attention (the plan checks the pack, shape and
 * workspace only). */
int fb_attention_plan(const fb_pack* pack, const fb_attn_shape* sh, void* ws,
                      size_t ws_bytes, void* stream);
int fb_wavefront_attention_planned(const void* q, const void* k_cache,
                                   const void* v_cache, const int32_t* page_table,
                                   const fb_pack* pack, const fb_attn_shape* sh,
                                   void* out, void* ws, size_t ws_bytes,
                                   void* stream);

/* ---- Eq. 1-3, Sec. 3.1, Alg. 1: denoise update -------------------------- */

/* Workspace bytes for fb_denoise_update with this pack and vocabulary. */
size_t fb_update_workspace_bytes(const fb_pack* pack, int V);

/* One denoising update of every live block, in the order of Alg. 1:
 *  1. per live row, over the vocabulary: x_hat = lowest index of max z,
 *     p = 1 / sum_v exp(z_v - max z) (Eq. 1 symbols), written to argmax[row]
 *     and conf[row] (float32);
 *  2. Eq. 1: Gamma = {[M] and p > tau_mask}, Delta = {revealed, x != x_hat,
 *     p > tau_edit, not prompt} (with FB_EDIT_MASKED also masked rows);
 *     x_{t+1} = x_hat on Gamma u Delta; a prediction equal to mask_id is never
 *     written.  Threshold compares use the float32 p widened to double;
 *  3. per live block g: rho = |{[M] and p >= tau_mask}| / |[M]| (Eq. 2, the
 *     masks before this update; 1 if none); post-edit counting and the
 *     locally-finished flag fin (Sec. 3.1; sticky);
 *  4. retire: while L < R and fin[L]: commit B_L, L++; a committed eos_id or
 *     L == n deactivates the request;
 *  5. admit (Eq. 3): if the window is empty admit one block; then while
 *     R - L < W, R < n and rho(B_{R-1}) >= theta_spawn: R++ (a block admitted
 *     in this step has rho = 0).
 *  With FB_SYNC_WINDOW, steps 4 and 5 act on the window all active requests
 *  share: retire while every one of them has finished B_L (a committed eos_id
 *  still stops only its own request), admit while the minimum of rho(B_{R-1})
 *  over them passes theta_spawn.  Active requests whose (L, R, n) differ are
 *  recorded as FB_DERR_STATE and no request retires or admits in that call.
 *   logits  [row_cap][V], dtype FB_BF16 or FB_F32; rows not live are not read;
 *           a live row holds no NaN or +inf and at least one finite value
 *           (-inf entries are allowed and weigh exp(-inf) = 0)
 *   tokens  int32[B][T_max], updated in place
 *   conf, argmax  [row_cap]; only live rows are written
 *   st      fb_req_state[B], updated in place
 *   pe, fin uint8[B][n_max] per-block post-edit count and finished flag
 *   stats   fb_req_stats[B] or NULL
 *   ws      device workspace of fb_update_workspace_bytes bytes
 * Requests the pack marked ill-formed are left untouched (stats.valid = 0). */
int fb_denoise_update(const void* logits, int V, int dtype, int32_t* tokens,
                      int T_max, float* conf, int32_t* argmax,
                      fb_req_state* st, uint8_t* pe, uint8_t* fin, int n_max,
                      const fb_pack* pack, const fb_update_params* prm,
                      fb_req_stats* stats, void* ws, size_t ws_bytes,
                      void* stream);

/* The two phases of fb_denoise_update, for callers that schedule or time
 * them separately.  fb_denoise_update(...) is exactly fb_vocab_reduce
 * followed by fb_denoise_apply on the same workspace.
 *
 * fb_vocab_reduce: step 1's streaming part (Eq. 1 symbols x_hat and p): for
 * every live packed row, partial (max, lowest argmax, sum of exponentials)
 * over vocabulary shares (a row's workgroups take its 32 KB pieces in turn),
 * written to `ws`.  Reads each live logit once. */
int fb_vocab_reduce(const void* logits, int V, int dtype, const fb_pack* pack,
                    void* ws, size_t ws_bytes, void* stream);

/* Workspace bytes of fb_lmhead_reduce (its own partials) for this pack,
 * vocabulary and hidden size; 0 if the arguments are invalid. */
size_t fb_lmhead_workspace_bytes(const fb_pack* pack, int V, int D);

/* The model's last layer and step 1's reduction in one pass: the logits of
 * the forward in Alg. 1, Z = hidden . weight^T, are reduced per live row to
 * x_hat and the partials of p exactly as fb_vocab_reduce would reduce them,
 * without Z ever being written to memory.  The result goes to the update
 * workspace `upd_ws` in the form fb_denoise_apply reads, so
 * fb_lmhead_reduce + fb_denoise_apply is fb_denoise_update on logits that
 * never exist.  The logits are accumulated in float32 (MFMA bf16 products),
 * so they may differ from an exact product by the accumulation error.
 *   hidden  bf16 [row_cap][D] (the packed rows' final hidden states)
 *   weight  bf16 [V][D] (one row per vocabulary id)
 *   D       a multiple of 64; V * D and row_cap * D below 2^30
 *   lm_ws   device workspace of fb_lmhead_workspace_bytes bytes
 *   upd_ws  the update workspace of fb_update_workspace_bytes(pack, V) bytes
 * Rows that are not live are not reduced. */
int fb_lmhead_reduce(const void* hidden, const void* weight, int D, int V,
                     const fb_pack* pack, void* lm_ws, size_t lm_ws_bytes, void* upd_ws,
                     size_t upd_ws_bytes, void* stream);

/* fb_denoise_apply: steps 1 (merge of the partials: x_hat, p) through 5 of
 * fb_denoise_update, from the workspace fb_vocab_reduce filled for the same
 * pack and V. */
int fb_denoise_apply(int V, int32_t* tokens, int T_max, float* conf,
                     int32_t* argmax, fb_req_state* st, uint8_t* pe, uint8_t* fin,
                     int n_max, const fb_pack* pack, const fb_update_params* prm,
                     fb_req_stats* stats, const void* ws, size_t ws_bytes,
                     void* stream);

/* ---- The update without a caller workspace ------------------------------ */

/* Bytes of the library's own update workspace, one per device. */
#define FB_NOALLOC_SCRATCH_BYTES (4 << 20)

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * fb_denoise_update with the same arguments, results and errors, minus the
 * workspace, which is a file-scope device array of FB_NOALLOC_SCRATCH_BYTES
 * that each GPU the library runs on holds until the process ends.  Nothing
 * is allocated or freed by the call (its address is looked up once per
 * device, on the first call with that device current).
 *   Limit: fb_update_workspace_bytes(pack, V) must not exceed
 *   FB_NOALLOC_SCRATCH_BYTES (row_cap up to about 250K rows); above it the
 *   call returns FB_E_UNSUPPORTED before enqueueing anything.
 *   Every call on one GPU uses that GPU's one array: calls that overlap on
 *   one GPU (different streams, or threads without ordering) race and give
 *   undefined results.  Calls ordered on one stream are safe.  Nothing in the
 *   array needs to start at zero: each call writes every value it reads. */
int fb_denoise_update_noalloc(const void* logits, int V, int dtype, int32_t* tokens,
                              int T_max, float* conf, int32_t* argmax, fb_req_state* st,
                              uint8_t* pe, uint8_t* fin, int n_max, const fb_pack* pack,
                              const fb_update_params* prm, fb_req_stats* stats,
                              void* stream);

/* ---- Measured HBM ceilings ---------------------------------------------- */

/* Workgroups of the probes: fb_hbm_read_probe writes one word per workgroup. */
#define FB_PROBE_BLOCKS 2048

/* Read-only stream over `bytes` of device memory at `src` with the load form
 * of the vocabulary pass (16-byte nontemporal loads), in the fastest read
 * pattern measured (the workgroups walk the buffer together in 32 KB blocks,
 * eight loads in flight per thread): the measured read ceiling the
 * vocabulary reduction is set against.  out (device uint32[FB_PROBE_BLOCKS])
 * receives, per workgroup, the XOR of the 32-bit words it read; the XOR of
 * all of them is the XOR of every word of the buffer.
 *   src     16-byte aligned; bytes a positive multiple of 16 */
int fb_hbm_read_probe(const void* src, size_t bytes, uint32_t* out, void* stream);

/* Device copy of `bytes` from src to dst (16-byte loads and stores, a
 * contiguous share per workgroup): the measured read+write ceiling.  Both 16-byte aligned, not
 * overlapping; bytes a positive multiple of 16. */
int fb_hbm_copy_probe(const void* src, void* dst, size_t bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* FLOWBLOCK_H */
