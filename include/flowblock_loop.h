/*
 * flowblock_loop.h -- the multi-step decode loop of Alg. 1 on the device,
 * driven by a deterministic synthetic model in place of f_theta.
 *
 * Alg. 1 repeats one step -- forward the live windows, update, retire,
 * admit -- until every request has committed its blocks.  The step's own
 * calls are in flowblock.h; this header adds what a loop needs around them:
 *
 *   fb_synth_embed       synthetic q / k / v rows of the live window tokens
 *   fb_synth_logits      synthetic logits of the live rows (the model output)
 *   fb_decode_loop       enqueue steps until no request is active, reading one
 *                        device flag every `check_every` steps (optionally
 *                        replaying the steps as a captured HIP graph)
 *
 * The synthetic model exists because no trained weights are part of this
 * library: it is a hash model whose logits depend on exactly the tokens a
 * block may see under the block-causal visibility of Sec. 4.1, so that the
 * loop's schedule (admission, T2T repair of stale drafts, retirement) can be
 * run and checked end to end.  Its definition (SplitMix64, Steele, Lea and
 * Flood, OOPSLA 2014, used as a counter-based hash):
 *
 *   H(s, n) = mix(s + (n + 1) * 0x9E3779B97F4A7C15)   (the n-th output of
 *             SplitMix64 seeded with s; all arithmetic mod 2^64), where
 *   mix(z): z ^= z >> 30; z *= 0xBF58476D1CE4E5B9; z ^= z >> 27;
 *           z *= 0x94D049BB133111EB; z ^= z >> 31
 *
 *   c(j, x) = H(seed, j * 2^32 + x)          contribution of token x at j
 *   t(p)    = H(seed, 2^63 + p) mod (V - 1)  the "true" token of position p
 *   block [lo, hi = lo + bl) of request b (block 0 at gen_start_b):
 *     ctx   = sum of c(j, x_j) over j < hi with x_j != mask_id   (mod 2^64)
 *     stale = number of j in [gen_start_b, lo) with x_j == mask_id
 *     first = lowest position of the block holding mask_id, if any
 *   row p of the block, h = H(ctx, p):
 *     k = t(p) if stale == 0 or bit 63 of h is 0, else h mod (V - 1)
 *     l = (h >> 32) & 3, or 3 when p == first
 *     logits: z_v = 0 for v != k, z_k = levels[l]
 *   embeddings (kind 0 = q, 1 = k, 2 = v) of a row at position p with token
 *   x, head hd, dimension i (head_dim d):
 *     e = ((H(H(H(seed, 2^62 + kind * 2^59 + p), x), hd * d + i) >> 56)
 *          - 128) / 256
 *
 * mask_id must be V - 1 (the model never predicts it).  Every function
 * follows the conventions of flowblock.h (caller-owned device memory,
 * stream-ordered, FB_* status, fb_last_error()).
 */
#ifndef FLOWBLOCK_LOOP_H
#define FLOWBLOCK_LOOP_H

#include "flowblock.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Parameters of the synthetic model. */
typedef struct fb_synth_model {
    uint64_t seed;
    float    levels[4];   /* peak heights: finite, > 0 and exactly
                             representable in the logits dtype              */
} fb_synth_model;

/* Device counters of a decode loop (caller-owned, zero before the loop). */
typedef struct fb_loop_counters {
    int32_t steps;        /* steps that began with an active request          */
    int32_t any_active;   /* 1 while some request is active (last check)     */
    int32_t reserved[2];
} fb_loop_counters;

/* Synthetic q [row_cap][Hq][d], k_new and v_new [row_cap][Hkv][d] (dtype of
 * the shape) for every live row of the pack, from the row's position and the
 * token the pack gathered for it (row_tok: call fb_pack_wavefronts with a
 * non-NULL `tokens`).  Rows that are not live are not written. */
int fb_synth_embed(const fb_pack* pack, const fb_attn_shape* sh, uint64_t seed,
                   void* q, void* k_new, void* v_new, void* stream);

/* Synthetic logits of every live row, per the model above, from the tokens
 * at the start of the step (before fb_denoise_update changes them).
 *   st      device fb_req_state[B] (gen_start, L of each request)
 *   tokens  device int32[B][T_max]
 *   pred    device int32[row_cap][2], written: {k, level} of each live row
 *   logits  device [row_cap][V], FB_BF16 or FB_F32; live rows written whole
 * Requests the pack marked ill-formed produce no rows. */
int fb_synth_logits(const fb_req_state* st, const int32_t* tokens, int T_max,
                    const fb_pack* pack, const fb_synth_model* model, int V,
                    int dtype, int32_t* pred, void* logits, void* stream);

/* Everything one step of the loop reads and writes.  Device pointers unless
 * noted; the loop updates st, tokens, pe, fin in place. */
typedef struct fb_loop_args {
    /* request state */
    fb_req_state* st;
    int32_t*      tokens;
    int32_t       T_max;
    int32_t       n_max;
    uint8_t*      pe;
    uint8_t*      fin;
    /* host structs */
    const fb_pack*          pack;     /* its device buffer is rewritten each step */
    const fb_update_params* prm;      /* FB_SYNC_WINDOW selects the synchronous
                                         variant                                 */
    const fb_synth_model*   model;
    /* model output and update */
    void*         logits;             /* [row_cap][V]                            */
    int32_t       V;
    int32_t       logit_dtype;        /* FB_BF16 or FB_F32                       */
    int32_t*      pred;               /* int32[row_cap][2]                       */
    float*        conf;               /* [row_cap]                               */
    int32_t*      argmax;             /* [row_cap]                               */
    fb_req_stats* stats;              /* [B] or NULL                             */
    void*         upd_ws;
    size_t        upd_ws_bytes;
    /* optional attention leg: window KV write (Eq. 6) and attention
       (Sec. 4.1) on synthetic embeddings; shape NULL skips it */
    const fb_attn_shape* shape;       /* host struct                             */
    void*          q;
    void*          k_new;
    void*          v_new;
    void*          k_cache;
    void*          v_cache;
    const int32_t* page_table;
    void*          attn_out;
    void*          attn_ws;
    size_t         attn_ws_bytes;
    uint64_t       embed_seed;
    /* loop bookkeeping */
    fb_loop_counters* counters;
    int32_t*          forwards;       /* int32[B]: steps in which the request had
                                         a live window (its forwards)             */
} fb_loop_args;

/* Alg. 1's outer loop: one step is
 *   count (counters, forwards) -> fb_pack_wavefronts
 *   [-> fb_synth_embed -> fb_write_window_kv -> fb_wavefront_attention]
 *   -> fb_synth_logits -> fb_denoise_update,
 * all enqueued on `stream` with no host wait.  Steps are enqueued in groups
 * of `check_every`; after each group one 4-byte flag (any request still
 * active) is copied to the host and waited for, and the loop ends when it is
 * 0 or `max_steps` steps have been enqueued.  A step that begins with no
 * active request changes nothing, so a group may overrun the end.  With
 * `use_graph` the group is captured once into a HIP graph on `stream` (which
 * must then not be the null stream) and replayed; the graph is destroyed
 * before return.
 *   steps_out  host: steps enqueued (>= the counted steps); may be NULL
 *   done_out   host: 1 if no request is active at the end; may be NULL
 * The counted steps and per-request forwards are in counters / forwards. */
int fb_decode_loop(const fb_loop_args* args, int max_steps, int check_every,
                   int use_graph, int* steps_out, int* done_out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* FLOWBLOCK_LOOP_H */
