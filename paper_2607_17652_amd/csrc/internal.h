// Internal declarations shared by the translation units of libflowblock.so.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "flowblock.h"
#include "flowblock_loop.h"

namespace fb {

// ---- packed-batch buffer (int32 units) ------------------------------------
constexpr int kHdrInts = 16;
constexpr int kTileInts = 8;
enum HeaderField { kHdrRows = 0, kHdrTiles = 1, kHdrStatus = 2 };
enum TileField { kTB = 0, kTS, kTG, kTRow0, kTPos0, kTO, kTKvLen, kTW };

struct PackView {
    int32_t* hdr;
    int32_t* tiles;
    int32_t* req_w;
    int32_t* req_row0;
    int32_t* row_req;
    int32_t* row_pos;
    int32_t* row_tok;
};

inline void pack_offsets_ints(int B, int tile_cap, int row_cap, size_t o[8]) {
    o[0] = 0;                                          // header
    o[1] = kHdrInts;                                   // tiles
    o[2] = o[1] + (size_t)tile_cap * kTileInts;        // req_w
    o[3] = o[2] + (size_t)B;                           // req_row0
    o[4] = o[3] + (size_t)B;                           // row_req
    o[5] = o[4] + (size_t)row_cap;                     // row_pos
    o[6] = o[5] + (size_t)row_cap;                     // row_tok
    o[7] = o[6] + (size_t)row_cap;                     // total
}

inline PackView pack_view(const fb_pack* p) {
    size_t o[8];
    pack_offsets_ints(p->B, p->tile_cap, p->row_cap, o);
    int32_t* base = static_cast<int32_t*>(p->buf);
    return PackView{base + o[0], base + o[1], base + o[2], base + o[3],
                    base + o[4], base + o[5], base + o[6]};
}

// Record a device-side error for request `req`: the status word keeps the
// lowest (request, code) key, so the result does not depend on timing.
__device__ inline void record_error(int32_t* hdr, int req, int code) {
    atomicMin(&hdr[kHdrStatus], req * 16 + code);
}

// ---- launchers (each returns the launch status) ---------------------------
hipError_t launch_pack(const fb_req_state* st, const int32_t* tokens, int n_max,
                       int T_max, const fb_pack* pack, hipStream_t stream);

hipError_t launch_write_kv(const void* k_new, const void* v_new, void* k_cache,
                           void* v_cache, const int32_t* page_table,
                           const fb_pack* pack, const fb_attn_shape* sh,
                           hipStream_t stream);

struct AttnPlanSizes {
    int rows_per_unit;    // bl * (Hq / Hkv)
    int row_groups;       // 128-row groups per unit
    int unit_cap;         // tile_cap * Hkv * row_groups
    int item_cap;         // work items the plan may emit
    int slot_cap;         // split partial slots
    int target_items;     // automatic split target
    int split_cap;        // units with more than one piece (slot_cap / 2)
    size_t off_items, off_units, off_counts, off_split, off_part_o, off_part_lse, total;
};
AttnPlanSizes attention_sizes(const fb_pack* pack, const fb_attn_shape* sh,
                              int cu_count);
// the plan kernel alone (no-op for fp32)
hipError_t launch_attention_plan(const fb_pack* pack, const fb_attn_shape* sh, void* ws,
                                 const AttnPlanSizes& sz, hipStream_t stream);
// plan (unless `planned`: ws already holds this pack's plan), attention, combine
hipError_t launch_attention(const void* q, const void* k_cache,
                            const void* v_cache, const int32_t* page_table,
                            const fb_pack* pack, const fb_attn_shape* sh,
                            void* out, void* ws, const AttnPlanSizes& sz,
                            hipStream_t stream, bool planned = false);

struct UpdateSizes {
    int nsplit;      // workgroups (partials) per row in the first pass
    size_t off_rho;  // per-request readiness of the window's last block
    size_t total;    // workspace bytes
};
UpdateSizes update_sizes(const fb_pack* pack, int V, int cu_count);
hipError_t launch_vocab_reduce(const void* logits, int V, int dtype,
                               const fb_pack* pack, void* ws, const UpdateSizes& sz,
                               hipStream_t stream);
hipError_t launch_apply(int32_t* tokens, int T_max, float* conf, int32_t* argmax,
                        fb_req_state* st, uint8_t* pe, uint8_t* fin, int n_max,
                        const fb_pack* pack, const fb_update_params* prm,
                        fb_req_stats* stats, const void* ws, const UpdateSizes& sz,
                        hipStream_t stream);

size_t prologue_smem_bytes(const fb_pack* pack, const fb_attn_shape* sh, int* pitch_out);
hipError_t launch_window_prologue(const void* q_in, void* q_out, const void* k_new,
                                  const void* v_new, void* k_cache, void* v_cache,
                                  const int32_t* page_table, const fb_pack* pack,
                                  const fb_attn_shape* sh, double rope_base,
                                  hipStream_t stream);

struct LmSizes {
    int n_rtiles;        // 256-token tiles over row_cap
    int n_vtiles;        // 256-id vocabulary tiles
    int cu;              // compute units the partition count is chosen for
    int grid;            // workgroups: the most any row count needs
    size_t total;        // workspace bytes (256 partials per workgroup)
};
LmSizes lm_sizes(const fb_pack* pack, int V, int D, int cu_count);
hipError_t launch_lmhead(const void* hidden, const void* weight, int D, int V,
                         const fb_pack* pack, void* lm_ws, const LmSizes& z, void* upd_ws,
                         const UpdateSizes& uz, hipStream_t stream);

struct SynthSizes {
    int nsplit;      // vocabulary partitions per row of the logits fill
    int chunk;       // elements per partition (multiple of 8)
};
SynthSizes synth_sizes(const fb_pack* pack, int V);
hipError_t launch_synth_logits(const fb_req_state* st, const int32_t* tokens, int T_max,
                               const fb_pack* pack, const fb_synth_model* m, int V,
                               int dtype, int32_t* pred, void* logits, hipStream_t stream);
hipError_t launch_synth_embed(const fb_pack* pack, const fb_attn_shape* sh, uint64_t seed,
                              void* q, void* k_new, void* v_new, hipStream_t stream);
hipError_t launch_read_probe(const void* src, size_t bytes, uint32_t* out,
                             hipStream_t stream);
hipError_t launch_copy_probe(const void* src, void* dst, size_t bytes, hipStream_t stream);
hipError_t launch_loop_count(const fb_req_state* st, int B, fb_loop_counters* counters,
                             int32_t* forwards, int count, hipStream_t stream);

}  // namespace fb
