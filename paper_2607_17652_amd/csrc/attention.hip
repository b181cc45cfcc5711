// W-shaped block-causal window attention (Sec. 4.1; Eq. 5 per packed row).
//
// The mask of Eq. 5 reduces, for window slot s of request b, to one key count
// kv_len = o_b + (s+1)*bl: every query of that block sees keys [0, kv_len) of
// its KV head -- the frozen prefix, the earlier live blocks and its own block.
// So the work is a set of independent "prefix attentions", one per
// (live block, KV head), each with bl*(Hq/Hkv) query rows sharing one K/V
// stream (GQA rows packed together).
//
// Work decomposition (all shapes fixed by capacity, so graph-capturable):
//   unit  = (tile, KV head, 128-row group); rows are the block's
//           (position, head-in-group) pairs flattened position-major
//   item  = a unit's key range [kb, ke), a multiple of 32 keys long except at
//           kv_len; long units are split so the grid has enough items
//   plan_kernel    one workgroup: counts key tiles, picks the split size,
//                  emits items (longest first, each with its tile's request
//                  and first row), per-unit split counts and partial slots,
//                  and the list of split units
//   attn_bf16      one workgroup (4 waves x 32 rows) per item: 32-key K and
//                  V^T tiles streamed through an LDS ring (3 stages at
//                  D = 128, K refilled a step ahead of V^T; 4 below) by
//                  direct global->LDS loads,
//                  S^T = K Q^T and O^T += V^T P^T on
//                  v_mfma_f32_32x32x16_bf16, online softmax in the exp2
//                  domain with lazy rescaling
//   combine        merges split partials with their log-sum-exp weights,
//                  walking the plan's list of split units
//   attn_f32       a plain fp32 path (small problems, exactness reference)
#include <type_traits>
#include <utility>

#include "internal.h"

namespace fb {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kRowsPerWg = 128;     // 4 waves x 32 query rows
constexpr int kAttnThreads = 256;
constexpr int kWgsPerCu = 3;          // resident attention workgroups per CU
constexpr int kKeyTile = 32;
constexpr int kMinChunkTiles = 4;   // never split below 128 keys
constexpr int kMaxSplits = 64;      // splits of one unit the combine can merge
constexpr int kMaxHeadDim = 128;    // largest head_dim built (32, 64, 128)
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kRescaleSlack = 8.0f;  // lazy rescale: running max may lag by 2^8

// A work item: its unit, key range and partial slot, and the request and
// first packed row of its tile (copied here so the attention workgroup's
// first dependent loads are the item and then the page table).
enum ItemField { kIUnit = 0, kIKb, kIKe, kISlot, kIB, kIRow0, kIItemInts = 8 };
enum UnitField { kUSplits = 0, kUSlot0 };
enum CountField { kCItems = 0, kCUnits, kCChunk, kCSplit };

struct AttnWs {
    int32_t* items;    // [item_cap][kIItemInts]
    int32_t* units;    // [unit_cap][2]
    int32_t* counts;   // [4]
    int4* split;       // [split_cap]: {unit, pieces, first slot, first row} of the
                       // units with more than one piece
    float* part_o;     // [slot_cap][128][D]
    float* part_lse;   // [slot_cap][128]
};

// Capacities a plan record must respect to belong to this pack and shape.
// The attention and the combine check every record they read against them,
// so a workspace used without its plan (fb_wavefront_attention_planned
// before fb_attention_plan) is reported, never followed out of bounds.
struct PlanBounds {
    int n_req;          // requests of the pack
    int row_cap;        // packed rows
    int unit_cap;       // units
    int slot_cap;       // split partial slots
    long long max_keys; // keys the page table can address
};


// ---------------------------------------------------------------- plan ----
constexpr int kPlanThreads = 256;   // 4 waves: shorter barrier and scan rounds than 16 (measured 2-4%)
constexpr int kPlanWaves = kPlanThreads / 64;

// Workgroup sum of v[0] and maximum of v[1] (one pair of barriers): each
// wave reduces its 64 lanes, then every wave reduces the kPlanWaves wave
// results itself and broadcasts lane 0's (no serial loop on one thread).
__device__ void wg_sum_max(long long (&v)[2], long long (*lds)[kPlanWaves]) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        v[0] += __shfl_xor(v[0], off, 64);
        const long long o = __shfl_xor(v[1], off, 64);
        if (o > v[1]) v[1] = o;
    }
    if (lane == 0) {
        lds[0][wave] = v[0];
        lds[1][wave] = v[1];
    }
    __syncthreads();
    long long sm = lane < kPlanWaves ? lds[0][lane] : 0;
    long long mx = lane < kPlanWaves ? lds[1][lane] : 0;
#pragma unroll
    for (int off = kPlanWaves / 2; off > 0; off >>= 1) {
        sm += __shfl_xor(sm, off, 64);
        const long long o = __shfl_xor(mx, off, 64);
        if (o > mx) mx = o;
    }
    v[0] = __shfl(sm, 0, 64);
    v[1] = __shfl(mx, 0, 64);
    __syncthreads();
}

// Exclusive scans of three ints per thread across the workgroup (one pair of
// barriers for all three): v[i] becomes its exclusive prefix, tot[i] the
// workgroup total.
__device__ void wg_excl_scan3(int (&v)[3], int (&tot)[3], int3* lds) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int x[3] = {v[0], v[1], v[2]};
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
#pragma unroll
        for (int i = 0; i < 3; ++i) {
            const int u = __shfl_up(x[i], off, 64);
            if (lane >= off) x[i] += u;
        }
    }
    if (lane == 63) lds[wave] = make_int3(x[0], x[1], x[2]);
    __syncthreads();
    const int3 l = lane < kPlanWaves ? lds[lane] : make_int3(0, 0, 0);
    int w[3] = {l.x, l.y, l.z};
#pragma unroll
    for (int off = 1; off < kPlanWaves; off <<= 1) {
#pragma unroll
        for (int i = 0; i < 3; ++i) {
            const int u = __shfl_up(w[i], off, 64);
            if (lane >= off) w[i] += u;
        }
    }
#pragma unroll
    for (int i = 0; i < 3; ++i) {
        const int before = __shfl(w[i], wave > 0 ? wave - 1 : 0, 64);
        tot[i] = __shfl(w[i], kPlanWaves - 1, 64);
        v[i] = (wave > 0 ? before : 0) + x[i] - v[i];
    }
    __syncthreads();
}

// Exclusive scan of one int per thread across the workgroup, and the total.
__device__ int wg_excl_scan(int v, int* lds, int* total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int x = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        int y = __shfl_up(x, off, 64);
        if (lane >= off) x += y;
    }
    if (lane == 63) lds[wave] = x;
    __syncthreads();
    // every wave scans the wave totals itself
    int w = lane < kPlanWaves ? lds[lane] : 0;
#pragma unroll
    for (int off = 1; off < kPlanWaves; off <<= 1) {
        int y = __shfl_up(w, off, 64);
        if (lane >= off) w += y;
    }
    const int before = wave > 0 ? __shfl(w, wave - 1, 64) : 0;
    *total = __shfl(w, kPlanWaves - 1, 64);
    __syncthreads();
    return before + x - v;
}

// Items are written longest first (a counting sort on their key-tile count,
// counts of kLenBuckets-1 or more sharing the top bucket): the grid then
// dispatches long items before short ones, which keeps the tail short.  The
// plan works per tile: the per_tile units of a tile (kv-heads x row groups)
// have the same key range, so they get the same split and adjacent items
// (with 8 kv-heads the round-robin dispatch then keeps each kv-head on one
// XCD).  Thread i handles tiles i, i + kPlanThreads, ...; the fields of its
// first kPlanCache tiles are read once and kept in LDS.
constexpr int kLenBuckets = kPlanThreads;
constexpr int kPlanCache = 4;
constexpr int kPlanPieces = 1024;   // pieces of one round staged in LDS

struct PlanTile {
    int kt;   // key tiles of the tile; 0 (skipped, error) past the page table
    int kr;   // sort key: key tiles of its request's last live block
    int kv;   // keys the tile attends to
    int b;    // request
    int row0; // first packed row
};

__device__ inline PlanTile plan_tile(const int32_t* tiles, int t, int n_tiles, long long max_keys) {
    PlanTile p{0, 0, 0, 0, 0};
    if (t >= n_tiles) return p;
    const int32_t* tl = tiles + (size_t)t * kTileInts;
    p.kv = tl[kTKvLen];
    p.b = tl[kTB];
    p.row0 = tl[kTRow0];
    p.kt = (long long)p.kv > max_keys ? 0 : (p.kv + kKeyTile - 1) / kKeyTile;
    // the blocks of one request read the same prefix K/V: keyed by the
    // request's longest block they land in the same buckets next to each
    // other and run together, sharing the prefix through L2
    const long long blen = tl[kTKvLen] - tl[kTPos0];
    const long long kv_last = tl[kTO] + (long long)tl[kTW] * blen;
    const long long kr = (kv_last + kKeyTile - 1) / kKeyTile;
    p.kr = kr > p.kt ? (int)kr : p.kt;
    return p;
}

__global__ void __launch_bounds__(kPlanThreads)
plan_kernel(PackView pv, AttnWs ws, int Hkv, int RG, int item_cap, int slot_cap,
            int split_cap, int target_items, int fixed_chunk_tiles, long long max_keys) {
    __shared__ long long sum_lds[2][kPlanWaves];
    __shared__ int scan_lds[kPlanWaves + 1];
    __shared__ int3 trio_lds[kPlanWaves];
    __shared__ int bucket[kLenBuckets];
    const int n_tiles = pv.hdr[kHdrTiles];
    const int per_tile = Hkv * RG;
    const int n_units = n_tiles * per_tile;
    const int n_rounds = (n_tiles + kPlanThreads - 1) / kPlanThreads;

    // this thread's first kPlanCache tiles, read once; kept in LDS (a
    // register array indexed by the round would live in scratch memory)
    __shared__ PlanTile s_cache[kPlanCache * kPlanThreads];
#pragma unroll
    for (int j = 0; j < kPlanCache; ++j)
        s_cache[j * kPlanThreads + threadIdx.x] =
            plan_tile(pv.tiles, j * kPlanThreads + threadIdx.x, n_tiles, max_keys);
    // this thread's tile of round c (zeros past the end)
    auto tile_of = [&](int c) -> PlanTile {
        if (c >= kPlanCache)
            return plan_tile(pv.tiles, c * kPlanThreads + threadIdx.x, n_tiles, max_keys);
        return s_cache[c * kPlanThreads + threadIdx.x];
    };

    // key tiles summed over the tiles, and the longest tile
    long long red[2] = {0, 0};
    for (int c = 0; c < n_rounds; ++c) {
        const int kt = tile_of(c).kt;
        red[0] += kt;
        if (kt > red[1]) red[1] = kt;
    }
    wg_sum_max(red, sum_lds);
    const long long total_tiles = red[0] * per_tile;
    const long long kt_max = red[1];

    // Split size.  With chunk >= total_tiles / target_items the items and
    // the partial slots always fit: a unit of kt key tiles makes
    // ceil(kt/chunk) <= kt/chunk + 1 items, so all units make at most
    // total_tiles/chunk + n_units <= item_cap, and a split unit's
    // ceil(kt/chunk) < 2 kt/chunk slots sum to at most 2 target_items =
    // slot_cap.  A chunk >= kt_max / kMaxSplits keeps every unit within the
    // splits the combine merges.  A requested split size is doubled until
    // both hold.  (Sizes stay below 2^30 key tiles: 32-bit math below.)
    long long need = (total_tiles + target_items - 1) / target_items;
    const long long need_m = (kt_max + kMaxSplits - 1) / kMaxSplits;
    if (need_m > need) need = need_m;
    long long chunk_ll;
    if (fixed_chunk_tiles > 0) {
        chunk_ll = fixed_chunk_tiles;
        while (chunk_ll < need) chunk_ll *= 2;
    } else {
        chunk_ll = need > kMinChunkTiles ? need : kMinChunkTiles;
    }
    if (chunk_ll >= (1 << 30)) {
        // beyond any real cache (over 2^30 key tiles per item): nothing is
        // planned and the first tile's request is flagged
        if (threadIdx.x == 0) {
            record_error(pv.hdr, pv.tiles[kTB], FB_DERR_PAGE);
            ws.counts[kCItems] = 0;
            ws.counts[kCUnits] = 0;
            ws.counts[kCChunk] = -1;
            ws.counts[kCSplit] = 0;
        }
        return;
    }
    const int chunk = (int)chunk_ll;

    // Histogram of item lengths, then each bucket's first position with the
    // longest bucket first.
    // A unit of at most 1.5 chunks stays whole (a piece of half a chunk or
    // less costs more in its partial result and merge than it saves in
    // balance: measured 5% on hetero64's attention); longer units are cut
    // into chunk-sized pieces and a shorter last one.  Either way a unit
    // makes at most ceil(kt / chunk) items, so the bounds above hold.
    auto nsplit = [&](int kt) -> int {
        return 2LL * kt > 3LL * chunk ? (kt + chunk - 1) / chunk : (kt > 0 ? 1 : 0);
    };
    auto len_key = [&](int kt, int k) -> int {
        const int nsk = nsplit(kt);
        int len = nsk == 1 ? kt : kt - k * chunk;
        if (nsk > 1 && len > chunk) len = chunk;
        return len >= kLenBuckets - 1 ? kLenBuckets - 1 : len;
    };
    bucket[threadIdx.x] = 0;
    __syncthreads();
    for (int c = 0; c < n_rounds; ++c) {
        const PlanTile p = tile_of(c);
        const int ns = nsplit(p.kt);
        for (int k = 0; k < ns; ++k) atomicAdd(&bucket[len_key(p.kr, k)], per_tile);
    }
    __syncthreads();
    {
        const int rev = kLenBuckets - 1 - threadIdx.x;   // descending length order
        const int cnt = bucket[rev];
        int total_items;
        const int first = wg_excl_scan(cnt, scan_lds, &total_items);
        bucket[rev] = first;
        __syncthreads();
    }

    // A round's pieces are staged in LDS, then their items (a piece's
    // per_tile items are contiguous) and the round's units are written by
    // consecutive threads to consecutive entries, so the stores coalesce;
    // a round with more pieces than the stage holds writes its items from
    // the owning thread instead.
    __shared__ int4 s_pc[kPlanPieces];   // per piece: first item, kb, ke, slot base (or -1)
    __shared__ int4 s_pt[kPlanPieces];   // per piece: tile, splits of the tile, request, first row
    __shared__ int4 s_tl[kPlanThreads];  // per tile of the round: splits, first slot, first
                                         // split entry, first row
    // the entries a thread writes: unit / item j of every tpi-th tile or
    // piece from my_tl on (no division per entry)
    const int tpi = per_tile <= kPlanThreads ? kPlanThreads / per_tile : 1;
    const int my_tl = per_tile <= kPlanThreads ? (int)threadIdx.x / per_tile : 0;
    const int my_j = per_tile <= kPlanThreads ? (int)threadIdx.x % per_tile : 0;
    const bool by_lane = per_tile <= kPlanThreads;
    int items_before = 0, slots_before = 0, split_before = 0;
    for (int c = 0; c < n_rounds; ++c) {
        const int t = c * kPlanThreads + threadIdx.x;
        const PlanTile p = tile_of(c);
        const int ns = nsplit(p.kt);
        if (t < n_tiles && p.kt == 0)
            record_error(pv.hdr, pv.tiles[(size_t)t * kTileInts + kTB], FB_DERR_PAGE);
        // items, partial slots and split units of this round's tiles
        int ex[3] = {ns * per_tile, ns > 1 ? ns * per_tile : 0, ns > 1 ? per_tile : 0};
        int tot[3];
        wg_excl_scan3(ex, tot, trio_lds);
        const int slot_t = slots_before + ex[1];     // unit j owns slots slot_t + j*ns ..
        const int split_t = split_before + ex[2];    // and, when split, list entry split_t + j
        const int piece0 = ex[0] / per_tile;         // this tile's first piece in the round
        const int round_pieces = tot[0] / per_tile;
        const bool staged = round_pieces <= kPlanPieces;
        s_tl[threadIdx.x] = make_int4(ns, slot_t, split_t, p.row0);
        if (t < n_tiles) {
            for (int k = 0; k < ns; ++k) {
                const int pos = atomicAdd(&bucket[len_key(p.kr, k)], per_tile);
                const long long kb = (long long)k * chunk * kKeyTile;
                long long ke = k == ns - 1 ? (long long)p.kv : kb + (long long)chunk * kKeyTile;
                if (ke > p.kv) ke = p.kv;
                const int slot_k = ns > 1 ? slot_t + k : -1;
                if (staged) {
                    s_pc[piece0 + k] = make_int4(pos, (int)kb, (int)ke, slot_k);
                    s_pt[piece0 + k] = make_int4(t, ns, p.b, p.row0);
                } else {
                    for (int j = 0; j < per_tile; ++j) {
                        if (pos + j >= item_cap) break;   // cannot happen: the caps hold
                        int4* it = reinterpret_cast<int4*>(ws.items + (size_t)(pos + j) * kIItemInts);
                        it[0] = make_int4(t * per_tile + j, (int)kb, (int)ke,
                                          slot_k < 0 ? -1 : slot_k + j * ns);
                        it[1] = make_int4(p.b, p.row0, 0, 0);
                    }
                }
            }
        }
        __syncthreads();
        int round_tiles = n_tiles - c * kPlanThreads;
        if (round_tiles > kPlanThreads) round_tiles = kPlanThreads;
        auto write_unit = [&](int tl, int j) {
            const int4 q = s_tl[tl];
            const int u = (c * kPlanThreads + tl) * per_tile + j;
            ws.units[(size_t)u * 2 + kUSplits] = q.x;
            ws.units[(size_t)u * 2 + kUSlot0] = q.x > 1 ? q.y + j * q.x : -1;
            if (q.x > 1 && q.z + j < split_cap)
                ws.split[q.z + j] = make_int4(u, q.x, q.y + j * q.x, q.w);
        };
        auto write_item = [&](int pc, int j) {
            const int4 a = s_pc[pc];
            const int4 m = s_pt[pc];
            if (a.x + j >= item_cap) return;   // cannot happen: the caps hold
            int4* it = reinterpret_cast<int4*>(ws.items + (size_t)(a.x + j) * kIItemInts);
            it[0] = make_int4(m.x * per_tile + j, a.y, a.z, a.w < 0 ? -1 : a.w + j * m.y);
            it[1] = make_int4(m.z, m.w, 0, 0);
        };
        if (by_lane) {
            if (my_tl < tpi) {
                for (int tl = my_tl; tl < round_tiles; tl += tpi) write_unit(tl, my_j);
                if (staged)
                    for (int pc = my_tl; pc < round_pieces; pc += tpi) write_item(pc, my_j);
            }
        } else {
            for (int e = threadIdx.x; e < round_tiles * per_tile; e += kPlanThreads)
                write_unit(e / per_tile, e % per_tile);
            if (staged)
                for (int e = threadIdx.x; e < round_pieces * per_tile; e += kPlanThreads)
                    write_item(e / per_tile, e % per_tile);
        }
        __syncthreads();   // the stage is reused by the next round
        items_before += tot[0];
        slots_before += tot[1];
        split_before += tot[2];
    }
    if (threadIdx.x == 0) {
        ws.counts[kCItems] = items_before < item_cap ? items_before : item_cap;
        ws.counts[kCUnits] = n_units;
        ws.counts[kCChunk] = chunk < (1 << 30) / kKeyTile ? chunk * kKeyTile : -1;   // keys
        ws.counts[kCSplit] = split_before < split_cap ? split_before : split_cap;
    }
}

// --------------------------------------------------------- bf16 MFMA ------
// S^T accumulator layout of v_mfma_f32_32x32x16_bf16 (32x32 fp32 result):
// lane l holds column l%32 and rows (i/4)*8 + (l/32)*4 + i%4 for i = 0..15.
// Loading K row perm(m) into A-row m, with perm swapping index bits 2 and 3,
// makes lane l's value i belong to tile key 16*(i/8) + 8*(l/32) + i%8, i.e.
// eight consecutive keys per MFMA k-step -- exactly the k-slots the PV
// product needs from P^T, so P moves from the S^T accumulator into the B
// operand of the PV MFMA without any data exchange.
__device__ inline int swap_bits23(int m) {
    return (m & ~12) | ((m & 4) << 1) | ((m & 8) >> 1);
}

__device__ inline float wave_xor32_max(float x) {
    return fmaxf(x, __shfl_xor(x, 32, 64));
}

// K/V staging: a ring of Ring<D>::kStages key tiles in LDS, filled by direct
// global->LDS loads (global_load_lds_dwordx4: lane i of a wave writes 16 bytes
// at M0 + 16*i).  A stage holds the K tile [32 keys][D] followed by the V^T
// tile [D][32 keys], both in 16-byte chunks whose position inside a row is
// XOR-swizzled (K: chunk ^ (key % (D/8)); V^T: chunk ^ ((d/4) % 4)) so that
// the MFMA operand reads of 16 lanes hit 16 distinct bank groups.  The loads
// are issued from inline asm so the compiler neither sees nor waits on them;
// the kernel orders them itself with explicit vmcnt waits and raw barriers.
template <int N, typename F, int... I>
__device__ __attribute__((always_inline)) inline void static_for_impl(F& f, std::integer_sequence<int, I...>) {
    (f(std::integral_constant<int, I>{}), ...);
}
// f(std::integral_constant<int, 0>) ... f(std::integral_constant<int, N-1>)
template <int N, typename F>
__device__ __attribute__((always_inline)) inline void static_for(F&& f) {
    static_for_impl<N>(f, std::make_integer_sequence<int, N>{});
}

template <int D>
struct Ring {
    // Stages of the ring: three workgroups per CU (12 waves, 3 per SIMD)
    // share its 160 KB of LDS -- 3 x 48 KB at D = 128.  The third wave per
    // SIMD hides more of the exp and DMA issue work behind other waves'
    // MFMAs than a fourth ring stage would hide load latency.
    static constexpr int kStages = D == 128 ? 3 : 4;
    static constexpr int kKCh = kKeyTile * D / 8;   // K chunks per stage
    static constexpr int kVCh = D * kKeyTile / 8;   // V^T chunks per stage
    static constexpr int kCh = kKCh + kVCh;
    static constexpr int kStageBytes = kCh * 16;
    static constexpr int kPerThread = kCh / kAttnThreads;   // D / 32
    static_assert(kCh % kAttnThreads == 0, "chunks must divide the workgroup");
};

__device__ inline void dma16(const void* src, uint32_t lds_wave_base) {
    asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off"
                 :: "s"(lds_wave_base), "v"(src) : "memory");
}

__device__ inline void barrier_raw() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Wait until at most n of this wave's vector-memory loads are outstanding.
__device__ inline void wait_vm(int n) {
    switch (n) {
        case 0: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
        case 1: asm volatile("s_waitcnt vmcnt(1)" ::: "memory"); break;
        case 2: asm volatile("s_waitcnt vmcnt(2)" ::: "memory"); break;
        case 3: asm volatile("s_waitcnt vmcnt(3)" ::: "memory"); break;
        case 4: asm volatile("s_waitcnt vmcnt(4)" ::: "memory"); break;
        case 6: asm volatile("s_waitcnt vmcnt(6)" ::: "memory"); break;
        case 8: asm volatile("s_waitcnt vmcnt(8)" ::: "memory"); break;
        case 12: asm volatile("s_waitcnt vmcnt(12)" ::: "memory"); break;
        default: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
    }
}

// FAST: pages hold whole key tiles (page_size >= 32), so a tile's loads share
// one scalar base; otherwise each lane picks its page.
template <int D, bool FAST>
__global__ void __launch_bounds__(kAttnThreads, kWgsPerCu)
attn_bf16_kernel(const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_cache,
                 const uint16_t* __restrict__ v_cache,
                 const int32_t* __restrict__ page_table, PackView pv, AttnWs ws,
                 uint16_t* __restrict__ out, int Hq, int Hkv, int g, int bl, int RG,
                 int ps, int ps_shift, int max_pages, int num_pages, float scale_log2,
                 PlanBounds bounds) {
    using RG_ = Ring<D>;
    constexpr int NS = RG_::kStages;
    __shared__ __attribute__((aligned(16))) unsigned char ring[NS * RG_::kStageBytes];
    constexpr int KK = D / 16;      // k-steps of the S^T product
    constexpr int DT = D / 32;      // 32-wide d tiles of O^T
    constexpr int NCH = RG_::kPerThread;
    constexpr int CPR = D / 8;      // 16-byte chunks per K row
    // A thread's loads j < NK fetch K and the rest V^T, for every wave when
    // the K chunks fill whole loads.  Then (D = 128) K and V^T are refilled
    // separately, K one step ahead (the split ring below).
    constexpr int NK = RG_::kKCh / kAttnThreads;
    constexpr bool SPLIT_RING = NS == 3 && RG_::kKCh % kAttnThreads == 0;

    // The item's record is read together with the item count (the grid has
    // item_cap workgroups, so the record is always inside the buffer).
    const int item = blockIdx.x;
    const int32_t* it = ws.items + (size_t)item * kIItemInts;
    const int u = it[kIUnit], kb = it[kIKb], ke = it[kIKe], slot = it[kISlot];
    const int b = it[kIB], row0 = it[kIRow0];
    const int n_items = ws.counts[kCItems];
    // (the empty asm keeps the compiler from sinking the record's loads below
    // the count check, which would serialize the two round trips)
    asm volatile("" :: "s"(u), "s"(kb), "s"(ke), "s"(slot), "s"(b), "s"(row0), "s"(n_items));
    if (item >= n_items) return;
    if ((unsigned)u >= (unsigned)bounds.unit_cap || kb < 0 || (kb & (kKeyTile - 1)) != 0 ||
        ke <= kb || (long long)ke > bounds.max_keys || slot < -1 || slot >= bounds.slot_cap ||
        (unsigned)b >= (unsigned)bounds.n_req || row0 < 0 || row0 > bounds.row_cap - bl) {
        if (threadIdx.x == 0) record_error(pv.hdr, 0, FB_DERR_PLAN);
        return;
    }
    const int rg = u % RG;
    const int c = (u / RG) % Hkv;
    const int32_t* pt = page_table + (size_t)b * max_pages;

    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const int lane = tid & 63;
    const int n = lane & 31;
    const int h = lane >> 5;
    const int r_local = wave * 32 + n;
    const int r = rg * kRowsPerWg + r_local;
    const bool row_ok = r < bl * g;
    const int pos_local = row_ok ? r / g : 0;
    const int hg = row_ok ? r % g : 0;
    const size_t q_off = ((size_t)(row0 + pos_local) * Hq + c * g + hg) * D;

    // Q fragments, loaded right after the first ring loads are issued so
    // that both latencies overlap (the first wait covers both).
    bf16x8 qf[KK];
    auto load_q = [&]() {
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
            if (row_ok) qf[kk] = *reinterpret_cast<const bf16x8*>(q + q_off + kk * 16 + h * 8);
            else qf[kk] = bf16x8{};
        }
    };

    // Per-thread chunk geometry, the same for every key tile: byte offset of
    // the chunk inside its page (K: [slot][d], V^T: [d][slot]) and the key
    // offset of its first key inside the tile.  Each (load j, wave) is all-K
    // or all-V, so the global base can be a wave-uniform scalar pair.
    uint32_t ch_off[NCH];
    int ch_key[NCH];
    bool ch_isk[NCH];
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
        const int s = j * kAttnThreads + tid;
        if (s < RG_::kKCh) {
            const int key = s / CPR;
            const int dchunk = (s % CPR) ^ (key % CPR);
            ch_isk[j] = true;
            ch_key[j] = key;
            ch_off[j] = (uint32_t)(key * D + dchunk * 8) * 2u;
        } else {
            const int s2 = s - RG_::kKCh;
            const int d = s2 >> 2;
            const int kc = (s2 & 3) ^ ((d >> 2) & 3);
            ch_isk[j] = false;
            ch_key[j] = kc * 8;
            ch_off[j] = (uint32_t)(d * ps + kc * 8) * 2u;
        }
    }
    // Which loads fetch K is wave-uniform; make it scalar so the choice of
    // base pointer is a scalar select, not a divergent branch.
    bool ld_isk[NCH];
#pragma unroll
    for (int j = 0; j < NCH; ++j) ld_isk[j] = __builtin_amdgcn_readfirstlane((int)ch_isk[j]) != 0;
    uint32_t m0_base[NCH];
    const uint32_t ring_base = (uint32_t)(uintptr_t)&ring[0];
#pragma unroll
    for (int j = 0; j < NCH; ++j)
        m0_base[j] = __builtin_amdgcn_readfirstlane(ring_base + j * 4096 + wave * 1024);
    const size_t k_head = (size_t)c * ps * D;        // head c inside a K page
    const size_t v_head = (size_t)c * D * ps;        // head c inside a V page
    const size_t page_elems = (size_t)Hkv * ps * D;  // one page of one cache
    const uint32_t page_bytes = (uint32_t)(page_elems * 2);
    const unsigned char* kb0 = reinterpret_cast<const unsigned char*>(k_cache + k_head);
    const unsigned char* vb0 = reinterpret_cast<const unsigned char*>(v_cache + v_head);

    // Per-lane LDS byte offsets of the MFMA operand reads (stage 0).
    const int krow = swap_bits23(n);
    const int kswz = krow % CPR;
    // chunk (2kk + h) ^ kswz of row krow: the row part and the chunk part
    // occupy disjoint bits, so k-step kk is one XOR away from k-step 0
    const uint32_t kx = (uint32_t)(krow * D + ((h ^ kswz) * 8)) * 2u;
    auto koff = [&](int kk) -> uint32_t { return kx ^ (uint32_t)(kk << 5); };
    // V^T rows d = dt*32 + n share the swizzle of row n ((d/4)%4 does not
    // depend on dt), so d tile dt is a constant offset from d tile 0.
    uint32_t voff0[2];
#pragma unroll
    for (int tt = 0; tt < 2; ++tt)
        voff0[tt] = RG_::kKCh * 16 + (uint32_t)(n * kKeyTile + (((tt * 2 + h) ^ ((n >> 2) & 3)) * 8)) * 2u;
    constexpr uint32_t kVdt = 32 * kKeyTile * 2;   // bytes between d tiles of V^T
    auto voff = [&](int dt, int tt) -> uint32_t { return voff0[tt] + dt * kVdt; };

    // Issue the loads of key tile kt into stage STAGE.
    // Page id of key tile kt when a page holds whole tiles (ps >= kKeyTile);
    // loaded one step before the tile is issued so the scalar load's latency
    // is off the path.
    auto tile_page = [&](int kt) -> int { return pt[(kt * kKeyTile) >> ps_shift]; };
    bool page_err = false;   // a bad page id on the whole-tile path (recorded once at the end)
    // PART 0: the tile's K loads, 1: its V^T loads, 2: both
    auto issue_part = [&](int kt, auto stage_c, int page, auto part_c) __attribute__((always_inline)) {
        constexpr int STAGE = decltype(stage_c)::value;
        constexpr int PART = decltype(part_c)::value;
        constexpr int J0 = PART == 1 ? NK : 0;
        constexpr int J1 = PART == 0 ? NK : NCH;
        const int key0 = kt * kKeyTile;
        if (FAST) {
            // one page per tile: uniform base + per-lane constant offsets
            const bool okp = (unsigned)page < (unsigned)num_pages;
            page_err |= !okp;
            page = okp ? page : 0;
            const uint32_t inpage = (uint32_t)(key0 & (ps - 1));
            const size_t poff = (size_t)(uint32_t)page * (size_t)page_bytes;
            const unsigned char* kbase = kb0 + poff + inpage * (uint32_t)(D * 2);
            const unsigned char* vbase = vb0 + poff + inpage * 2u;
#pragma unroll
            for (int j = J0; j < J1; ++j) {
                const uint32_t m0 = m0_base[j] + STAGE * RG_::kStageBytes;
                // for D >= 64 the K chunks are exactly the first kKCh/256 loads
                const bool isk = (RG_::kKCh % kAttnThreads == 0) ? (j * kAttnThreads < RG_::kKCh)
                                                                 : ld_isk[j];
                const unsigned char* base = isk ? kbase : vbase;
                asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
                             :: "s"(m0), "v"(ch_off[j]), "s"(base) : "memory");
            }
        } else {
            (void)page;
            // several pages per tile: per-lane page selection
            const int pbase = key0 >> ps_shift;
            const int plast = (ke - 1) >> ps_shift;
            int pid[4];
            const int npg = kKeyTile / ps;
#pragma unroll
            for (int i = 0; i < 4; ++i)
                pid[i] = (i < npg && pbase + i <= plast) ? pt[pbase + i] : -1;
#pragma unroll
            for (int j = J0; j < J1; ++j) {
                const int kg = key0 + ch_key[j];
                const int pi = (kg >> ps_shift) - pbase;
                int page = pid[0];
#pragma unroll
                for (int i = 1; i < 4; ++i) page = pi == i ? pid[i] : page;
                const bool ok = kg < ke && page >= 0 && page < num_pages;
                if (kg < ke && !ok) record_error(pv.hdr, b, FB_DERR_PAGE);
                const unsigned char* src = reinterpret_cast<const unsigned char*>(k_cache);
                if (ok) {
                    // ch_off addresses the chunk as if its tile began at slot
                    // 0 of a page; move it to key kg's slot of its page
                    const ptrdiff_t shift = (ptrdiff_t)(kg & (ps - 1)) - ch_key[j];
                    const uint16_t* base =
                        ch_isk[j] ? k_cache + (size_t)page * page_elems + k_head + shift * D
                                  : v_cache + (size_t)page * page_elems + v_head + shift;
                    src = reinterpret_cast<const unsigned char*>(base) + ch_off[j];
                }
                const uint32_t m0 = m0_base[j] + STAGE * RG_::kStageBytes;
                asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off"
                             :: "s"(m0), "v"(src) : "memory");
            }
        }
    };
    auto issue_tile = [&](int kt, auto stage_c, int page) {
        issue_part(kt, stage_c, page, std::integral_constant<int, 2>{});
    };

    floatx16 o[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[dt] = floatx16{};
    float m_run = -INFINITY;   // running max of scores, log2 domain
    float thr_raw = -INFINITY;  // raw score above which the running max moves
    // max over the two lane halves (rows are shared by lanes l and l+32);
    // plain v_max_f32 on values that are never NaN here
    auto half_max = [&](float mx) -> float {
        const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx),
                                                         false, false);
        float r;
        asm("v_max_f32 %0, %1, %2" : "=v"(r) : "v"(__uint_as_float(sw[0])), "v"(__uint_as_float(sw[1])));
        return r;
    };
    float l_acc[2] = {0.f, 0.f};   // this lane's share of the denominator
    bf16x8 pb[2];              // P^T of the current tile (B operand of PV)

    const int kt0 = kb / kKeyTile;
    const int nt = (ke + kKeyTile - 1) / kKeyTile - kt0;
    const int valid_last = ke - (kt0 + nt - 1) * kKeyTile;   // keys of the last tile below ke
    constexpr int kAhead = KK < 2 ? KK : 2;   // LDS operand reads kept in flight

    // S^T of one key tile (K fragments from stage kst) into acc.
    auto s_mfmas = [&](const unsigned char* kst, floatx16& acc) {
        bf16x8 fr[kAhead];
#pragma unroll
        for (int m = 0; m < kAhead; ++m) fr[m] = *reinterpret_cast<const bf16x8*>(kst + koff(m));
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
            const bf16x8 a = fr[kk % kAhead];
            if (kk + kAhead < KK)
                fr[kk % kAhead] = *reinterpret_cast<const bf16x8*>(kst + koff(kk + kAhead));
            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[kk], acc, 0, 0, 0);
        }
    };
    // O^T += V^T P^T of one key tile (V^T fragments from stage vst).
    auto pv_mfmas = [&](const unsigned char* vst) {
        constexpr int NX = DT * 2;
        constexpr int A = NX < 2 ? NX : 2;
        bf16x8 fr[A];
        // product x: d tile x % DT, key half x / DT (consecutive products
        // accumulate into different tiles)
#pragma unroll
        for (int x = 0; x < A; ++x)
            fr[x] = *reinterpret_cast<const bf16x8*>(vst + voff(x % DT, x / DT));
#pragma unroll
        for (int x = 0; x < NX; ++x) {
            const bf16x8 a = fr[x % A];
            if (x + A < NX)
                fr[x % A] = *reinterpret_cast<const bf16x8*>(vst + voff((x + A) % DT, (x + A) / DT));
            o[x % DT] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[x / DT], o[x % DT], 0, 0, 0);
        }
    };
    // Row max of a score tile in the log2 domain (both lane halves hold
    // different keys of the same query row).
    auto tile_max = [&](const floatx16& s) -> float {
        float mx = fmaxf(fmaxf(s[0], s[1]), s[2]);
#pragma unroll
        for (int x = 3; x < 16; x += 2) mx = fmaxf(fmaxf(mx, s[x]), x + 1 < 16 ? s[x + 1] : s[x]);
        return half_max(mx) * scale_log2;
    };
    // P^T = exp2(S^T * scale - m) rounded to bf16, and the denominator from
    // the same rounded weights the PV product uses.
    auto softmax_p = [&](const floatx16& s) {
#pragma unroll
        for (int x = 0; x < 16; ++x)
            pb[x >> 3][x & 7] = (__bf16)__builtin_amdgcn_exp2f(fmaf(s[x], scale_log2, -m_run));
        typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
        const bf16x2 one2 = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
        for (int x = 0; x < 8; x += 2) {
            const bf16x2 p0 = {pb[0][x], pb[0][x + 1]};
            const bf16x2 p1 = {pb[1][x], pb[1][x + 1]};
            l_acc[0] = __builtin_amdgcn_fdot2_f32_bf16(p0, one2, l_acc[0], false);
            l_acc[1] = __builtin_amdgcn_fdot2_f32_bf16(p1, one2, l_acc[1], false);
        }
    };
    // Scores of keys at or past ke (only in the last tile) become -inf.
    auto mask_tail = [&](floatx16& s) {
#pragma unroll
        for (int x = 0; x < 16; ++x) {
            const int key = 16 * (x >> 3) + 8 * h + (x & 7);
            if (key >= valid_last) s[x] = -INFINITY;
        }
    };
    // Lazy rescale: move the running max only when a row's tile max passes
    // it by more than the slack; O and the denominator follow.
    // mx is a raw row max (not scaled); rescale when it passes thr_raw
    auto update_max = [&](float mx) {
        const bool need = mx > thr_raw;
        if (__any(need)) {
            const float m_new = need ? mx * scale_log2 : m_run;
            const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
#pragma unroll
                for (int x = 0; x < 16; ++x) o[dt][x] *= alpha;
            l_acc[0] *= alpha;
            l_acc[1] *= alpha;
            m_run = m_new;
            thr_raw = (m_run + kRescaleSlack) / scale_log2;
        }
    };

    // Phase 1 of a step: S^T of the next tile (K fragments from kst) on the
    // matrix core, while the VALU turns the current tile's scores into P^T.
    // Each group holds one MFMA and a share of the VALU work; scheduling
    // barriers between groups keep that interleave.
    auto phase1 = [&](const unsigned char* kst, const floatx16& sc, floatx16& acc) {
        constexpr int SPG = 16 / KK;   // scores per group
        static_assert(SPG % 2 == 0, "scores go in pairs");
        typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
        const bf16x2 one2 = {(__bf16)1.0f, (__bf16)1.0f};
        bf16x8 fr[kAhead];
#pragma unroll
        for (int m = 0; m < kAhead; ++m) fr[m] = *reinterpret_cast<const bf16x8*>(kst + koff(m));
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
            const bf16x8 a = fr[kk % kAhead];
            if (kk + kAhead < KK)
                fr[kk % kAhead] = *reinterpret_cast<const bf16x8*>(kst + koff(kk + kAhead));
            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[kk], acc, 0, 0, 0);
#pragma unroll
            for (int y = 0; y < SPG; y += 2) {
                const int x = kk * SPG + y;
                const __bf16 p0 = (__bf16)__builtin_amdgcn_exp2f(fmaf(sc[x], scale_log2, -m_run));
                const __bf16 p1 = (__bf16)__builtin_amdgcn_exp2f(fmaf(sc[x + 1], scale_log2, -m_run));
                pb[x >> 3][x & 7] = p0;
                pb[x >> 3][(x & 7) + 1] = p1;
                const bf16x2 pp = {p0, p1};
                l_acc[x >> 3] = __builtin_amdgcn_fdot2_f32_bf16(pp, one2, l_acc[x >> 3], false);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    // Phase 2: O^T += V^T P^T of the current tile (V^T fragments from vst)
    // while the VALU takes the row max of the next tile's scores.
    auto phase2 = [&](const unsigned char* vst, const floatx16& sn) -> float {
        constexpr int NX = DT * 2;
        constexpr int A = NX < 2 ? NX : 2;
        constexpr int VPG = 16 / NX;   // scores per group
        bf16x8 fr[A];
#pragma unroll
        for (int x = 0; x < A; ++x)
            fr[x] = *reinterpret_cast<const bf16x8*>(vst + voff(x % DT, x / DT));
        float mx = -INFINITY;
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int x = 0; x < NX; ++x) {
            const bf16x8 a = fr[x % A];
            if (x + A < NX)
                fr[x % A] = *reinterpret_cast<const bf16x8*>(vst + voff((x + A) % DT, (x + A) / DT));
            o[x % DT] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[x / DT], o[x % DT], 0, 0, 0);
#pragma unroll
            for (int y = 0; y < VPG; ++y) mx = fmaxf(mx, sn[x * VPG + y]);
            __builtin_amdgcn_sched_barrier(0);
        }
        return half_max(mx);
    };

    // Software pipeline over key tiles, one step per tile i < nt-1:
    //   wait for tile i+1 and barrier; refill the stage of tile i-1 (read by
    //   every wave before this barrier) with tile i+NS-1 (the split ring
    //   below waits and refills per half instead);
    //   phase 1: S^T(i+1) on the matrix core while the VALU turns S^T(i)
    //            into P^T(i);
    //   phase 2: O^T += V^T(i) P^T(i) while the VALU takes the row max of
    //            S^T(i+1);
    //   then the (rare) rescale for tile i+1.
    // Stages in use: i (V), i+1 (K), i+2 .. i+NS-1 in flight.
    static_assert(NS >= 3, "the ring needs the current, next and one loading stage");
    floatx16 s_cur = floatx16{};
    int pg_next = (!SPLIT_RING && FAST && NS - 1 < nt) ? tile_page(kt0 + NS - 1) : 0;
    // KIND 0: a step with a refill and the steady-state wait (no runtime
    // checks); 1: a step near the end; 2: the step that brings in the last
    // tile (which may be partial).
    auto step = [&](int i, auto stage_c, auto kind_c) {
        constexpr int STAGE = decltype(stage_c)::value;
        constexpr int KIND = decltype(kind_c)::value;
        constexpr int NXT = (STAGE + 1) % NS;
        constexpr int FREE = (STAGE + NS - 1) % NS;
        if constexpr (KIND == 0) {
            wait_vm((NS - 3) * NCH);
            barrier_raw();
            issue_tile(kt0 + i + NS - 1, std::integral_constant<int, FREE>{}, pg_next);
            if (FAST) {
                const int nx = i + NS < nt ? i + NS : nt - 1;   // clamped: no branch
                pg_next = tile_page(kt0 + nx);
            }
        } else {
            int behind = nt - 2 - i;            // tiles issued after tile i+1
            if (behind > NS - 3) behind = NS - 3;
            wait_vm(behind * NCH);
            barrier_raw();
            if (i + NS - 1 < nt) {
                issue_tile(kt0 + i + NS - 1, std::integral_constant<int, FREE>{}, pg_next);
                if (FAST && i + NS < nt) pg_next = tile_page(kt0 + i + NS);
            }
        }
        const unsigned char* kst = ring + NXT * RG_::kStageBytes;
        const unsigned char* vst = ring + STAGE * RG_::kStageBytes;   // V^T offsets include the K part

        floatx16 s_nxt = floatx16{};
        phase1(kst, s_cur, s_nxt);
        if constexpr (KIND == 2) {
            if (valid_last < kKeyTile) mask_tail(s_nxt);
        }
        const float mx = phase2(vst, s_nxt);
        update_max(mx);
        s_cur = s_nxt;
    };

    // The split ring (D = 128, three stages).  K(t) and V^T(t) still share
    // stage t % 3, but the K half is free a step before the V^T half (the
    // scores of tile t are taken in step t-1, its PV product in step t), so
    // step i refills them separately: K(i+3) into the K half of tile i's
    // stage and V^T(i+2) into the V^T half of tile i-1's.  Both then arrive
    // two steps before use (one for K when a tile's halves move together),
    // and step i waits only for what it reads -- K(i+1) and V^T(i), loaded
    // in step i-2 -- while the loads of step i-1 stay in flight.
    // KIND 0: both refills, no runtime checks; 1: a step near the end
    // (K(i+3) may not exist); 2: step nt-2, which takes the last tile's
    // scores and leaves only V^T(nt-1) in flight.
    int pg_k = 0, pg_v = 0;   // page ids of the next K and V^T tiles to load
    auto step_split = [&](int i, auto stage_c, auto kind_c) __attribute__((always_inline)) {
        constexpr int STAGE = decltype(stage_c)::value;
        constexpr int KIND = decltype(kind_c)::value;
        constexpr int NXT = (STAGE + 1) % NS;
        constexpr int FREE = (STAGE + NS - 1) % NS;
        using KPart = std::integral_constant<int, 0>;
        using VPart = std::integral_constant<int, 1>;
        // step i-1 loaded K(i+2) (when i+2 < nt, true but in the last step)
        // and V^T(i+1)
        wait_vm(KIND == 2 ? NCH - NK : NCH);
        barrier_raw();
        if constexpr (KIND != 2) {
            if (KIND == 0 || i + 3 < nt) issue_part(kt0 + i + 3, stage_c, pg_k, KPart{});
            issue_part(kt0 + i + 2, std::integral_constant<int, FREE>{}, pg_v, VPart{});
            if (FAST) {
                pg_v = pg_k;
                const int nx = i + 4 < nt ? i + 4 : nt - 1;   // clamped: no branch
                pg_k = tile_page(kt0 + nx);
            }
        }
        const unsigned char* kst = ring + NXT * RG_::kStageBytes;
        const unsigned char* vst = ring + STAGE * RG_::kStageBytes;
        floatx16 s_nxt = floatx16{};
        phase1(kst, s_cur, s_nxt);
        if constexpr (KIND == 2) {
            if (valid_last < kKeyTile) mask_tail(s_nxt);
        }
        const float mx = phase2(vst, s_nxt);
        update_max(mx);
        s_cur = s_nxt;
    };

    if constexpr (SPLIT_RING) if (nt > 0) {
        using C0 = std::integral_constant<int, 0>;
        using C1 = std::integral_constant<int, 1>;
        using C2 = std::integral_constant<int, 2>;
        using KPart = std::integral_constant<int, 0>;
        using VPart = std::integral_constant<int, 1>;
        const int p0 = FAST ? tile_page(kt0) : 0;
        const int p1 = (FAST && nt > 1) ? tile_page(kt0 + 1) : 0;
        const int p2 = (FAST && nt > 2) ? tile_page(kt0 + 2) : 0;
        // K(0), K(1), V^T(0), then Q.  The explicit wait is for K(0) alone
        // (it does not count on Q's loads, which a wave without valid rows
        // skips); Q is waited for where it is used, and as loads complete in
        // order that wait covers K(1) and V^T(0) too.
        issue_part(kt0, C0{}, p0, KPart{});
        if (nt > 1) issue_part(kt0 + 1, C1{}, p1, KPart{});
        issue_part(kt0, C0{}, p0, VPart{});
        load_q();
        wait_vm(nt > 1 ? NCH : NCH - NK);
        barrier_raw();
        s_mfmas(ring, s_cur);
        // the loads "step -1" makes: K(2) and V^T(1)
        if (nt > 2) issue_part(kt0 + 2, C2{}, p2, KPart{});
        if (nt > 1) issue_part(kt0 + 1, C1{}, p1, VPart{});
        if (FAST) {
            pg_v = p2;
            pg_k = nt > 3 ? tile_page(kt0 + 3) : p2;
        }
        if (nt == 1 && valid_last < kKeyTile) mask_tail(s_cur);
        m_run = tile_max(s_cur);
        thr_raw = (m_run + kRescaleSlack) / scale_log2;
        using Full = std::integral_constant<int, 0>;
        using Near = std::integral_constant<int, 1>;
        using Last = std::integral_constant<int, 2>;
        // steps 0 .. nt-4 make both refills; the tail steps check (one
        // runtime-checked kind keeps the register pressure of the loop down)
        const int n_full = nt - 3 > 0 ? nt - 3 : 0;
        int i0 = 0;
        for (; i0 + NS <= n_full; i0 += NS) {
            static_for<NS>([&](auto j) { step_split(i0 + j, j, Full{}); });
        }
        for (; i0 < nt - 2; i0 += NS) {
            static_for<NS>([&](auto j) {
                if (i0 + j < nt - 2) step_split(i0 + j, j, Near{});
            });
        }
        if (nt >= 2) {
            const int st = (nt - 2) % NS;
            static_for<NS>([&](auto j) {
                if (st == j) step_split(nt - 2, j, Last{});
            });
        }
        // V^T of the last tile
        wait_vm(0);
        barrier_raw();
    }
    if (nt > 0) {
        if constexpr (!SPLIT_RING) {
            int pg0[NS - 1];   // page ids of the first tiles, all requested before any load
            static_for<NS - 1>([&](auto j) { pg0[j] = (FAST && j < nt) ? tile_page(kt0 + j) : 0; });
            static_for<NS - 1>([&](auto j) {
                if (j < nt) issue_tile(kt0 + j, j, pg0[j]);
            });
            load_q();
            wait_vm((nt - 1 < NS - 2 ? nt - 1 : NS - 2) * NCH);
            barrier_raw();
            s_mfmas(ring, s_cur);
            if (nt == 1 && valid_last < kKeyTile) mask_tail(s_cur);
            m_run = tile_max(s_cur);
            thr_raw = (m_run + kRescaleSlack) / scale_log2;
            using Full = std::integral_constant<int, 0>;
            using Near = std::integral_constant<int, 1>;
            using Last = std::integral_constant<int, 2>;
            // steps 0 .. n_full-1 refill the ring (and, as NS >= 3, are not the last)
            const int n_full = nt - NS + 1 > 0 ? nt - NS + 1 : 0;
            int i0 = 0;
            for (; i0 + NS <= n_full; i0 += NS) {
                static_for<NS>([&](auto j) { step(i0 + j, j, Full{}); });
            }
            for (; i0 < nt - 2; i0 += NS) {
                static_for<NS>([&](auto j) {
                    if (i0 + j < nt - 2) step(i0 + j, j, Near{});
                });
            }
            // the step that brings in the last tile (which may be partial)
            if (nt >= 2) {
                const int st2 = (nt - 2) % NS;
                static_for<NS>([&](auto j) {
                    if (st2 == j) step(nt - 2, j, Last{});
                });
            }
        }
        // last tile: P^T, then its PV product
        softmax_p(s_cur);
        const int last_stage = (nt - 1) % NS;
        unsigned char* slast = ring + last_stage * RG_::kStageBytes;
        if (valid_last < kKeyTile) {
            // V^T columns of keys past ke may hold anything (even NaN); zero
            // them so their 0-weight products stay 0.  One 16-byte chunk (8
            // keys of one d) per thread and pass.
            unsigned char* vlds = slast + RG_::kKCh * 16;
#pragma unroll 1
            for (int e = tid; e < D * (kKeyTile / 8); e += kAttnThreads) {
                const int d = e >> 2, kc = e & 3;
                const int first = valid_last - kc * 8;   // keys >= first are past ke
                if (first >= 8) continue;
                uint4* p = reinterpret_cast<uint4*>(vlds + (d * kKeyTile + ((kc ^ ((d >> 2) & 3)) * 8)) * 2);
                if (first <= 0) {
                    *p = make_uint4(0, 0, 0, 0);
                } else {
                    const uint4 v = *p;
                    uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                    for (int k = 0; k < 8; ++k)
                        if (k >= first) w[k >> 1] &= (k & 1) ? 0x0000ffffu : 0xffff0000u;
                    *p = make_uint4(w[0], w[1], w[2], w[3]);
                }
            }
            barrier_raw();
        }
        pv_mfmas(slast);
    }

    if (page_err && tid == 0) record_error(pv.hdr, b, FB_DERR_PAGE);
    float l_part = l_acc[0] + l_acc[1];
    const float l = l_part + __shfl_xor(l_part, 32, 64);
    const float inv_l = 1.0f / l;
    if (slot < 0) {
        if (!row_ok) return;
        uint16_t* orow = out + q_off;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
            for (int grp = 0; grp < 4; ++grp) {
                const int d0 = dt * 32 + grp * 8 + h * 4;
                __bf16 v4[4];
#pragma unroll
                for (int x = 0; x < 4; ++x) v4[x] = (__bf16)(o[dt][grp * 4 + x] * inv_l);
                *reinterpret_cast<uint2*>(orow + d0) = *reinterpret_cast<const uint2*>(v4);
            }
        }
    } else {
        float* po = ws.part_o + ((size_t)slot * kRowsPerWg + r_local) * D;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
            for (int grp = 0; grp < 4; ++grp) {
                const int d0 = dt * 32 + grp * 8 + h * 4;
                float4 v4 = make_float4(o[dt][grp * 4 + 0] * inv_l, o[dt][grp * 4 + 1] * inv_l,
                                        o[dt][grp * 4 + 2] * inv_l, o[dt][grp * 4 + 3] * inv_l);
                *reinterpret_cast<float4*>(po + d0) = v4;
            }
        }
        if (h == 0) ws.part_lse[(size_t)slot * kRowsPerWg + r_local] = m_run + __log2f(l);
    }
}

// ------------------------------------------------------------ combine -----
// Four consecutive output elements of one row.
template <typename T>
__device__ inline void store_out4(T* p, const float4& v);
template <>
__device__ inline void store_out4<uint16_t>(uint16_t* p, const float4& v) {
    __bf16 x[4] = {(__bf16)v.x, (__bf16)v.y, (__bf16)v.z, (__bf16)v.w};
    *reinterpret_cast<uint2*>(p) = *reinterpret_cast<const uint2*>(x);
}
template <>
__device__ inline void store_out4<float>(float* p, const float4& v) {
    *reinterpret_cast<float4*>(p) = v;
}

// Each split unit's rows are merged by kCombineParts workgroups of
// kCombineRows rows (workgroup b takes entry b / kCombineParts of the plan's
// list of split units, so the grid covers only units that can be split): a row's per-split log-sum-exp weights go to LDS once,
// then every thread merges 16-byte columns of its rows, up to eight splits'
// loads in flight at a time.
constexpr int kCombineRows = 32;
constexpr int kCombineParts = kRowsPerWg / kCombineRows;

template <typename T>
__global__ void __launch_bounds__(kAttnThreads)
combine_kernel(PackView pv, AttnWs ws, T* __restrict__ out, int Hq, int Hkv,
               int g, int bl, int RG, int D, PlanBounds bounds) {
    __shared__ float wgt[kMaxSplits][kCombineRows];
    __shared__ float inv_den[kCombineRows];
    const int su = blockIdx.x / kCombineParts;
    const int part = blockIdx.x % kCombineParts;
    if (su >= ws.counts[kCSplit]) return;
    // the plan's record of this split unit: no further lookups before the loads
    const int4 rec = ws.split[su];
    const int u = rec.x;
    const int ns = rec.y;   // 2 .. kMaxSplits (plan)
    if (ns <= 1) return;
    const int slot0 = rec.z;
    const int row0 = rec.w;
    if ((unsigned)u >= (unsigned)bounds.unit_cap || ns > kMaxSplits || slot0 < 0 ||
        slot0 > bounds.slot_cap - ns || row0 < 0 || row0 > bounds.row_cap - bl) {
        if (threadIdx.x == 0) record_error(pv.hdr, 0, FB_DERR_PLAN);
        return;
    }
    const int rg = u % RG;
    const int c = (u / RG) % Hkv;
    const int rbase = part * kCombineRows;
    const int nrows = min(kCombineRows, bl * g - rg * kRowsPerWg - rbase);
    if (nrows <= 0) return;
    const int per_row = D / 4;
    const int n_el = nrows * per_row;
    const size_t stride = (size_t)kRowsPerWg * D;   // one split's partial O
    auto src_of = [&](int e) {
        return ws.part_o + ((size_t)slot0 * kRowsPerWg + rbase + e / per_row) * D +
               (e % per_row) * 4;
    };
    typedef float f32x4 __attribute__((ext_vector_type(4)));
    // A row's split weights exp2(lse_k - max) and 1/sum: its log-sum-exps
    // are loaded eight at a time (one round trip for up to eight splits) and
    // kept in LDS until the maximum is known.
    auto weights = [&]() {
        if (threadIdx.x < nrows) {
            const float* lse = ws.part_lse + (size_t)slot0 * kRowsPerWg + rbase + threadIdx.x;
            float mx = -INFINITY;
            for (int k0 = 0; k0 < ns; k0 += 8) {
                float l[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) l[j] = lse[(size_t)min(k0 + j, ns - 1) * kRowsPerWg];
#pragma unroll
                for (int j = 0; j < 8; ++j) mx = fmaxf(mx, l[j]);   // repeats do not move it
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    if (k0 + j < ns) wgt[k0 + j][threadIdx.x] = l[j];
            }
            float den = 0.f;
            for (int k = 0; k < ns; ++k) {
                const float w = __builtin_amdgcn_exp2f(wgt[k][threadIdx.x] - mx);
                wgt[k][threadIdx.x] = w;
                den += w;
            }
            inv_den[threadIdx.x] = 1.0f / den;
        }
        __syncthreads();
    };
    auto store = [&](int e, const float4& acc) {
        const int rr = e / per_row;
        const int d0 = (e % per_row) * 4;
        const float id = inv_den[rr];
        const int r = rg * kRowsPerWg + rbase + rr;
        const int pos_local = r / g, hg = r % g;
        T* dst = out + ((size_t)(row0 + pos_local) * Hq + c * g + hg) * D + d0;
        store_out4<T>(dst, make_float4(acc.x * id, acc.y * id, acc.z * id, acc.w * id));
    };
    auto add = [](float4& acc, float w, const f32x4& v) {
        acc.x += w * v[0];
        acc.y += w * v[1];
        acc.z += w * v[2];
        acc.w += w * v[3];
    };
    // Up to kFastSplits splits (the plan's usual few pieces): every load of
    // the thread's column groups (at most kMaxGroups) is issued before the
    // weights are computed, so the workgroup waits for one round trip.
    constexpr int kFastSplits = 4;
    constexpr int kMaxGroups = kCombineRows * kMaxHeadDim / 4 / kAttnThreads;
    const int n_grp = (n_el + kAttnThreads - 1) / kAttnThreads;   // workgroup-uniform
    if (ns <= kFastSplits && n_grp <= kMaxGroups) {
        f32x4 v[kMaxGroups][kFastSplits];
#pragma unroll
        for (int m = 0; m < kMaxGroups; ++m) {
            if (m < n_grp) {
                const float* src = src_of(min((int)threadIdx.x + m * kAttnThreads, n_el - 1));
#pragma unroll
                for (int k = 0; k < kFastSplits; ++k)   // past the last split: reload it, unused
                    v[m][k] = *reinterpret_cast<const f32x4*>(src + (size_t)min(k, ns - 1) * stride);
            }
        }
        weights();
#pragma unroll
        for (int m = 0; m < kMaxGroups; ++m) {
            const int e = (int)threadIdx.x + m * kAttnThreads;
            if (m < n_grp && e < n_el) {
                const int rr = e / per_row;
                float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
                for (int k = 0; k < kFastSplits; ++k)
                    if (k < ns) add(acc, wgt[k][rr], v[m][k]);
                store(e, acc);
            }
        }
        return;
    }
    // More splits: a thread's first column group has its loads (up to eight)
    // issued before the weights are ready; then eight at a time per group.
    constexpr int kInFlight = 8;
    f32x4 first[kInFlight];
    {
        const float* src = src_of(min((int)threadIdx.x, n_el - 1));
#pragma unroll
        for (int j = 0; j < kInFlight; ++j)   // past the last split: reload it, unused
            first[j] = *reinterpret_cast<const f32x4*>(src + (size_t)min(j, ns - 1) * stride);
#pragma unroll
        for (int j = 0; j < kInFlight; ++j) asm volatile("" :: "v"(first[j]));
    }
    weights();
    for (int e = threadIdx.x; e < n_el; e += kAttnThreads) {
        const int rr = e / per_row;
        const float* src = src_of(e);
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int k0 = 0; k0 < ns; k0 += kInFlight) {
            f32x4 v[kInFlight];
            if (k0 == 0 && e == (int)threadIdx.x) {
#pragma unroll
                for (int j = 0; j < kInFlight; ++j) v[j] = first[j];
            } else {
#pragma unroll
                for (int j = 0; j < kInFlight; ++j)
                    v[j] = *reinterpret_cast<const f32x4*>(
                        src + (size_t)min(k0 + j, ns - 1) * stride);
            }
#pragma unroll
            for (int j = 0; j < kInFlight; ++j)
                if (k0 + j < ns) add(acc, wgt[k0 + j][rr], v[j]);
        }
        store(e, acc);
    }
}

// ---------------------------------------------------------------- fp32 ----
// One workgroup per (tile, query head); each wave walks its rows with an
// online softmax over 64-key chunks, one key per lane.
constexpr int kF32MaxD = 256;

__global__ void __launch_bounds__(kAttnThreads)
attn_f32_kernel(const float* __restrict__ q, const float* __restrict__ k_cache,
                const float* __restrict__ v_cache, const int32_t* __restrict__ page_table,
                PackView pv, float* __restrict__ out, int Hq, int Hkv, int D, int bl,
                int ps, int max_pages, int num_pages, float sm_scale) {
    const int t = blockIdx.x;
    const int hq = blockIdx.y;
    if (t >= pv.hdr[kHdrTiles]) return;
    const int32_t* tile = pv.tiles + (size_t)t * kTileInts;
    const int b = tile[kTB];
    const int row0 = tile[kTRow0];
    const int kv_len = tile[kTKvLen];
    const int c = hq / (Hq / Hkv);
    const int32_t* pt = page_table + (size_t)b * max_pages;
    // Every page the tile reads must be valid, else the tile is skipped.
    __shared__ int bad_page;
    if (threadIdx.x == 0) bad_page = 0;
    __syncthreads();
    if ((long long)kv_len > (long long)max_pages * ps) {
        if (threadIdx.x == 0) bad_page = 1;
    } else {
        for (int p = threadIdx.x; p * ps < kv_len; p += kAttnThreads) {
            const int id = pt[p];
            if (id < 0 || id >= num_pages) bad_page = 1;
        }
    }
    __syncthreads();
    if (bad_page) {
        if (threadIdx.x == 0) record_error(pv.hdr, b, FB_DERR_PAGE);
        return;
    }
    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    constexpr int kAcc = kF32MaxD / 64;

    for (int i = wave; i < bl; i += kAttnThreads / 64) {
        const float* qrow = q + ((size_t)(row0 + i) * Hq + hq) * D;
        float m = -INFINITY, l = 0.f;
        float acc[kAcc];
#pragma unroll
        for (int j = 0; j < kAcc; ++j) acc[j] = 0.f;
        for (int k0 = 0; k0 < kv_len; k0 += 64) {
            const int key = k0 + lane;
            float s = -INFINITY;
            if (key < kv_len) {
                const int page = pt[key / ps];
                const float* krow = k_cache + (((size_t)page * Hkv + c) * ps + key % ps) * D;
                float dot = 0.f;
                for (int d = 0; d < D; ++d) dot = fmaf(qrow[d], krow[d], dot);
                s = dot * sm_scale;
            }
            float cm = s;
#pragma unroll
            for (int off = 32; off > 0; off >>= 1) cm = fmaxf(cm, __shfl_xor(cm, off, 64));
            const float m_new = fmaxf(m, cm);
            const float alpha = expf(m - m_new);
            const float p = key < kv_len ? expf(s - m_new) : 0.f;
            float ps_sum = p;
#pragma unroll
            for (int off = 32; off > 0; off >>= 1) ps_sum += __shfl_xor(ps_sum, off, 64);
            l = l * alpha + ps_sum;
#pragma unroll
            for (int j = 0; j < kAcc; ++j) acc[j] *= alpha;
            const int nk = min(64, kv_len - k0);
            for (int jj = 0; jj < nk; ++jj) {
                const float pj = __shfl(p, jj, 64);
                const int kk = k0 + jj;
                const int page = pt[kk / ps];
                const float* vcol = v_cache + ((size_t)page * Hkv + c) * D * ps + kk % ps;
#pragma unroll
                for (int j = 0; j < kAcc; ++j) {
                    const int d = lane + 64 * j;
                    if (d < D) acc[j] = fmaf(pj, vcol[(size_t)d * ps], acc[j]);
                }
            }
            m = m_new;
        }
        float* orow = out + ((size_t)(row0 + i) * Hq + hq) * D;
#pragma unroll
        for (int j = 0; j < kAcc; ++j) {
            const int d = lane + 64 * j;
            if (d < D) orow[d] = acc[j] / l;
        }
    }
}

}  // namespace

AttnPlanSizes attention_sizes(const fb_pack* pack, const fb_attn_shape* sh,
                              int cu_count) {
    AttnPlanSizes z{};
    const int g = sh->Hq / sh->Hkv;
    z.rows_per_unit = pack->bl * g;
    z.row_groups = (z.rows_per_unit + kRowsPerWg - 1) / kRowsPerWg;
    z.unit_cap = pack->tile_cap * sh->Hkv * z.row_groups;
    // One item per workgroup the chip holds at once (kWgsPerCu per CU): more
    // splits cost more in partial writes, the merge and per-item start-up
    // than they win in balance (measured: 8 per CU was 2-25% slower).
    z.target_items = kWgsPerCu * (cu_count > 0 ? cu_count : 256);
    z.item_cap = z.unit_cap + z.target_items;
    z.slot_cap = 2 * z.target_items;
    z.split_cap = z.target_items;   // a split unit holds at least two of the slots
    const size_t D = sh->head_dim;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        size_t at = off;
        off += (bytes + 255) & ~(size_t)255;
        return at;
    };
    z.off_items = take((size_t)z.item_cap * kIItemInts * sizeof(int32_t));
    z.off_units = take((size_t)z.unit_cap * 2 * sizeof(int32_t));
    z.off_counts = take(4 * sizeof(int32_t));
    z.off_split = take((size_t)z.split_cap * sizeof(int4));
    if (sh->dtype == FB_BF16) {
        z.off_part_o = take((size_t)z.slot_cap * kRowsPerWg * D * sizeof(float));
        z.off_part_lse = take((size_t)z.slot_cap * kRowsPerWg * sizeof(float));
    } else {
        z.off_part_o = z.off_part_lse = off;
    }
    z.total = off;
    return z;
}

namespace {

AttnWs ws_view(void* wsp, const AttnPlanSizes& z) {
    char* base = static_cast<char*>(wsp);
    return AttnWs{reinterpret_cast<int32_t*>(base + z.off_items),
                  reinterpret_cast<int32_t*>(base + z.off_units),
                  reinterpret_cast<int32_t*>(base + z.off_counts),
                  reinterpret_cast<int4*>(base + z.off_split),
                  reinterpret_cast<float*>(base + z.off_part_o),
                  reinterpret_cast<float*>(base + z.off_part_lse)};
}

}  // namespace

hipError_t launch_attention_plan(const fb_pack* pack, const fb_attn_shape* sh, void* wsp,
                                 const AttnPlanSizes& z, hipStream_t stream) {
    if (sh->dtype == FB_F32) return hipSuccess;   // the fp32 path has no plan
    const int fixed_chunk = sh->kv_split > 0 ? sh->kv_split / kKeyTile : 0;
    const long long max_keys = (long long)sh->max_pages * sh->page_size;
    hipLaunchKernelGGL(plan_kernel, dim3(1), dim3(kPlanThreads), 0, stream, pack_view(pack),
                       ws_view(wsp, z), sh->Hkv, z.row_groups, z.item_cap, z.slot_cap,
                       z.split_cap, z.target_items, fixed_chunk, max_keys);
    return hipGetLastError();
}

hipError_t launch_attention(const void* q, const void* k_cache,
                            const void* v_cache, const int32_t* page_table,
                            const fb_pack* pack, const fb_attn_shape* sh,
                            void* out, void* wsp, const AttnPlanSizes& z,
                            hipStream_t stream, bool planned) {
    PackView pv = pack_view(pack);
    const int g = sh->Hq / sh->Hkv;
    const float scale = sh->sm_scale > 0.f ? sh->sm_scale
                                           : 1.0f / sqrtf((float)sh->head_dim);
    if (sh->dtype == FB_F32) {
        hipLaunchKernelGGL(attn_f32_kernel, dim3(pack->tile_cap, sh->Hq),
                           dim3(kAttnThreads), 0, stream,
                           static_cast<const float*>(q),
                           static_cast<const float*>(k_cache),
                           static_cast<const float*>(v_cache), page_table, pv,
                           static_cast<float*>(out), sh->Hq, sh->Hkv,
                           sh->head_dim, pack->bl, sh->page_size, sh->max_pages,
                           sh->num_pages, scale);
        return hipGetLastError();
    }
    const AttnWs ws = ws_view(wsp, z);
    const PlanBounds bounds{pack->B, pack->row_cap, z.unit_cap, z.slot_cap,
                            (long long)sh->max_pages * sh->page_size};
    hipError_t e = planned ? hipSuccess : launch_attention_plan(pack, sh, wsp, z, stream);
    if (e != hipSuccess) return e;
    int shift = 0;
    while ((1 << shift) < sh->page_size) ++shift;
    const float scale_log2 = scale * kLog2e;
    const uint16_t* qb = static_cast<const uint16_t*>(q);
    const uint16_t* kc = static_cast<const uint16_t*>(k_cache);
    const uint16_t* vc = static_cast<const uint16_t*>(v_cache);
    uint16_t* ob = static_cast<uint16_t*>(out);
    const bool fast = sh->page_size >= kKeyTile;
    auto launch = [&](auto kernel) {
        hipLaunchKernelGGL(kernel, dim3(z.item_cap), dim3(kAttnThreads), 0, stream, qb, kc, vc,
                           page_table, pv, ws, ob, sh->Hq, sh->Hkv, g, pack->bl, z.row_groups,
                           sh->page_size, shift, sh->max_pages, sh->num_pages, scale_log2, bounds);
    };
    switch (sh->head_dim) {
        case 32:
            if (fast) launch(attn_bf16_kernel<32, true>);
            else launch(attn_bf16_kernel<32, false>);
            break;
        case 64:
            if (fast) launch(attn_bf16_kernel<64, true>);
            else launch(attn_bf16_kernel<64, false>);
            break;
        default:
            if (fast) launch(attn_bf16_kernel<128, true>);
            else launch(attn_bf16_kernel<128, false>);
            break;
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(combine_kernel<uint16_t>, dim3(z.split_cap * kCombineParts), dim3(kAttnThreads),
                       0, stream, pv, ws, ob, sh->Hq, sh->Hkv, g, pack->bl,
                       z.row_groups, sh->head_dim, bounds);
    return hipGetLastError();
}

}  // namespace fb
