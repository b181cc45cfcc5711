// LM head with the vocabulary reduction as its epilogue: the last layer of
// the forward f_theta of Alg. 1, Z = H W^T, reduced per row to the symbols of
// Eq. 1 (max, lowest index of the max, sum of exponentials) without the
// logits ever reaching memory.
//
// lmhead_kernel   one workgroup of 8 waves per (256-row token tile, vocabulary
//                 partition).  It walks the partition's 256-id vocabulary
//                 tiles; for each, Z^T tile = W_tile . H_tile^T on
//                 v_mfma_f32_32x32x16_bf16 over K = D in 64-wide stages
//                 (double-buffered LDS, filled by direct global->LDS loads
//                 with a scalar base and a per-lane offset fixed for the
//                 whole kernel), then folds the tile into a running
//                 (max, index, scaled sum) per token.  Wave (wv, wt) owns
//                 vocabulary rows wv*128.. and tokens wt*64.. of the tile.
//                 With Z^T in the accumulators each lane holds one token and
//                 16 vocabulary ids per MFMA tile, so the per-token reduction
//                 is mostly in-lane.
// lm_merge_kernel one wave per row: merges the row's partition partials in a
//                 fixed order into the first partial of the update workspace
//                 (the rest are set empty), the input of the update kernel.
#include <climits>
#include <map>
#include <mutex>
#include <tuple>

#include "internal.h"
#include "top.h"

namespace fb {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kLmThreads = 512;                   // 8 waves
constexpr int kTileV = 256;                       // vocabulary ids per tile
constexpr int kTileT = 256;                       // tokens per tile
constexpr int kBK = 64;                           // K per stage
constexpr int kRowBytes = kBK * 2;                // 128 B: one row of a stage
constexpr int kHalfBytes = kTileV * kRowBytes;    // 32 KB: W part of a stage
constexpr int kStageBytes = 2 * kHalfBytes;       // W part, then H part
constexpr int kStages = 2;
constexpr int kMergeThreads = 256;

// LDS reads drained, then a workgroup barrier.  The wait is the builtin, not
// inline asm, so the compiler knows the reads issued before it are complete
// and does not wait for them again after the barrier (behind newer reads).
__device__ inline void lds_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0); vmcnt and expcnt not waited
    asm volatile("s_barrier" ::: "memory");
}
__device__ inline void wait_vm0() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Vocabulary partitions for n_lt token tiles.  One workgroup runs per CU at
// a time, so the kernel takes about (rounds of workgroups over the CUs) x
// (tiles of the largest partition + a workgroup's fixed start and end,
// about 1/8 of a tile); the partition count P minimizes that (the smallest
// such P), with P <= kMaxParts.  Host and device evaluate the same integer
// expression, so both sides agree on P.
constexpr int kMaxParts = 1024;
__host__ __device__ inline long long lm_cost(int n_lt, int nv, int cu, int P) {
    return (long long)((n_lt * P + cu - 1) / cu) * (((nv + P - 1) / P) * 8 + 1);
}
inline int lm_parts_host(int n_lt, int nv, int cu) {
    const int pmax = nv < kMaxParts ? nv : kMaxParts;
    int best = 1;
    long long best_c = lm_cost(n_lt, nv, cu, 1);
    for (int P = 2; P <= pmax; ++P) {
        const long long c = lm_cost(n_lt, nv, cu, P);
        if (c < best_c) best_c = c, best = P;
    }
    return best;
}
// the same choice by one wave (lane i tries P = i + 1, i + 65, ...); every
// lane returns it
__device__ inline int lm_parts_dev(int n_lt, int nv, int cu) {
    const int lane = threadIdx.x & 63;
    const int pmax = nv < kMaxParts ? nv : kMaxParts;
    long long key = LLONG_MAX;   // cost * 2048 + P: the minimum is the smallest P of least cost
    for (int P = lane + 1; P <= pmax; P += 64) {
        const long long k = lm_cost(n_lt, nv, cu, P) * 2048 + P;
        key = k < key ? k : key;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const long long o = __shfl_xor(key, off, 64);
        key = o < key ? o : key;
    }
    return __builtin_amdgcn_readfirstlane((int)(key & 2047));   // uniform: keeps it scalar
}

__global__ void __launch_bounds__(kLmThreads, 1)
lmhead_kernel(const uint16_t* __restrict__ H, const uint16_t* __restrict__ W, int D, int V,
              int row_cap, int padded, int n_vtiles, int cu, PackView pv,
              float4* __restrict__ part) {
    __shared__ __attribute__((aligned(16))) unsigned char lds[kStages * kStageBytes];
    __shared__ Top s_top[kTileT];
    __shared__ int s_live;

    const int tid = threadIdx.x;
    // token tiles that can hold live rows (ragged rows are the first
    // header-count rows; padded rows sit anywhere below row_cap), and the
    // partitions for them; block b is token tile b mod n_lt of partition
    // b / n_lt, and workgroup i takes blocks i, i + gridDim.x, ...
    const int n_lt = ((padded ? row_cap : pv.hdr[kHdrRows]) + kTileT - 1) / kTileT;
    const int P = n_lt > 0 ? lm_parts_dev(n_lt, n_vtiles, cu) : 0;
    for (int blk = blockIdx.x; blk < n_lt * P; blk += gridDim.x) {
    const int rt = blk % n_lt;
    const int pidx = blk / n_lt;
    const int row0 = rt * kTileT;
    // partitions of floor or ceil(n_vtiles / P) tiles
    const int vt0 = (int)((long long)pidx * n_vtiles / P);
    const int vt1 = (int)((long long)(pidx + 1) * n_vtiles / P);
    if (vt0 >= vt1) continue;
    // skip token tiles without a live row (the first barrier also keeps the
    // previous block's last reads of s_live and s_top before these writes)
    __syncthreads();
    if (tid == 0) s_live = 0;
    __syncthreads();
    if (tid < kTileT && row0 + tid < row_cap && pv.row_req[row0 + tid] >= 0) s_live = 1;
    __syncthreads();
    if (!s_live) continue;

    const int wave = tid >> 6;
    const int lane = tid & 63;
    const int n = lane & 31;
    const int h = lane >> 5;
    const int wv = wave & 1;          // vocabulary half of the tile
    const int wt = wave >> 1;         // token quarter of the tile

    // ---- DMA assignment: wave w fills W rows [32w, 32w+32) and H rows
    // [32w, 32w+32) of each stage, 8 rows (1 KB) per instruction; lane L
    // writes LDS chunk L%8 of row r = 32w + 8j + L/8, which holds logical K
    // chunk (L%8) ^ ((r/2)%8).  With 128-byte rows, 16 consecutive rows then
    // cover all 16 bank groups of 16 bytes at any logical chunk, so the
    // operand reads (16 lanes = 16 rows per access) are conflict-free.
    const int lrow = lane >> 3;
    uint32_t h_off[4];
    int w_row[4], w_chunk[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int r = wave * 32 + j * 8 + lrow;
        const int c = (lane & 7) ^ ((r >> 1) & 7);
        const int tr = min(row0 + r, row_cap - 1);
        h_off[j] = (uint32_t)(((size_t)tr * D + c * 8) * 2);
        w_row[j] = r;
        w_chunk[j] = c;
    }
    uint32_t m0_w[4], m0_h[4];
    const uint32_t lds_base = (uint32_t)(uintptr_t)&lds[0];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        m0_w[j] = __builtin_amdgcn_readfirstlane(lds_base + (wave * 4 + j) * 1024);
        m0_h[j] = __builtin_amdgcn_readfirstlane(lds_base + kHalfBytes + (wave * 4 + j) * 1024);
    }
    uint32_t w_off[4];
    auto set_vtile = [&](int vt) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int vr = min(vt * kTileV + w_row[j], V - 1);
            w_off[j] = (uint32_t)(((size_t)vr * D + w_chunk[j] * 8) * 2);
        }
    };
    const int KS = D / kBK;
    // issue K step ks of the current DMA tile into `stage`
    auto issue = [&](int ks, int stage) {
        const int k0 = ks * kBK;
        const uint16_t* wb = W + k0;
        const uint16_t* hb = H + k0;
        const uint32_t so = stage * kStageBytes;
#pragma unroll
        for (int j = 0; j < 4; ++j)
            asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
                         :: "s"(m0_w[j] + so), "v"(w_off[j]), "s"(wb) : "memory");
#pragma unroll
        for (int j = 0; j < 4; ++j)
            asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
                         :: "s"(m0_h[j] + so), "v"(h_off[j]), "s"(hb) : "memory");
    };

    // operand reads: row r of a stage part, logical chunk 2kk + h, stored at
    // chunk (2kk + h) ^ ((r/2)%8); every row read here has (r/2)%8 == (n/2)%8
    const uint32_t swz = (uint32_t)((h ^ ((n >> 1) & 7)) * 16);
    const uint32_t a_row = (uint32_t)((wv * 128 + n) * kRowBytes);
    const uint32_t b_row = (uint32_t)(kHalfBytes + (wt * 64 + n) * kRowBytes);

    floatx16 acc[4][2];
#pragma unroll
    for (int vi = 0; vi < 4; ++vi)
#pragma unroll
        for (int ti = 0; ti < 2; ++ti) acc[vi][ti] = floatx16{};
    Top top[2] = {top_empty(), top_empty()};

    // Operand fragments of one k step (16 of K): four of W, two of H, in two
    // register sets so the reads of k step kk + 1 overlap the eight MFMAs of
    // k step kk.
    constexpr int KK = kBK / 16;
    bf16x8 a[2][4], b[2][2];
    auto read = [&](int stage, int kk, int buf) {
        const unsigned char* st = lds + stage * kStageBytes;
        const uint32_t ko = swz ^ (uint32_t)(kk << 5);
#pragma unroll
        for (int vi = 0; vi < 4; ++vi)
            a[buf][vi] = *reinterpret_cast<const bf16x8*>(st + a_row + vi * 32 * kRowBytes + ko);
#pragma unroll
        for (int ti = 0; ti < 2; ++ti)
            b[buf][ti] = *reinterpret_cast<const bf16x8*>(st + b_row + ti * 32 * kRowBytes + ko);
    };
    // MFMAs x0 .. x1-1 of a k step (x = 2 vi + ti)
    auto mfmas = [&](int buf, int x0 = 0, int x1 = 8) {
#pragma unroll
        for (int x = x0; x < x1; ++x)
            acc[x >> 1][x & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                a[buf][x >> 1], b[buf][x & 1], acc[x >> 1][x & 1], 0, 0, 0);
    };

    // fold the finished tile vt into the running tops; lane value (vi, r)
    // is vocabulary id vt*256 + wv*128 + vi*32 + (r/4)*8 + h*4 + r%4 --
    // increasing in (vi, r), so the first maximum in that order is the
    // lowest id.
    auto fold = [&](int vt, auto partial) {
        const int vbase = vt * kTileV + wv * 128 + h * 4;
#pragma unroll
        for (int ti = 0; ti < 2; ++ti) {
            float f[64];
#pragma unroll
            for (int vi = 0; vi < 4; ++vi)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int v = vbase + vi * 32 + (r >> 2) * 8 + (r & 3);
                    f[vi * 16 + r] = (!partial || v < V) ? acc[vi][ti][r] : -INFINITY;
                }
            // maxima of the four 16-id groups (one MFMA tile each), then the
            // tile maximum
            float g[4];
#pragma unroll
            for (int vi = 0; vi < 4; ++vi) {
                g[vi] = f[vi * 16];
#pragma unroll
                for (int r = 1; r < 16; ++r) g[vi] = fmaxf(g[vi], f[vi * 16 + r]);
            }
            const float vmax = fmaxf(fmaxf(g[0], g[1]), fmaxf(g[2], g[3]));
            Top& t = top[ti];
            if (vmax > t.m) {
#pragma clang fp contract(off)
                // lowest position of the maximum: the first group that holds
                // it (every earlier group is below it), then the first
                // position inside that group
                int gs = 3;
#pragma unroll
                for (int vi = 2; vi >= 0; --vi)
                    if (g[vi] == vmax) gs = vi;
                // the group's values by bit masks (v_bfi: (m & a) | (~m & b)),
                // so the selection stays free of branches
                const uint32_t m1 = gs >= 1 ? ~0u : 0u, m2 = gs >= 2 ? ~0u : 0u,
                               m3 = gs >= 3 ? ~0u : 0u;
                auto bfi = [](uint32_t m, float a, float b) -> float {
                    uint32_t r;
                    asm("v_bfi_b32 %0, %1, %2, %3"
                        : "=v"(r) : "v"(m), "v"(__float_as_uint(a)), "v"(__float_as_uint(b)));
                    return __uint_as_float(r);
                };
                int r0 = 15;
#pragma unroll
                for (int r = 15; r >= 0; --r) {
                    const float x = bfi(m3, f[48 + r], bfi(m2, f[32 + r], bfi(m1, f[16 + r], f[r])));
                    if (x == vmax) r0 = r;
                }
                const int j0 = gs * 16 + r0;
                const float nmL = scaled_ref(vmax);
                t.s *= __builtin_amdgcn_exp2f(t.mL - nmL);
                t.m = vmax;
                t.mL = nmL;
                t.idx = vbase + (j0 >> 4) * 32 + ((j0 & 15) >> 2) * 8 + (j0 & 3);
            }
            if (t.m != -INFINITY) {
                float e[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int j = 0; j < 64; ++j)
                    e[j & 3] += __builtin_amdgcn_exp2f(fmaf(f[j], kLog2e, -t.mL));
                t.s += (e[0] + e[1]) + (e[2] + e[3]);
            }
        }
#pragma unroll
        for (int vi = 0; vi < 4; ++vi)
#pragma unroll
            for (int ti = 0; ti < 2; ++ti) acc[vi][ti] = floatx16{};
    };

    // ---- main loop over the partition's stages k (vocabulary tile
    // vt0 + k / KS, K step k % KS) in two LDS slots; stage k + 1 is loaded
    // while stage k is computed.  The last k step's fragments of a stage are
    // read before the barrier that hands its slot back to the loader, and
    // their MFMAs issue right after it, so the next stage's first reads
    // overlap eight MFMAs instead of stalling the matrix core.
    const int T = (vt1 - vt0) * KS;
    int ld_vt = vt0, ld_ks = 0;      // next stage to load
    set_vtile(vt0);
    auto issue_next = [&](int k) {
        issue(ld_ks, k & 1);
        if (++ld_ks == KS) {
            ld_ks = 0;
            if (++ld_vt < vt1) set_vtile(ld_vt);
        }
    };
    issue_next(0);
    wait_vm0();
    lds_barrier();
    if (T > 1) issue_next(1);
    read(0, 0, 0);
    // k steps 0 .. KK-2 of stage k: reads of step kk + 1 under the MFMAs of kk
    auto body = [&](int slot) {
#pragma unroll
        for (int kk = 0; kk + 1 < KK; ++kk) {
            read(slot, kk + 1, (kk + 1) & 1);
            __builtin_amdgcn_sched_barrier(0);
            mfmas(kk & 1);
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    int k = 0;
    for (int vt = vt0; vt < vt1; ++vt) {
        for (int ks = 0; ks + 1 < KS; ++ks, ++k) {
            const int slot = k & 1;
            body(slot);
            wait_vm0();
            lds_barrier();         // stage k + 1 landed; slot k & 1 is free
            read(slot ^ 1, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
            mfmas((KK - 1) & 1, 0, 2);
            __builtin_amdgcn_sched_barrier(0);
            if (k + 2 < T) issue_next(k + 2);   // under the MFMAs in flight
            __builtin_amdgcn_sched_barrier(0);
            mfmas((KK - 1) & 1, 2, 8);
            __builtin_amdgcn_sched_barrier(0);
        }
        // the tile's last stage: its last MFMAs, then the fold (no fragments
        // live across it), then the hand-over to the next stage
        const int slot = k & 1;
        body(slot);
        mfmas((KK - 1) & 1);
        if ((vt + 1) * kTileV > V)
            fold(vt, std::true_type{});
        else
            fold(vt, std::false_type{});
        if (k + 1 < T) {
            wait_vm0();
            lds_barrier();
            if (k + 2 < T) issue_next(k + 2);
            read(slot ^ 1, 0, 0);
        }
        ++k;
    }

    // ---- merge: lane halves, then the two vocabulary halves of each token
#pragma unroll
    for (int ti = 0; ti < 2; ++ti) {
        Top o;
        o.m = __shfl_xor(top[ti].m, 32, 64);
        o.mL = __shfl_xor(top[ti].mL, 32, 64);
        o.s = __shfl_xor(top[ti].s, 32, 64);
        o.idx = __shfl_xor(top[ti].idx, 32, 64);
        top[ti] = top_merge(top[ti], o);
    }
    __syncthreads();
    if (wv == 1 && h == 0) {
#pragma unroll
        for (int ti = 0; ti < 2; ++ti) s_top[wt * 64 + ti * 32 + n] = top[ti];
    }
    __syncthreads();
    if (wv == 0 && h == 0) {
#pragma unroll
        for (int ti = 0; ti < 2; ++ti) {
            const int tok = wt * 64 + ti * 32 + n;
            const int row = row0 + tok;
            const Top t = top_merge(top[ti], s_top[tok]);
            if (row < row_cap && pv.row_req[row] >= 0)
                part[(size_t)blk * kTileT + tok] = top_pack(t);
        }
    }
    }
}

// One wave per row: partials k = lane, lane + 64, ... (partition k of the
// row's token tile, written by block k * n_lt + tile) merged per lane in
// increasing k, then across lanes by a fixed butterfly.
__global__ void __launch_bounds__(kMergeThreads)
lm_merge_kernel(const float4* __restrict__ lm_part, int n_vtiles, int cu, PackView pv,
                int row_cap, int padded, float4* __restrict__ upd_part, int nsplit) {
    const int row = blockIdx.x * (kMergeThreads / 64) + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= row_cap || pv.row_req[row] < 0) return;
    const int n_lt = ((padded ? row_cap : pv.hdr[kHdrRows]) + kTileT - 1) / kTileT;
    const int P = lm_parts_dev(n_lt, n_vtiles, cu);
    const size_t base = (size_t)(row / kTileT) * kTileT + row % kTileT;
    const size_t stride = (size_t)n_lt * kTileT;
    Top t = top_empty();
    for (int k = lane; k < P; k += 64) t = top_merge(t, top_unpack(lm_part[base + k * stride]));
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        Top o;
        o.m = __shfl_xor(t.m, off, 64);
        o.mL = __shfl_xor(t.mL, off, 64);
        o.s = __shfl_xor(t.s, off, 64);
        o.idx = __shfl_xor(t.idx, off, 64);
        t = top_merge(t, o);
    }
    for (int k = lane; k < nsplit; k += 64)
        upd_part[(size_t)row * nsplit + k] = top_pack(k == 0 ? t : top_empty());
}

}  // namespace

LmSizes lm_sizes(const fb_pack* pack, int V, int D, int cu_count) {
    LmSizes z{};
    z.n_rtiles = (pack->row_cap + kTileT - 1) / kTileT;
    z.n_vtiles = (V + kTileV - 1) / kTileV;
    z.cu = cu_count > 0 ? cu_count : 256;
    // the grid: the largest n_lt * P over every count of token tiles the
    // rows can fill (memoized: the search is over n_rtiles x kMaxParts)
    static std::mutex mu;
    static std::map<std::tuple<int, int, int>, int> memo;
    const auto key = std::make_tuple(z.n_rtiles, z.n_vtiles, z.cu);
    int grid = 0;
    {
        std::lock_guard<std::mutex> lock(mu);
        auto it = memo.find(key);
        if (it != memo.end()) {
            grid = it->second;
        } else {
            for (int n = 1; n <= z.n_rtiles; ++n) {
                const int g = n * lm_parts_host(n, z.n_vtiles, z.cu);
                grid = g > grid ? g : grid;
            }
            memo.emplace(key, grid);
        }
    }
    // partials: one per block; workgroups: at most eight per CU, each taking
    // blocks in turn (blocks past n_lt * P end at once, but each still holds
    // its CU for a moment)
    z.total = (size_t)grid * kTileT * sizeof(float4);
    z.grid = grid < 8 * z.cu ? grid : 8 * z.cu;
    (void)D;
    return z;
}

hipError_t launch_lmhead(const void* hidden, const void* weight, int D, int V,
                         const fb_pack* pack, void* lm_ws, const LmSizes& z, void* upd_ws,
                         const UpdateSizes& uz, hipStream_t stream) {
    PackView pv = pack_view(pack);
    float4* lm_part = static_cast<float4*>(lm_ws);
    hipLaunchKernelGGL(lmhead_kernel, dim3((unsigned)z.grid), dim3(kLmThreads), 0, stream,
                       static_cast<const uint16_t*>(hidden), static_cast<const uint16_t*>(weight),
                       D, V, pack->row_cap, pack->layout == FB_PADDED ? 1 : 0, z.n_vtiles, z.cu,
                       pv, lm_part);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int rows_per_wg = kMergeThreads / 64;
    hipLaunchKernelGGL(lm_merge_kernel,
                       dim3((unsigned)((pack->row_cap + rows_per_wg - 1) / rows_per_wg)),
                       dim3(kMergeThreads), 0, stream, lm_part, z.n_vtiles, z.cu, pv,
                       pack->row_cap, pack->layout == FB_PADDED ? 1 : 0,
                       static_cast<float4*>(upd_ws), uz.nsplit);
    return hipGetLastError();
}

}  // namespace fb
