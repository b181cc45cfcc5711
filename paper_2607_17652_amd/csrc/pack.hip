// Heterogeneous Wavefront Packing, Eq. 4 (Sec. 4.2): the per-request
// wavefront states become the packed batch -- a compact list of live-block
// tiles plus per-row request / position / token maps.
//
// pack_kernel (one workgroup) validates every request and computes w_b; a
// block-wide exclusive scan of w_b gives each request its first tile (and, in
// the ragged layout, its first packed row).  Then every one of the row_cap
// row-map entries is written exactly once, live or not, so the output is
// fully defined without a separate clearing pass: for up to 4096 rows by the
// same workgroup, from the (request, first position) of each tile (ragged)
// or (w_b, o_b) of each request (padded) it kept in LDS; beyond, by
// rowmap_kernel, one thread per row.
#include "internal.h"

namespace fb {
namespace {

constexpr int kPackThreads = 1024;
constexpr int kPackWaves = kPackThreads / 64;

// Exclusive scan of one int per thread across the workgroup; also returns the
// total.  Each wave scans its 64 values, then every wave scans the
// kPackWaves wave totals itself.  `lds` holds kPackWaves ints.
__device__ int workgroup_exclusive_scan(int v, int* lds, int* total) {
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    int x = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        int y = __shfl_up(x, off, 64);
        if (lane >= off) x += y;
    }
    if (lane == 63) lds[wave] = x;
    __syncthreads();
    int w = lane < kPackWaves ? lds[lane] : 0;
#pragma unroll
    for (int off = 1; off < kPackWaves; off <<= 1) {
        int y = __shfl_up(w, off, 64);
        if (lane >= off) w += y;
    }
    const int before = __shfl(w, wave > 0 ? wave - 1 : 0, 64);
    *total = __shfl(w, kPackWaves - 1, 64);
    __syncthreads();
    return (wave > 0 ? before : 0) + x - v;
}

// Tiles (ragged) or requests (padded) whose row-map inputs the pack keeps in
// LDS to write the row maps itself, and the row maps one workgroup writes
// faster than a separate launch (measured: 1024 rows 10.7 -> 8.5 us, 32768
// rows 11 -> 20 us).
constexpr int kFusedMax = 4096;
constexpr int kFusedRows = 4096;

template <bool ROWS>
__global__ void __launch_bounds__(kPackThreads)
pack_kernel(const fb_req_state* __restrict__ st, const int32_t* __restrict__ tokens,
            int B, int W_max, int bl, int layout, int n_max, int T_max,
            PackView pv, int row_cap) {
    __shared__ int scan_lds[kPackWaves + 1];
    // ragged: request and first position of each tile; padded: w_b (-1 for a
    // bad state) and o_b of each request
    __shared__ int s_a[ROWS ? kFusedMax : 1];
    __shared__ int s_b[ROWS ? kFusedMax : 1];
    const int tid = threadIdx.x;
    if (tid == 0) pv.hdr[kHdrStatus] = FB_PACK_STATUS_NONE;
    __syncthreads();

    // ---- phase 1: validate, scan w_b, write per-request fields and tiles --
    int tiles_before = 0;
    for (int base = 0; base < B; base += kPackThreads) {
        const int b = base + tid;
        int w = 0;
        bool bad = false;
        fb_req_state s{};
        if (b < B) {
            s = st[b];
            if (s.active) {
                const long long end = (long long)s.gen_start + (long long)s.n_blocks * bl;
                const bool ok = s.L >= 0 && s.L <= s.R && s.R <= s.n_blocks &&
                                s.n_blocks <= n_max && s.R - s.L <= W_max &&
                                s.gen_start >= 0 && end <= (long long)T_max;
                if (ok) w = s.R - s.L;
                else bad = true;
            }
        }
        int total;
        const int excl = workgroup_exclusive_scan(w, scan_lds, &total);
        if (b < B) {
            const int tile0 = tiles_before + excl;
            const int row0 = (layout == FB_PADDED) ? b * W_max * bl : tile0 * bl;
            pv.req_w[b] = bad ? -1 : w;
            pv.req_row0[b] = row0;
            if (bad) record_error(pv.hdr, b, FB_DERR_STATE);
            const int o = s.gen_start + s.L * bl;
            if (ROWS && layout == FB_PADDED) {
                s_a[b] = bad ? -1 : w;
                s_b[b] = o;
            }
            for (int sl = 0; sl < w; ++sl) {
                if (ROWS && layout != FB_PADDED) {
                    s_a[tile0 + sl] = b;
                    s_b[tile0 + sl] = o + sl * bl;
                }
                int32_t* t = pv.tiles + (size_t)(tile0 + sl) * kTileInts;
                t[kTB] = b;
                t[kTS] = sl;
                t[kTG] = s.L + sl;
                t[kTRow0] = row0 + sl * bl;
                t[kTPos0] = o + sl * bl;
                t[kTO] = o;
                t[kTKvLen] = o + (sl + 1) * bl;
                t[kTW] = w;
            }
        }
        tiles_before += total;
    }
    if (tid == 0) {
        pv.hdr[kHdrRows] = tiles_before * bl;
        pv.hdr[kHdrTiles] = tiles_before;
    }
    if constexpr (ROWS) {
        // ---- phase 2: the row maps (as rowmap_kernel), four rows per
        // thread and pass with their token loads in flight together
        __syncthreads();
        const int n_rows = tiles_before * bl;
        const int q = W_max * bl;
        constexpr int U = 4;
        for (int r0 = tid; r0 < row_cap; r0 += U * kPackThreads) {
            int rb[U], rp[U], rt[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int r = r0 + u * kPackThreads;
                int b = -1, pos = -1;
                if (r < row_cap) {
                    if (layout == FB_PADDED) {
                        const int req = r / q;
                        if ((r % q) / bl < s_a[req]) {
                            b = req;
                            pos = s_b[req] + r % q;
                        }
                    } else if (r < n_rows) {
                        b = s_a[r / bl];
                        pos = s_b[r / bl] + r % bl;
                    }
                }
                rb[u] = b;
                rp[u] = pos;
            }
#pragma unroll
            for (int u = 0; u < U; ++u)
                rt[u] = (rb[u] >= 0 && tokens) ? tokens[(size_t)rb[u] * T_max + rp[u]] : -1;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int r = r0 + u * kPackThreads;
                if (r < row_cap) {
                    pv.row_req[r] = rb[u];
                    pv.row_pos[r] = rp[u];
                    pv.row_tok[r] = rt[u];
                }
            }
        }
    }
}

// Row maps (row -> request, position, token), one thread per packed row.
// Ragged rows are tile-major (row r belongs to tile r / bl); padded rows
// belong to request r / (W_max*bl).
constexpr int kRowThreads = 256;

__global__ void __launch_bounds__(kRowThreads)
rowmap_kernel(const fb_req_state* __restrict__ st, const int32_t* __restrict__ tokens,
              int W_max, int bl, int layout, int T_max, PackView pv, int row_cap) {
    const int r = blockIdx.x * kRowThreads + threadIdx.x;
    if (r >= row_cap) return;
    const int n_rows = pv.hdr[kHdrRows];
    const int q = W_max * bl;
    int b = -1, pos = -1;
    if (layout == FB_PADDED) {
        const int rb = r / q;
        const int slot = (r % q) / bl;
        const int w = pv.req_w[rb];
        if (slot < w) {
            const fb_req_state s = st[rb];
            b = rb;
            pos = s.gen_start + s.L * bl + (r % q);
        }
    } else if (r < n_rows) {
        const int32_t* t = pv.tiles + (size_t)(r / bl) * kTileInts;
        b = t[kTB];
        pos = t[kTPos0] + (r % bl);
    }
    pv.row_req[r] = b;
    pv.row_pos[r] = pos;
    pv.row_tok[r] = (b >= 0 && tokens) ? tokens[(size_t)b * T_max + pos] : -1;
}

}  // namespace

hipError_t launch_pack(const fb_req_state* st, const int32_t* tokens, int n_max,
                       int T_max, const fb_pack* pack, hipStream_t stream) {
    PackView pv = pack_view(pack);
    const bool rows = pack->row_cap <= kFusedRows &&
                      (pack->layout == FB_PADDED ? pack->B <= kFusedMax
                                                 : pack->tile_cap <= kFusedMax);
    if (rows) {
        hipLaunchKernelGGL(pack_kernel<true>, dim3(1), dim3(kPackThreads), 0, stream, st,
                           tokens, pack->B, pack->W_max, pack->bl, pack->layout,
                           n_max, T_max, pv, pack->row_cap);
        return hipGetLastError();
    }
    hipLaunchKernelGGL(pack_kernel<false>, dim3(1), dim3(kPackThreads), 0, stream, st,
                       tokens, pack->B, pack->W_max, pack->bl, pack->layout,
                       n_max, T_max, pv, pack->row_cap);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(rowmap_kernel, dim3((pack->row_cap + kRowThreads - 1) / kRowThreads),
                       dim3(kRowThreads), 0, stream, st, tokens, pack->W_max, pack->bl,
                       pack->layout, T_max, pv, pack->row_cap);
    return hipGetLastError();
}

}  // namespace fb
