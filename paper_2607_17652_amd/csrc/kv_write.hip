// Window KV write-back, Eq. 6 (Sec. 4.2, "KV retrieval and write-back"):
// the fresh K/V of each live block lands at its absolute positions of the
// paged caches.  One workgroup per (tile, KV head).  The block's K and V
// rows are loaded first, in 16-byte vectors, and K is copied into its page
// as the page ids arrive.  V is written key-innermost ([page][head][d][slot]):
// the block's V rows are staged in LDS; when the block starts
// on a 16-byte slot boundary each thread then gathers one 16-byte run of
// slots for one d from LDS and stores it whole (neighbouring lanes fill
// neighbouring runs of the same d row), otherwise element by element.
#include "internal.h"

namespace fb {
namespace {

constexpr int kKvThreads = 256;

template <typename T>
__global__ void __launch_bounds__(kKvThreads)
write_kv_kernel(const T* __restrict__ k_new, const T* __restrict__ v_new,
                T* __restrict__ k_cache, T* __restrict__ v_cache,
                const int32_t* __restrict__ page_table, PackView pv, int Hkv,
                int D, int bl, int ps, int max_pages, int num_pages, int pitch) {
    extern __shared__ unsigned char kv_smem[];
    T* vs = reinterpret_cast<T*>(kv_smem);   // [bl][pitch]
    const int t = blockIdx.x;
    const int c = blockIdx.y;
    if (t >= pv.hdr[kHdrTiles]) return;
    const int32_t* tile = pv.tiles + (size_t)t * kTileInts;
    const int b = tile[kTB];
    const int row0 = tile[kTRow0];
    const int pos0 = tile[kTPos0];
    const int32_t* pt = page_table + (size_t)b * max_pages;
    constexpr int VEC = 16 / sizeof(T);
    const int dch = D / VEC;

    // The window's K and V rows are loaded before any page id is known (their
    // addresses do not depend on it), together with the page-table reads;
    // a thread holds kBatch 16-byte chunks of each at a time.
    constexpr int kBatch = 2;
    const int n_ch = bl * dch;
    for (int e0 = 0; e0 < n_ch; e0 += kBatch * kKvThreads) {
        typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
        u32x4 kx[kBatch], vx[kBatch];
        int pg[kBatch];
#pragma unroll
        for (int j = 0; j < kBatch; ++j) {
            // past the block's last chunk a thread reloads that chunk (an
            // address inside the block) and stores nothing below
            const int e = min(e0 + j * kKvThreads + (int)threadIdx.x, n_ch - 1);
            const int i = e / dch;
            const int dc = e % dch;
            const size_t src = ((size_t)(row0 + i) * Hkv + c) * D + (size_t)dc * VEC;
            kx[j] = *reinterpret_cast<const u32x4*>(k_new + src);
            vx[j] = *reinterpret_cast<const u32x4*>(v_new + src);
            const int pidx = (pos0 + i) / ps;
            const int p = pt[min(pidx, max_pages - 1)];
            pg[j] = pidx < max_pages ? p : -1;
        }
        // every load above is issued before any of them is waited for (the
        // compiler would otherwise sink each load to its use)
#pragma unroll
        for (int j = 0; j < kBatch; ++j)
            asm volatile("" :: "v"(kx[j]), "v"(vx[j]), "v"(pg[j]));
#pragma unroll
        for (int j = 0; j < kBatch; ++j) {
            const int e = e0 + j * kKvThreads + threadIdx.x;
            if (e < n_ch) {
                const int i = e / dch;
                const int dc = e % dch;
                // V: staged in LDS ([bl][pitch]) for the key-innermost writes below
                *reinterpret_cast<u32x4*>(vs + (size_t)i * pitch + dc * VEC) = vx[j];
                // K: straight 16-byte copy into the page
                const int pos = pos0 + i;
                const int page = pg[j];
                if (page >= 0 && page < num_pages) {
                    const size_t dst = (((size_t)page * Hkv + c) * ps + (pos % ps)) * D +
                                       (size_t)dc * VEC;
                    *reinterpret_cast<u32x4*>(k_cache + dst) = kx[j];
                } else if (dc == 0) {
                    record_error(pv.hdr, b, FB_DERR_PAGE);
                }
            }
        }
    }
    __syncthreads();
    if (pos0 % VEC == 0 && ps % VEC == 0 && bl % VEC == 0) {
        // run ic of VEC slots for dimension d, gathered from LDS; lanes walk
        // the runs of a d row first, so a wave stores whole d rows of a page
        const int nrun = bl / VEC;
        for (int e = threadIdx.x; e < D * nrun; e += kKvThreads) {
            const int ic = e % nrun;
            const int d = e / nrun;
            const int pos = pos0 + ic * VEC;
            const int pidx = pos / ps;
            const int page = pidx < max_pages ? pt[pidx] : -1;
            if (page < 0 || page >= num_pages) continue;   // recorded by the K loop
            union {
                uint4 v;
                T x[VEC];
            } run;
#pragma unroll
            for (int k = 0; k < VEC; ++k) run.x[k] = vs[(size_t)(ic * VEC + k) * pitch + d];
            *reinterpret_cast<uint4*>(v_cache + (((size_t)page * Hkv + c) * D + d) * ps +
                                      (pos % ps)) = run.v;
        }
        return;
    }
    for (int e = threadIdx.x; e < bl * D; e += kKvThreads) {
        const int d = e / bl;
        const int i = e % bl;
        const int pos = pos0 + i;
        const int pidx = pos / ps;
        const int page = pidx < max_pages ? pt[pidx] : -1;
        if (page < 0 || page >= num_pages) continue;
        v_cache[(((size_t)page * Hkv + c) * D + d) * ps + (pos % ps)] =
            vs[(size_t)i * pitch + d];
    }
}

}  // namespace

hipError_t launch_write_kv(const void* k_new, const void* v_new, void* k_cache,
                           void* v_cache, const int32_t* page_table,
                           const fb_pack* pack, const fb_attn_shape* sh,
                           hipStream_t stream) {
    PackView pv = pack_view(pack);
    const dim3 grid(pack->tile_cap, sh->Hkv);
    // LDS rows padded by 16 bytes (when that still fits 64 KB) so the
    // column gathers of neighbouring rows fall in different banks
    const size_t elt = sh->dtype == FB_BF16 ? 2 : 4;
    int pitch = sh->head_dim + (int)(16 / elt);
    if ((size_t)pack->bl * pitch * elt > 65536) pitch = sh->head_dim;
    if (sh->dtype == FB_BF16) {
        const size_t smem = (size_t)pack->bl * pitch * 2;
        hipLaunchKernelGGL(write_kv_kernel<uint16_t>, grid, dim3(kKvThreads),
                           smem, stream, static_cast<const uint16_t*>(k_new),
                           static_cast<const uint16_t*>(v_new),
                           static_cast<uint16_t*>(k_cache),
                           static_cast<uint16_t*>(v_cache), page_table, pv,
                           sh->Hkv, sh->head_dim, pack->bl, sh->page_size,
                           sh->max_pages, sh->num_pages, pitch);
    } else {
        const size_t smem = (size_t)pack->bl * pitch * 4;
        hipLaunchKernelGGL(write_kv_kernel<float>, grid, dim3(kKvThreads), smem,
                           stream, static_cast<const float*>(k_new),
                           static_cast<const float*>(v_new),
                           static_cast<float*>(k_cache),
                           static_cast<float*>(v_cache), page_table, pv, sh->Hkv,
                           sh->head_dim, pack->bl, sh->page_size, sh->max_pages,
                           sh->num_pages, pitch);
    }
    return hipGetLastError();
}

}  // namespace fb
