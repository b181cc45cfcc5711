// Window prologue: rotary position embedding at absolute positions on the
// live rows' queries and keys (the "absolute RoPE position ids" of Sec. 4.2),
// fused with the Eq. 6 window KV write, so the fresh keys are rotated and
// land in the paged cache in one pass.
//
// rope_kv_kernel  one workgroup per (live block of bl rows, KV head c): the
//                 g = Hq/Hkv query heads of c, key head c and value head c;
//                 the block's cos/sin table (positions x d/2 pairs, angles
//                 formed and reduced to [-pi, pi] in float64, sin/cos in
//                 float) in LDS; queries
//                 rotated in place or into q_out; keys rotated and written to
//                 their absolute slots of the K cache; values staged in LDS
//                 and written key-innermost to the V cache.  Pair j of a head
//                 vector is (x_j, x_{j+d/2}) (rotate-half arrangement), angle
//                 p * base^(-2j/d).
#include "internal.h"

namespace fb {
namespace {

constexpr int kRopeThreads = 256;
constexpr double k2Pi = 6.283185307179586;
constexpr double kInv2Pi = 0.15915494309189535;

struct ThetaTable {
    double t[64];   // base^(-2j/d), j < d/2 <= 64
};

template <typename T>
struct Vec8;
template <>
struct Vec8<uint16_t> {   // bf16 x 8 in one 16-byte load
    __device__ static inline void load(const uint16_t* p, float (&f)[8]) {
        const uint4 u = *reinterpret_cast<const uint4*>(p);
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            f[2 * j] = __uint_as_float(w[j] << 16);
            f[2 * j + 1] = __uint_as_float(w[j] & 0xffff0000u);
        }
    }
    __device__ static inline void store(uint16_t* p, const float (&f)[8]) {
        uint32_t w[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const __bf16 a = (__bf16)f[2 * j], b = (__bf16)f[2 * j + 1];
            w[j] = (uint32_t)__builtin_bit_cast(uint16_t, a) |
                   ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
        }
        *reinterpret_cast<uint4*>(p) = make_uint4(w[0], w[1], w[2], w[3]);
    }
};
template <>
struct Vec8<float> {      // fp32 x 8 in two 16-byte loads
    __device__ static inline void load(const float* p, float (&f)[8]) {
        const float4 a = *reinterpret_cast<const float4*>(p);
        const float4 b = *reinterpret_cast<const float4*>(p + 4);
        f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w;
        f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
    }
    __device__ static inline void store(float* p, const float (&f)[8]) {
        *reinterpret_cast<float4*>(p) = make_float4(f[0], f[1], f[2], f[3]);
        *reinterpret_cast<float4*>(p + 4) = make_float4(f[4], f[5], f[6], f[7]);
    }
};

// Rotate the 8 pairs (lo[k], hi[k]) of group g of row i with the table.
__device__ inline void rotate8(float (&lo)[8], float (&hi)[8], const float2* cs) {
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        const float c = cs[k].x, s = cs[k].y;
        const float a = lo[k], b = hi[k];
        lo[k] = fmaf(a, c, -b * s);
        hi[k] = fmaf(b, c, a * s);
    }
}

template <typename T>
__global__ void __launch_bounds__(kRopeThreads)
rope_kv_kernel(const T* __restrict__ q_in, T* __restrict__ q_out, const T* __restrict__ k_new,
               const T* __restrict__ v_new, T* __restrict__ k_cache, T* __restrict__ v_cache,
               const int32_t* __restrict__ page_table, PackView pv, int Hq, int Hkv, int D,
               int bl, int ps, int max_pages, int num_pages, int pitch, ThetaTable theta) {
    extern __shared__ __attribute__((aligned(16))) unsigned char rope_smem[];
    float2* tab = reinterpret_cast<float2*>(rope_smem);   // [bl][D/2] (cos, sin)
    T* vs = reinterpret_cast<T*>(rope_smem);              // later: [bl][pitch]
    const int t = blockIdx.x;
    const int c = blockIdx.y;
    if (t >= pv.hdr[kHdrTiles]) return;
    const int g = Hq / Hkv;
    const int32_t* tile = pv.tiles + (size_t)t * kTileInts;
    const int b = tile[kTB];
    const int row0 = tile[kTRow0];
    const int pos0 = tile[kTPos0];
    const int32_t* pt = page_table + (size_t)b * max_pages;
    const int half = D / 2;
    const int ng = half / 8;                              // 8-pair groups per head

    for (int e = threadIdx.x; e < bl * half; e += kRopeThreads) {
        const int i = e / half;
        const int j = e % half;
        // angle in float64, reduced to [-pi, pi] in float64, then float sin/cos
        const double a = (double)(pos0 + i) * theta.t[j];
        const double r = a - rint(a * kInv2Pi) * k2Pi;
        float s, c;
        sincosf((float)r, &s, &c);
        tab[e] = make_float2(c, s);
    }
    __syncthreads();

    // queries of the heads that read KV head c
    for (int e = threadIdx.x; e < bl * g * ng; e += kRopeThreads) {
        const int gi = e % ng;
        const int hh = c * g + (e / ng) % g;
        const int i = e / (ng * g);
        const size_t base = ((size_t)(row0 + i) * Hq + hh) * D + gi * 8;
        float lo[8], hi[8];
        Vec8<T>::load(q_in + base, lo);
        Vec8<T>::load(q_in + base + half, hi);
        rotate8(lo, hi, tab + i * half + gi * 8);
        Vec8<T>::store(q_out + base, lo);
        Vec8<T>::store(q_out + base + half, hi);
    }
    // keys: rotated straight into their absolute slots
    for (int e = threadIdx.x; e < bl * ng; e += kRopeThreads) {
        const int gi = e % ng;
        const int i = e / ng;
        const int pos = pos0 + i;
        const int pidx = pos / ps;
        const int page = pidx < max_pages ? pt[pidx] : -1;
        if (page < 0 || page >= num_pages) {
            if (gi == 0) record_error(pv.hdr, b, FB_DERR_PAGE);
            continue;
        }
        const size_t src = ((size_t)(row0 + i) * Hkv + c) * D + gi * 8;
        float lo[8], hi[8];
        Vec8<T>::load(k_new + src, lo);
        Vec8<T>::load(k_new + src + half, hi);
        rotate8(lo, hi, tab + i * half + gi * 8);
        T* dst = k_cache + (((size_t)page * Hkv + c) * ps + (pos % ps)) * D + gi * 8;
        Vec8<T>::store(dst, lo);
        Vec8<T>::store(dst + half, hi);
    }
    __syncthreads();   // the table's LDS is reused for the values below

    // values of head c: key-innermost rows of the V cache
    constexpr int VEC = 16 / sizeof(T);
    const int dch = D / VEC;
    {
        for (int e = threadIdx.x; e < bl * dch; e += kRopeThreads) {
            const int i = e / dch;
            const int dc = e % dch;
            const size_t src = ((size_t)(row0 + i) * Hkv + c) * D + (size_t)dc * VEC;
            *reinterpret_cast<uint4*>(vs + (size_t)i * pitch + dc * VEC) =
                *reinterpret_cast<const uint4*>(v_new + src);
        }
        __syncthreads();
        if (pos0 % VEC == 0 && ps % VEC == 0 && bl % VEC == 0) {
            const int nrun = bl / VEC;
            for (int e = threadIdx.x; e < D * nrun; e += kRopeThreads) {
                const int ic = e % nrun;
                const int d = e / nrun;
                const int pos = pos0 + ic * VEC;
                const int pidx = pos / ps;
                const int page = pidx < max_pages ? pt[pidx] : -1;
                if (page < 0 || page >= num_pages) continue;   // recorded with the keys
                union {
                    uint4 v;
                    T x[VEC];
                } run;
#pragma unroll
                for (int k = 0; k < VEC; ++k) run.x[k] = vs[(size_t)(ic * VEC + k) * pitch + d];
                *reinterpret_cast<uint4*>(v_cache + (((size_t)page * Hkv + c) * D + d) * ps +
                                          (pos % ps)) = run.v;
            }
        } else {
            for (int e = threadIdx.x; e < bl * D; e += kRopeThreads) {
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
        __syncthreads();
    }
}

}  // namespace

size_t prologue_smem_bytes(const fb_pack* pack, const fb_attn_shape* sh, int* pitch_out) {
    const size_t elt = sh->dtype == FB_BF16 ? 2 : 4;
    int pitch = sh->head_dim + (int)(16 / elt);
    if ((size_t)pack->bl * pitch * elt > 65536) pitch = sh->head_dim;
    if (pitch_out) *pitch_out = pitch;
    const size_t table = (size_t)pack->bl * (sh->head_dim / 2) * sizeof(float2);
    const size_t vstage = (size_t)pack->bl * pitch * elt;
    return table > vstage ? table : vstage;
}

hipError_t launch_window_prologue(const void* q_in, void* q_out, const void* k_new,
                                  const void* v_new, void* k_cache, void* v_cache,
                                  const int32_t* page_table, const fb_pack* pack,
                                  const fb_attn_shape* sh, double rope_base,
                                  hipStream_t stream) {
    PackView pv = pack_view(pack);
    ThetaTable th{};
    const int D = sh->head_dim;
    for (int j = 0; j < D / 2; ++j) th.t[j] = pow(rope_base, -2.0 * j / D);
    int pitch = 0;
    const size_t smem = prologue_smem_bytes(pack, sh, &pitch);
    const dim3 grid(pack->tile_cap, sh->Hkv);
    if (sh->dtype == FB_BF16)
        hipLaunchKernelGGL(rope_kv_kernel<uint16_t>, grid, dim3(kRopeThreads), smem, stream,
                           static_cast<const uint16_t*>(q_in), static_cast<uint16_t*>(q_out),
                           static_cast<const uint16_t*>(k_new),
                           static_cast<const uint16_t*>(v_new), static_cast<uint16_t*>(k_cache),
                           static_cast<uint16_t*>(v_cache), page_table, pv, sh->Hq, sh->Hkv, D,
                           pack->bl, sh->page_size, sh->max_pages, sh->num_pages, pitch, th);
    else
        hipLaunchKernelGGL(rope_kv_kernel<float>, grid, dim3(kRopeThreads), smem, stream,
                           static_cast<const float*>(q_in), static_cast<float*>(q_out),
                           static_cast<const float*>(k_new), static_cast<const float*>(v_new),
                           static_cast<float*>(k_cache), static_cast<float*>(v_cache),
                           page_table, pv, sh->Hq, sh->Hkv, D, pack->bl, sh->page_size,
                           sh->max_pages, sh->num_pages, pitch, th);
    return hipGetLastError();
}

}  // namespace fb
