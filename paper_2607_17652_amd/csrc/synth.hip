// Synthetic model for the device-side decode loop: a SplitMix64 hash model
// standing in for f_theta (no weights are part of this library).  Its logits
// depend on exactly the tokens Sec. 4.1 lets a block see, [0, lo + bl) for
// the block at [lo, lo + bl), and its embeddings on (position, token).  The
// full definition is in flowblock_loop.h.
//
//   synth_pred_kernel   one workgroup per request: context hash, staleness
//                       and first mask of every live block, then (k, level)
//                       of every live row
//   synth_fill_kernel   (row, vocabulary split) workgroups write the logits:
//                       zeros with levels[level] at k
//   synth_embed_kernel  one workgroup per live row: q, k, v values
#include "internal.h"

namespace fb {
namespace {

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;
constexpr int kPredThreads = 256;
constexpr int kFillThreads = 256;
constexpr int kEmbedThreads = 256;

__device__ inline uint64_t sm_mix(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// n-th output of SplitMix64 seeded with s
__device__ inline uint64_t sm_hash(uint64_t s, uint64_t n) { return sm_mix(s + (n + 1) * kGamma); }

__device__ inline uint64_t token_term(uint64_t seed, int j, int x) {
    return sm_hash(seed, ((uint64_t)(uint32_t)j << 32) | (uint32_t)x);
}

__global__ void __launch_bounds__(kPredThreads)
synth_pred_kernel(const fb_req_state* __restrict__ st, const int32_t* __restrict__ tokens,
                  int T_max, PackView pv, int bl, int W_max, int V, uint64_t seed,
                  int2* __restrict__ pred) {
    __shared__ unsigned long long s_sum[64];     // per live slot (W_max <= 64)
    __shared__ int s_masks[64], s_first[64];
    __shared__ unsigned long long s_pre;
    __shared__ int s_stale;
    const int b = blockIdx.x;
    const int tid = threadIdx.x;
    const int w = pv.req_w[b];
    if (w <= 0) return;
    const fb_req_state s = st[b];
    const int M = V - 1;
    const int o = s.gen_start + s.L * bl;
    const int32_t* x = tokens + (size_t)b * T_max;
    if (tid < w) {
        s_sum[tid] = 0;
        s_masks[tid] = 0;
        s_first[tid] = 0x7fffffff;
    }
    if (tid == 0) {
        s_pre = 0;
        s_stale = 0;
    }
    __syncthreads();

    // frozen prefix [0, o): context terms and masks in [gen_start, o).
    // Integer sums mod 2^64 do not depend on the order of the additions.
    unsigned long long acc = 0;
    int stale = 0;
    for (int j = tid; j < o; j += kPredThreads) {
        const int xj = x[j];
        if (xj != M) acc += token_term(seed, j, xj);
        else if (j >= s.gen_start) stale += 1;
    }
    atomicAdd(&s_pre, acc);
    atomicAdd(&s_stale, stale);

    // live blocks: per-slot terms, masks and first mask
    const int nrows = w * bl;
    for (int i = tid; i < nrows; i += kPredThreads) {
        const int j = o + i;
        const int sl = i / bl;
        const int xj = x[j];
        if (xj != M) {
            atomicAdd(&s_sum[sl], (unsigned long long)token_term(seed, j, xj));
        } else {
            atomicAdd(&s_masks[sl], 1);
            atomicMin(&s_first[sl], j);
        }
    }
    __syncthreads();
    if (tid == 0) {
        unsigned long long ctx = s_pre;
        int stl = s_stale;
        for (int sl = 0; sl < w; ++sl) {
            ctx += s_sum[sl];
            s_sum[sl] = ctx;                 // context of slot sl: [0, lo + bl)
            const int m = s_masks[sl];
            s_masks[sl] = stl;               // staleness of slot sl: [gen_start, lo)
            stl += m;
        }
    }
    __syncthreads();

    const int row0 = pv.req_row0[b];
    for (int i = tid; i < nrows; i += kPredThreads) {
        const int sl = i / bl;
        const int p = o + i;
        const uint64_t h = sm_hash(s_sum[sl], (uint64_t)p);
        int k;
        if (s_masks[sl] == 0 || (h >> 63) == 0)
            k = (int)(sm_hash(seed, (1ull << 63) + (uint64_t)p) % (uint64_t)(V - 1));
        else
            k = (int)(h % (uint64_t)(V - 1));
        const int lvl = p == s_first[sl] ? 3 : (int)((h >> 32) & 3);
        pred[row0 + i] = make_int2(k, lvl);
    }
}

template <typename T>
__device__ inline T level_value(float a);
template <>
__device__ inline float level_value<float>(float a) { return a; }
template <>
__device__ inline uint16_t level_value<uint16_t>(float a) {
    return (uint16_t)(__float_as_uint(a) >> 16);   // exact: checked on the host
}

// One workgroup per (row, vocabulary split).  Vector path: rows start on a
// 16-byte boundary (V * sizeof(T) % 16 == 0), 16-byte stores; else one
// element per store.
template <typename T>
__global__ void __launch_bounds__(kFillThreads)
synth_fill_kernel(const int2* __restrict__ pred, PackView pv, int V, int nsplit, int chunk,
                  float4 levels, T* __restrict__ logits) {
    const int row = blockIdx.x / nsplit;
    const int k = blockIdx.x % nsplit;
    if (pv.row_req[row] < 0) return;
    const int2 pr = pred[row];
    const int l = pr.y & 3;
    const float lf = l == 0 ? levels.x : l == 1 ? levels.y : l == 2 ? levels.z : levels.w;
    const T a = level_value<T>(lf);
    const int v0 = k * chunk;
    const int v1 = min(V, v0 + chunk);
    T* z = logits + (size_t)row * V;
    constexpr int E = 16 / sizeof(T);
    if (((size_t)V * sizeof(T)) % 16 == 0) {
        // chunk is a multiple of 8 elements, so v0 is 16-byte aligned
        // v1 - v0 is a multiple of E here (chunk % 8 == 0 and V % E == 0)
        const uint32_t abits = sizeof(T) == 2 ? (uint32_t)(uint16_t)a : __float_as_uint((float)a);
        for (int v = v0 + threadIdx.x * E; v < v1; v += kFillThreads * E) {
            uint32_t wd[4] = {0u, 0u, 0u, 0u};
            const int off = pr.x - v;                       // in [0, E) if k is here
            if (off >= 0 && off < E) {
                const int word = sizeof(T) == 2 ? off >> 1 : off;
                const uint32_t val = sizeof(T) == 2 ? abits << ((off & 1) * 16) : abits;
#pragma unroll
                for (int i = 0; i < 4; ++i) wd[i] = i == word ? val : 0u;
            }
            *reinterpret_cast<uint4*>(z + v) = make_uint4(wd[0], wd[1], wd[2], wd[3]);
        }
    } else {
        for (int v = v0 + threadIdx.x; v < v1; v += kFillThreads)
            z[v] = v == pr.x ? a : T(0);
    }
}

template <typename T>
__device__ inline T embed_value(uint64_t h);
template <>
__device__ inline float embed_value<float>(uint64_t h) {
    return (float)((int)(h >> 56) - 128) * (1.0f / 256.0f);
}
template <>
__device__ inline uint16_t embed_value<uint16_t>(uint64_t h) {
    const float f = (float)((int)(h >> 56) - 128) * (1.0f / 256.0f);
    return (uint16_t)(__float_as_uint(f) >> 16);     // k/256, |k| <= 128: exact
}

template <typename T>
__global__ void __launch_bounds__(kEmbedThreads)
synth_embed_kernel(PackView pv, int Hq, int Hkv, int d, uint64_t seed, T* __restrict__ q,
                   T* __restrict__ kn, T* __restrict__ vn) {
    const int row = blockIdx.x;
    if (pv.row_req[row] < 0) return;
    const uint64_t p = (uint64_t)pv.row_pos[row];
    const uint64_t x = (uint64_t)(uint32_t)pv.row_tok[row];
    const int nq = Hq * d, nk = Hkv * d;
    for (int e = threadIdx.x; e < nq + 2 * nk; e += kEmbedThreads) {
        int kind, idx;
        T* dst;
        if (e < nq) {
            kind = 0; idx = e; dst = q + (size_t)row * nq;
        } else if (e < nq + nk) {
            kind = 1; idx = e - nq; dst = kn + (size_t)row * nk;
        } else {
            kind = 2; idx = e - nq - nk; dst = vn + (size_t)row * nk;
        }
        const uint64_t h1 = sm_hash(seed, (1ull << 62) + ((uint64_t)kind << 59) + p);
        const uint64_t h2 = sm_hash(h1, x);
        dst[idx] = embed_value<T>(sm_hash(h2, (uint64_t)idx));
    }
}

}  // namespace

SynthSizes synth_sizes(const fb_pack* pack, int V) {
    SynthSizes z{};
    // about 64 KB of logits per workgroup
    const int per = 32768;
    int ns = (V + per - 1) / per;
    if (ns < 1) ns = 1;
    int chunk = (V + ns - 1) / ns;
    chunk = (chunk + 7) / 8 * 8;
    z.nsplit = (V + chunk - 1) / chunk;
    z.chunk = chunk;
    (void)pack;
    return z;
}

hipError_t launch_synth_logits(const fb_req_state* st, const int32_t* tokens, int T_max,
                               const fb_pack* pack, const fb_synth_model* m, int V,
                               int dtype, int32_t* pred, void* logits, hipStream_t stream) {
    PackView pv = pack_view(pack);
    int2* pr = reinterpret_cast<int2*>(pred);
    hipLaunchKernelGGL(synth_pred_kernel, dim3(pack->B), dim3(kPredThreads), 0, stream, st,
                       tokens, T_max, pv, pack->bl, pack->W_max, V, m->seed, pr);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const SynthSizes z = synth_sizes(pack, V);
    const float4 lv = make_float4(m->levels[0], m->levels[1], m->levels[2], m->levels[3]);
    const dim3 grid((unsigned)pack->row_cap * (unsigned)z.nsplit);
    if (dtype == FB_BF16)
        hipLaunchKernelGGL(synth_fill_kernel<uint16_t>, grid, dim3(kFillThreads), 0, stream,
                           pr, pv, V, z.nsplit, z.chunk, lv, static_cast<uint16_t*>(logits));
    else
        hipLaunchKernelGGL(synth_fill_kernel<float>, grid, dim3(kFillThreads), 0, stream, pr,
                           pv, V, z.nsplit, z.chunk, lv, static_cast<float*>(logits));
    return hipGetLastError();
}

hipError_t launch_synth_embed(const fb_pack* pack, const fb_attn_shape* sh, uint64_t seed,
                              void* q, void* k_new, void* v_new, hipStream_t stream) {
    PackView pv = pack_view(pack);
    const dim3 grid((unsigned)pack->row_cap);
    if (sh->dtype == FB_BF16)
        hipLaunchKernelGGL(synth_embed_kernel<uint16_t>, grid, dim3(kEmbedThreads), 0, stream,
                           pv, sh->Hq, sh->Hkv, sh->head_dim, seed,
                           static_cast<uint16_t*>(q), static_cast<uint16_t*>(k_new),
                           static_cast<uint16_t*>(v_new));
    else
        hipLaunchKernelGGL(synth_embed_kernel<float>, grid, dim3(kEmbedThreads), 0, stream, pv,
                           sh->Hq, sh->Hkv, sh->head_dim, seed, static_cast<float*>(q),
                           static_cast<float*>(k_new), static_cast<float*>(v_new));
    return hipGetLastError();
}

}  // namespace fb
