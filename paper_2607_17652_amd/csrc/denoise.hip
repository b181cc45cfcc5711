// Denoise update: vocab-wide reduction, joint M2T/T2T update (Eq. 1), block
// readiness (Eq. 2), post-edit bookkeeping (Sec. 3.1), in-order retirement and
// readiness-gated admission (Alg. 1, Eq. 3).
//
// vocab_pass_kernel   a few workgroups per live row, each taking every
//                     nsplit-th 32 KB piece of the row: streams the logits
//                     once in 16-byte loads and keeps, per thread, (max,
//                     lowest index of the max, sum of
//                     exp2(z*log2e - round(max*log2e))); wavefront butterfly
//                     then LDS merge; one 16-byte partial per workgroup.
// request_kernel      one workgroup per request: merges a row's partials in
//                     workgroup order, applies Eq. 1, counts each live block,
//                     then retires and admits on one thread.
// Every reduction has a fixed order, so results are bit-reproducible.
#include "internal.h"
#include "top.h"

namespace fb {
namespace {

constexpr int kVocabThreads = 512;   // 8 waves per (row, partition): measured 1% faster than 4
constexpr int kUpdThreads = 256;

// Maximum of the values (logits hold no NaN, so the max needs no quieting
// of its inputs: three-input v_max3 steps instead of fmaxf chains).
template <int N>
__device__ inline float max_of(const float (&f)[N]) {
    if constexpr (N == 1) {
        return f[0];
    } else {
        float m = f[0];
        int j = 1;
        for (; j + 1 < N; j += 2)
            asm("v_max3_f32 %0, %1, %2, %3" : "=v"(m) : "v"(m), "v"(f[j]), "v"(f[j + 1]));
        if (j < N) asm("v_max_f32 %0, %1, %2" : "=v"(m) : "v"(m), "v"(f[j]));
        return m;
    }
}

// Fold n consecutive values starting at index v into t (values in index order).
template <int N>
__device__ inline void top_fold(Top& t, const float (&f)[N], int v) {
    const float vmax = max_of(f);
    if (vmax > t.m) {
#pragma clang fp contract(off)
        int j0 = N - 1;
#pragma unroll
        for (int j = N - 1; j >= 0; --j)
            if (f[j] == vmax) j0 = j;
        const float nmL = scaled_ref(vmax);
        t.s *= __builtin_amdgcn_exp2f(t.mL - nmL);
        t.m = vmax;
        t.mL = nmL;
        t.idx = v + j0;
    }
    // While t is empty (mL = -inf, only before the first finite value) the
    // reference is the lowest finite float instead, so -inf logits give
    // exp2(-inf) = 0 rather than -inf + inf: no branch on all -inf groups.
    const float ref = fmaxf(t.mL, -3.402823466e38f);
    float e[N];
#pragma unroll
    for (int j = 0; j < N; ++j) e[j] = __builtin_amdgcn_exp2f(fmaf(f[j], kLog2e, -ref));
#pragma unroll
    for (int w = 1; w < N; w <<= 1)
#pragma unroll
        for (int j = 0; j + w < N; j += 2 * w) e[j] += e[j + w];
    t.s += e[0];
}

// 16-byte load of logits that are read exactly once: the nontemporal hint
// keeps the stream from displacing reusable lines in the caches, which
// measurably raises the achieved HBM read rate of this pass.
template <typename T>
__device__ inline uint4 load_stream16(const T* p) {
    typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
    const u32x4 x = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
    return make_uint4(x[0], x[1], x[2], x[3]);
}

template <typename T>
struct VecTraits;
template <>
struct VecTraits<uint16_t> {   // bf16
    static constexpr int N = 8;
    __device__ static inline void unpack(const uint4& u, float (&f)[8]) {
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            f[2 * j] = __uint_as_float(w[j] << 16);
            f[2 * j + 1] = __uint_as_float(w[j] & 0xffff0000u);
        }
    }
    __device__ static inline float scalar(const uint16_t* p) {
        return __uint_as_float(((uint32_t)*p) << 16);
    }
};
template <>
struct VecTraits<float> {
    static constexpr int N = 4;
    __device__ static inline void unpack(const uint4& u, float (&f)[4]) {
        f[0] = __uint_as_float(u.x);
        f[1] = __uint_as_float(u.y);
        f[2] = __uint_as_float(u.z);
        f[3] = __uint_as_float(u.w);
    }
    __device__ static inline float scalar(const float* p) { return *p; }
};

// A row's nsplit workgroups take its 16-byte-aligned body in pieces of
// kBatch loads per thread (32 KB), in turn: workgroup k reads pieces k,
// k + nsplit, ...  Neighbouring workgroups then read neighbouring memory,
// which the HBM serves faster than the same bytes in one contiguous share
// per workgroup.
constexpr int kVocabBatch = 4;

template <typename T>
__global__ void __launch_bounds__(kVocabThreads)
vocab_pass_kernel(const T* __restrict__ logits, int V, int nsplit,
                  PackView pv, float4* __restrict__ part, int bl, int padded) {
    using VT = VecTraits<T>;
    constexpr int N = VT::N;
    constexpr int kBatch = kVocabBatch;
    const int slot = blockIdx.x / nsplit;
    const int k = blockIdx.x % nsplit;
    int row = slot;
    if (padded) {
        // workgroups walk the live tiles' rows first, so the padding rows
        // of the layout are not interleaved with live ones in the grid
        const int t = slot / bl;
        if (t >= pv.hdr[kHdrTiles]) return;
        row = pv.tiles[(size_t)t * kTileInts + kTRow0] + slot % bl;
    } else if (pv.row_req[row] < 0) {   // ragged rows are tile-major: live ones first
        return;
    }
    const T* rp = logits + (size_t)row * V;
    const int tid = threadIdx.x;

    // Body [a, e) is 16-byte aligned in memory; head [0, a) and tail [e, V)
    // are taken one element at a time by the first threads of workgroup 0.
    const size_t abs0 = (size_t)row * V;
    int a = (int)((N - (abs0 % N)) % N);
    if (a > V) a = V;
    const int e = a + ((V - a) / N) * N;

    Top t = top_empty();
    if (k == 0 && tid < a) {
        float f[1] = {VT::scalar(rp + tid)};
        top_fold<1>(t, f, tid);
    }
    const int stride = kVocabThreads * N;
    const int piece = kBatch * stride;
    for (int base = a + k * piece + tid * N; base < e; base += nsplit * piece) {
        uint4 raw[kBatch];
#pragma unroll
        for (int j = 0; j < kBatch; ++j) {
            const int v = base + j * stride;
            raw[j] = v < e ? load_stream16(rp + v) : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int j = 0; j < kBatch; ++j) {
            const int v = base + j * stride;
            if (v < e) {
                float f[N];
                VT::unpack(raw[j], f);
                top_fold<N>(t, f, v);
            }
        }
    }
    if (k == 0 && tid < V - e) {
        float f[1] = {VT::scalar(rp + e + tid)};
        top_fold<1>(t, f, e + tid);
    }

    // Wavefront butterfly (every lane ends with the same value), then waves
    // merged in order by thread 0.
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        Top o;
        o.m = __shfl_xor(t.m, off, 64);
        o.mL = __shfl_xor(t.mL, off, 64);
        o.s = __shfl_xor(t.s, off, 64);
        o.idx = __shfl_xor(t.idx, off, 64);
        t = top_merge(t, o);
    }
    __shared__ Top wtop[kVocabThreads / 64];
    if ((tid & 63) == 0) wtop[tid >> 6] = t;
    __syncthreads();
    if (tid == 0) {
        Top r = wtop[0];
        for (int w = 1; w < kVocabThreads / 64; ++w) r = top_merge(r, wtop[w]);
        part[(size_t)row * nsplit + k] = make_float4(r.m, r.s, __int_as_float(r.idx), r.mL);
    }
}

struct UpdParams {
    double tau_mask, tau_edit, theta;
    int mask_id, eos_id, S_pe, W;
    unsigned flags;
};

enum RowFlag : uint8_t {
    kMaskedBefore = 1,
    kDecodable = 2,
    kWritten = 8,
    kForceable = 16,
};

__global__ void __launch_bounds__(kUpdThreads)
request_kernel(const float4* __restrict__ part, int nsplit, PackView pv,
               int32_t* __restrict__ tokens, int T_max, float* __restrict__ conf_out,
               int32_t* __restrict__ argmax_out, fb_req_state* __restrict__ st,
               uint8_t* __restrict__ pe, uint8_t* __restrict__ fin, int n_max, int bl,
               int W_max, UpdParams prm, fb_req_stats* __restrict__ stats,
               double* __restrict__ rho_last) {
    extern __shared__ unsigned char upd_smem[];
    const int rows_cap = W_max * bl;
    float* s_conf = reinterpret_cast<float*>(upd_smem);
    int* s_xhat = reinterpret_cast<int*>(s_conf + rows_cap);
    uint8_t* s_flag = reinterpret_cast<uint8_t*>(s_xhat + rows_cap);
    __shared__ double s_rho[64];
    __shared__ int s_m2t[64], s_t2t[64];
    __shared__ uint8_t s_fin[64];   // fin of the live blocks after this step

    const int b = blockIdx.x;
    const int tid = threadIdx.x;
    // the request's fields are read together (each is in bounds for any b)
    const int w = pv.req_w[b];
    const fb_req_state s = st[b];
    const int row0 = pv.req_row0[b];
    if (w < 0) {
        if (tid == 0 && stats) {
            fb_req_stats z{};
            z.valid = 0;
            z.rho_frontier = -1.0;
            stats[b] = z;
        }
        return;
    }
    const int nrows = w * bl;
    const int o = s.gen_start + s.L * bl;
    int32_t* tok = tokens + (size_t)b * T_max;

    // ---- rows: merge partials, Eq. 1 ----------------------------------------
    for (int i = tid; i < nrows; i += kUpdThreads) {
        const int row = row0 + i;
        const int pos = o + i;
        const float4* pr = part + (size_t)row * nsplit;
        // the row's token and its first partials are loaded together before
        // any is used (merged below in partition order, as before)
        constexpr int kPre = 4;
        typedef float f32x4 __attribute__((ext_vector_type(4)));
        f32x4 pre[kPre];
#pragma unroll
        for (int k = 0; k < kPre; ++k)
            pre[k] = *reinterpret_cast<const f32x4*>(pr + (k < nsplit ? k : nsplit - 1));
        const int x = tok[pos];
#pragma unroll
        for (int k = 0; k < kPre; ++k) asm volatile("" :: "v"(pre[k]));
        asm volatile("" :: "v"(x));
        Top t{pre[0][0], pre[0][3], pre[0][1], __float_as_int(pre[0][2])};
#pragma unroll
        for (int k = 1; k < kPre; ++k)
            if (k < nsplit)
                t = top_merge(t, Top{pre[k][0], pre[k][3], pre[k][1], __float_as_int(pre[k][2])});
        for (int k = kPre; k < nsplit; ++k) {
            const float4 pk = pr[k];
            t = top_merge(t, Top{pk.x, pk.w, pk.y, __float_as_int(pk.z)});
        }
        // s is relative to round(m*log2e); undo that rounding exactly.
        const float resid = fmaf(t.m, kLog2e, -t.mL);
        const float conf = 1.0f / (t.s * __builtin_amdgcn_exp2f(-resid));
        const int xhat = t.idx;
        const bool masked = x == prm.mask_id;
        const bool prompt = pos < s.prompt_len;
        const double c = (double)conf;
        const bool gamma = masked && c > prm.tau_mask && xhat != prm.mask_id;
        const bool delta = ((prm.flags & FB_EDIT_MASKED) || !masked) && !prompt &&
                           xhat != x && c > prm.tau_edit && xhat != prm.mask_id;
        uint8_t f = 0;
        if (masked) f |= kMaskedBefore;
        if (masked && c >= prm.tau_mask) f |= kDecodable;
        if (gamma || delta) {
            f |= kWritten;
            tok[pos] = xhat;
        }
        if (masked && xhat != prm.mask_id) f |= kForceable;
        conf_out[row] = conf;
        argmax_out[row] = xhat;
        s_conf[i] = conf;
        s_xhat[i] = xhat;
        s_flag[i] = f;
    }
    __syncthreads();

    // ---- blocks: one wavefront per live block --------------------------------
    const int wave = tid >> 6;
    const int lane = tid & 63;
    for (int sl = wave; sl < w; sl += kUpdThreads / 64) {
        int m_before = 0, dec = 0, u = 0, wr_masked = 0;
        float best_c = -1.f;
        int best_i = 0x7fffffff;
        for (int i = sl * bl + lane; i < (sl + 1) * bl; i += 64) {
            const uint8_t f = s_flag[i];
            m_before += (f & kMaskedBefore) ? 1 : 0;
            dec += (f & kDecodable) ? 1 : 0;
            u += (f & kWritten) ? 1 : 0;
            wr_masked += ((f & kWritten) && (f & kMaskedBefore)) ? 1 : 0;
            if ((f & kForceable) && s_conf[i] > best_c) {
                best_c = s_conf[i];
                best_i = i;
            }
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
            m_before += __shfl_xor(m_before, off, 64);
            dec += __shfl_xor(dec, off, 64);
            u += __shfl_xor(u, off, 64);
            wr_masked += __shfl_xor(wr_masked, off, 64);
            const float oc = __shfl_xor(best_c, off, 64);
            const int oi = __shfl_xor(best_i, off, 64);
            if (oc > best_c || (oc == best_c && oi < best_i)) {
                best_c = oc;
                best_i = oi;
            }
        }
        if (lane == 0) {
            // Forced progress only where no masked row was revealed (by
            // Gamma, or by Delta under FB_EDIT_MASKED): every candidate is
            // then still masked and no row is counted twice.
            if ((prm.flags & FB_FORCE_PROGRESS) && m_before > 0 && wr_masked == 0 &&
                best_i != 0x7fffffff) {
                tok[o + best_i] = s_xhat[best_i];
                u += 1;
                wr_masked += 1;
            }
            const int m_after = m_before - wr_masked;
            const int g = s.L + sl;
            uint8_t* pe_g = pe + (size_t)b * n_max + g;
            uint8_t* fin_g = fin + (size_t)b * n_max + g;
            const uint8_t fin0 = *fin_g;
            bool now = false;
            if (m_before == 0) {
                const int npe = min(255, (int)*pe_g + 1);
                *pe_g = (uint8_t)npe;
                now = u == 0 || npe >= prm.S_pe;
            } else if (m_after == 0 && prm.S_pe == 0) {
                now = true;
            }
            if (now) *fin_g = 1;
            s_fin[sl] = (fin0 || now) ? 1 : 0;
            s_rho[sl] = m_before == 0 ? 1.0 : (double)dec / (double)m_before;
            s_m2t[sl] = wr_masked;
            s_t2t[sl] = u - wr_masked;
        }
    }
    __syncthreads();

    // ---- retire, then admit (Alg. 1) -----------------------------------------
    if (tid != 0) return;
    fb_req_stats rs{};
    rs.valid = 1;
    rs.rho_frontier = w > 0 ? s_rho[w - 1] : -1.0;
    for (int sl = 0; sl < w; ++sl) {
        rs.m2t += s_m2t[sl];
        rs.t2t += s_t2t[sl];
    }
    if (prm.flags & FB_SYNC_WINDOW) {
        // the shared window moves in sync_window_kernel, after every request
        // has finished its blocks' bookkeeping
        rho_last[b] = w > 0 ? s_rho[w - 1] : 0.0;
        if (stats) stats[b] = rs;
        return;
    }
    fb_req_state ns = s;
    if (ns.active) {
        // every block in [L, R) is live this step, so its fin is in s_fin
        while (ns.L < ns.R && s_fin[ns.L - s.L]) {
            const int g = ns.L;
            ns.L += 1;
            rs.committed += 1;
            if (prm.eos_id >= 0) {
                const int lo = ns.gen_start + g * bl;
                bool hit = false;
                for (int i = 0; i < bl; ++i) hit |= tok[lo + i] == prm.eos_id;
                if (hit) {
                    ns.active = 0;
                    ns.eos_hit = 1;
                    rs.eos = 1;
                    rs.done = 1;
                    break;
                }
            }
        }
        if (ns.active && ns.L >= ns.n_blocks) {
            ns.active = 0;
            rs.done = 1;
        }
        if (ns.active) {
            const int L0 = s.L, R0 = s.R;
            auto admit = [&]() {
                pe[(size_t)b * n_max + ns.R] = 0;
                fin[(size_t)b * n_max + ns.R] = 0;
                ns.R += 1;
                rs.spawned += 1;
            };
            if (ns.L == ns.R && ns.R < ns.n_blocks) admit();
            while (ns.R - ns.L < prm.W && ns.R < ns.n_blocks) {
                const int g = ns.R - 1;
                double rho;
                if (g < ns.L) rho = 1.0;                      // committed
                else if (g >= L0 && g < R0) rho = s_rho[g - L0];  // live this step
                else rho = 0.0;                               // admitted this step
                if (!(rho >= prm.theta)) break;
                admit();
            }
        }
    }
    st[b] = ns;
    if (stats) stats[b] = rs;
}

// Batch-synchronous retire and admit (FB_SYNC_WINDOW; the synchronous
// wavefront of the Sec. 5 ablation): one workgroup over all requests.  The
// requests taking part are the active, well-formed ones; they must share
// (L, R, n).  Thread i owns requests i, i + blockDim.x, ... and is the only
// writer of their state and statistics.
constexpr int kSyncThreads = 1024;

__global__ void __launch_bounds__(kSyncThreads)
sync_window_kernel(PackView pv, int B, fb_req_state* __restrict__ st,
                   const int32_t* __restrict__ tokens, int T_max,
                   uint8_t* __restrict__ pe, uint8_t* __restrict__ fin, int n_max, int bl,
                   UpdParams prm, fb_req_stats* __restrict__ stats,
                   const double* __restrict__ rho_last) {
    __shared__ int s_cnt, s_lo[3], s_hi[3], s_all;
    __shared__ double s_min[kSyncThreads / 64];
    const int tid = threadIdx.x;
    if (tid == 0) {
        s_cnt = 0;
        for (int k = 0; k < 3; ++k) {
            s_lo[k] = 0x7fffffff;
            s_hi[k] = -0x7fffffff;
        }
    }
    __syncthreads();
    auto part = [&](int b) { return st[b].active != 0 && pv.req_w[b] >= 0; };
    for (int b = tid; b < B; b += kSyncThreads) {
        if (!part(b)) continue;
        const fb_req_state s = st[b];
        const int v[3] = {s.L, s.R, s.n_blocks};
        atomicAdd(&s_cnt, 1);
        for (int k = 0; k < 3; ++k) {
            atomicMin(&s_lo[k], v[k]);
            atomicMax(&s_hi[k], v[k]);
        }
    }
    __syncthreads();
    if (s_cnt == 0) return;
    if (s_lo[0] != s_hi[0] || s_lo[1] != s_hi[1] || s_lo[2] != s_hi[2]) {
        for (int b = tid; b < B; b += kSyncThreads)
            if (part(b)) record_error(pv.hdr, b, FB_DERR_STATE);
        return;
    }
    const int L0 = s_lo[0], R0 = s_lo[1], n = s_lo[2];

    // ---- retire: block L goes when every taking-part request finished it --
    int L = L0;
    while (L < R0) {
        if (tid == 0) s_all = 1;
        __syncthreads();
        for (int b = tid; b < B; b += kSyncThreads)
            if (part(b) && !fin[(size_t)b * n_max + L]) s_all = 0;
        __syncthreads();
        const int all = s_all;
        __syncthreads();
        if (!all) break;
        for (int b = tid; b < B; b += kSyncThreads) {
            if (!part(b)) continue;
            fb_req_state s = st[b];
            s.L = L + 1;
            int eos = 0;
            if (prm.eos_id >= 0) {
                const int32_t* blk = tokens + (size_t)b * T_max + s.gen_start + L * bl;
                for (int i = 0; i < bl; ++i) eos |= blk[i] == prm.eos_id;
            }
            if (eos) {
                s.active = 0;
                s.eos_hit = 1;
            }
            st[b] = s;
            if (stats) {
                stats[b].committed += 1;
                if (eos) {
                    stats[b].eos = 1;
                    stats[b].done = 1;
                }
            }
        }
        L += 1;
        __syncthreads();
    }
    if (L >= n) {
        for (int b = tid; b < B; b += kSyncThreads) {
            if (!part(b)) continue;
            st[b].active = 0;
            if (stats) stats[b].done = 1;
        }
        return;
    }

    // ---- admit, gated by the smallest readiness of B_{R-1} ------------------
    int R = R0;
    auto admit = [&]() {
        for (int b = tid; b < B; b += kSyncThreads) {
            if (!part(b)) continue;
            pe[(size_t)b * n_max + R] = 0;
            fin[(size_t)b * n_max + R] = 0;
            if (stats) stats[b].spawned += 1;
        }
        R += 1;
    };
    if (L == R && R < n) admit();
    while (R - L < prm.W && R < n) {
        const int g = R - 1;
        double m = 2.0;    // above any readiness
        for (int b = tid; b < B; b += kSyncThreads) {
            if (!part(b)) continue;
            const double rho = g < L ? 1.0 : (g < R0 ? rho_last[b] : 0.0);
            m = fmin(m, rho);
        }
        for (int off = 32; off > 0; off >>= 1) m = fmin(m, __shfl_xor(m, off, 64));
        if ((tid & 63) == 0) s_min[tid >> 6] = m;
        __syncthreads();
        double mm = s_min[0];
        for (int k = 1; k < kSyncThreads / 64; ++k) mm = fmin(mm, s_min[k]);
        __syncthreads();
        if (!(mm >= prm.theta)) break;
        admit();
    }
    for (int b = tid; b < B; b += kSyncThreads)
        if (part(b)) st[b].R = R;
}

}  // namespace

UpdateSizes update_sizes(const fb_pack* pack, int V, int cu_count) {
    UpdateSizes z{};
    const int target = 8 * (cu_count > 0 ? cu_count : 256);
    // workgroups per row: enough for about eight per CU, at least two (their
    // interleaved pieces read faster than one workgroup's whole row), at
    // most one per 32 KB piece of the row and 64
    const int pieces = (V + kVocabBatch * kVocabThreads * 8 - 1) / (kVocabBatch * kVocabThreads * 8);
    int ns = (target + pack->row_cap - 1) / pack->row_cap;
    if (ns < 2) ns = 2;
    if (ns > pieces) ns = pieces;
    if (ns > 64) ns = 64;
    if (ns < 1) ns = 1;
    z.nsplit = ns;
    z.off_rho = (size_t)pack->row_cap * z.nsplit * sizeof(float4);
    z.total = z.off_rho + ((size_t)pack->B * sizeof(double) + 15) / 16 * 16;
    return z;
}

hipError_t launch_vocab_reduce(const void* logits, int V, int dtype,
                               const fb_pack* pack, void* ws, const UpdateSizes& z,
                               hipStream_t stream) {
    PackView pv = pack_view(pack);
    float4* part = static_cast<float4*>(ws);
    const dim3 grid((unsigned)pack->row_cap * (unsigned)z.nsplit);
    if (dtype == FB_BF16) {
        hipLaunchKernelGGL(vocab_pass_kernel<uint16_t>, grid, dim3(kVocabThreads), 0,
                           stream, static_cast<const uint16_t*>(logits), V, z.nsplit,
                           pv, part, pack->bl, pack->layout == FB_PADDED ? 1 : 0);
    } else {
        hipLaunchKernelGGL(vocab_pass_kernel<float>, grid, dim3(kVocabThreads), 0,
                           stream, static_cast<const float*>(logits), V, z.nsplit,
                           pv, part, pack->bl, pack->layout == FB_PADDED ? 1 : 0);
    }
    return hipGetLastError();
}

hipError_t launch_apply(int32_t* tokens, int T_max, float* conf, int32_t* argmax,
                        fb_req_state* st, uint8_t* pe, uint8_t* fin, int n_max,
                        const fb_pack* pack, const fb_update_params* p,
                        fb_req_stats* stats, const void* ws, const UpdateSizes& z,
                        hipStream_t stream) {
    PackView pv = pack_view(pack);
    UpdParams prm{p->tau_mask, p->tau_edit, p->theta_spawn, p->mask_id,
                  p->eos_id,   p->S_pe,     p->W,           p->flags};
    const size_t rows_cap = (size_t)pack->W_max * pack->bl;
    const size_t smem = rows_cap * (sizeof(float) + sizeof(int) + 1);
    double* rho_last = reinterpret_cast<double*>(static_cast<char*>(const_cast<void*>(ws)) +
                                                 z.off_rho);
    hipLaunchKernelGGL(request_kernel, dim3(pack->B), dim3(kUpdThreads), smem, stream,
                       static_cast<const float4*>(ws), z.nsplit, pv, tokens, T_max,
                       conf, argmax, st, pe, fin, n_max, pack->bl, pack->W_max, prm,
                       stats, rho_last);
    if (p->flags & FB_SYNC_WINDOW) {
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(sync_window_kernel, dim3(1), dim3(kSyncThreads), 0, stream, pv,
                           pack->B, st, tokens, T_max, pe, fin, n_max, pack->bl, prm,
                           stats, rho_last);
    }
    return hipGetLastError();
}

}  // namespace fb
