// Bookkeeping kernel of the device-side decode loop (Alg. 1's outer loop):
// at the start of every step, count the step if some request is active and
// count a forward for every request with a live window; the same kernel with
// count = 0 only refreshes the any-active flag the host polls.
#include "internal.h"

namespace fb {
namespace {

constexpr int kCountThreads = 256;

__global__ void __launch_bounds__(kCountThreads)
loop_count_kernel(const fb_req_state* __restrict__ st, int B,
                  fb_loop_counters* __restrict__ counters, int32_t* __restrict__ forwards,
                  int count) {
    __shared__ int s_any;
    if (threadIdx.x == 0) s_any = 0;
    __syncthreads();
    int any = 0;
    for (int b = threadIdx.x; b < B; b += kCountThreads) {
        const fb_req_state s = st[b];
        if (s.active) {
            any = 1;
            if (count && s.R > s.L) forwards[b] += 1;
        }
    }
    if (any) atomicOr(&s_any, 1);
    __syncthreads();
    if (threadIdx.x == 0) {
        counters->any_active = s_any;
        if (count && s_any) counters->steps += 1;
    }
}

}  // namespace

hipError_t launch_loop_count(const fb_req_state* st, int B, fb_loop_counters* counters,
                             int32_t* forwards, int count, hipStream_t stream) {
    hipLaunchKernelGGL(loop_count_kernel, dim3(1), dim3(kCountThreads), 0, stream, st, B,
                       counters, forwards, count);
    return hipGetLastError();
}

}  // namespace fb
