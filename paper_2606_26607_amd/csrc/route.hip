// Gating kernel: softmax top-k over router logits, one lane group per token
// (route_dev.h).
#include "route_dev.h"

namespace moe {
namespace {

using route_dev::route_token;

template <int G, int S>
__global__ __launch_bounds__(256) void route_kernel(const float *__restrict__ logits, int64_t T,
                                                    int E, int k, int32_t *__restrict__ ids,
                                                    float *__restrict__ w)
{
    constexpr int TPB = 256 / G;  // tokens per block per sweep
    const int sub = threadIdx.x % G;
    for (int64_t t = (int64_t)blockIdx.x * TPB + threadIdx.x / G; t < T;
         t += (int64_t)gridDim.x * TPB)
        route_token<G, S>(logits + t * E, E, k, sub, ids + t * k, w + t * k);
}

template <int G, int S>
hipError_t go(const float *logits, int64_t T, int E, int k, int32_t *ids, float *w, hipStream_t s)
{
    constexpr int TPB = 256 / G;
    int64_t blocks = ceil_div(T, TPB);
    if (blocks > 16384) blocks = 16384;
    route_kernel<G, S><<<dim3((unsigned)blocks), dim3(256), 0, s>>>(logits, T, E, k, ids, w);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_route(const float *logits, int64_t T, int E, int k, int32_t *ids, float *w,
                        hipStream_t s)
{
    if (T == 0) return hipSuccess;
    KernelTimer timer(MOE_K_ROUTE, s);
    // Many tokens: 16 lanes per token, each holding several logits (a round
    // of the top-k is S local compares and 4 DPP steps, and a wavefront
    // serves 4 tokens).  Few tokens: 64 lanes per token, so the work spreads
    // over more wavefronts and each lane holds fewer logits.  (The fused
    // layer launches make the same choice: ffn.hip, by_experts.)
    if (E <= 8) return go<8, 1>(logits, T, E, k, ids, w, s);
    if (E <= 16) return go<16, 1>(logits, T, E, k, ids, w, s);
    if (T >= 4096) {
        if (E <= 32) return go<16, 2>(logits, T, E, k, ids, w, s);
        if (E <= 64) return go<16, 4>(logits, T, E, k, ids, w, s);
        if (E <= 128) return go<16, 8>(logits, T, E, k, ids, w, s);
        if (E <= 256) return go<16, 16>(logits, T, E, k, ids, w, s);
        if (E <= 512) return go<16, 32>(logits, T, E, k, ids, w, s);
    }
    if (E <= 64) return go<64, 1>(logits, T, E, k, ids, w, s);
    if (E <= 128) return go<64, 2>(logits, T, E, k, ids, w, s);
    if (E <= 256) return go<64, 4>(logits, T, E, k, ids, w, s);
    if (E <= 512) return go<64, 8>(logits, T, E, k, ids, w, s);
    return go<64, 16>(logits, T, E, k, ids, w, s);
}

}  // namespace moe
