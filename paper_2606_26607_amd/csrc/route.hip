// Gating: softmax top-k over router logits, one lane group per token.
//
// A token's E logits are spread over a group of G lanes (G = 8..64, a power
// of two no smaller than min(E, 64)), S logits per lane.  Each logit becomes
// a 64-bit key whose high word orders floats (with -0.0 folded onto +0.0)
// and whose low word is ~id, so the largest key is the largest logit with
// the lowest expert id.  k rounds of a group-wide max over the keys pick the
// experts in rank order; the weights are exp(l_j - l_0) / sum_i exp(l_i - l_0)
// over the kept logits, which equals the full softmax renormalised over the
// kept experts.
#include "moe_internal.h"

namespace moe {
namespace {

__device__ __forceinline__ uint32_t order_key(float f)
{
    uint32_t u = __float_as_uint(f);
    if ((u << 1) == 0) u = 0;  // -0.0 -> +0.0
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float key_value(uint32_t o)
{
    uint32_t u = (o & 0x80000000u) ? (o & 0x7fffffffu) : ~o;
    return __uint_as_float(u);
}

template <int G>
__device__ __forceinline__ uint64_t group_max(uint64_t v)
{
#pragma unroll
    for (int off = G / 2; off > 0; off >>= 1) {
        uint64_t o = __shfl_xor(v, off, G);
        v = o > v ? o : v;
    }
    return v;
}

template <int G>
__device__ __forceinline__ float group_sum(float v)
{
#pragma unroll
    for (int off = G / 2; off > 0; off >>= 1) v += __shfl_xor(v, off, G);
    return v;
}

template <int G, int S>
__global__ __launch_bounds__(256) void route_kernel(const float *__restrict__ logits, int64_t T,
                                                    int E, int k, int32_t *__restrict__ ids,
                                                    float *__restrict__ w)
{
    constexpr int TPB = 256 / G;  // tokens per block per sweep
    const int sub = threadIdx.x % G;
    for (int64_t t = (int64_t)blockIdx.x * TPB + threadIdx.x / G; t < T;
         t += (int64_t)gridDim.x * TPB) {
        const float *row = logits + t * E;
        uint64_t key[S];
#pragma unroll
        for (int m = 0; m < S; ++m) {
            int e = sub + m * G;
            key[m] = e < E ? ((uint64_t)order_key(row[e]) << 32) | (uint32_t)(~e) : 0ull;
        }
        uint64_t mine = 0, top = 0;
        for (int j = 0; j < k; ++j) {
            uint64_t best = 0;
#pragma unroll
            for (int m = 0; m < S; ++m) best = key[m] > best ? key[m] : best;
            uint64_t win = group_max<G>(best);
#pragma unroll
            for (int m = 0; m < S; ++m)
                if (key[m] == win) key[m] = 0;  // ids are unique: exactly one slot matches
            if (j == 0) top = win;
            if (sub == j) mine = win;
        }
        float l0 = key_value((uint32_t)(top >> 32));
        float ex = 0.f;
        if (sub < k) ex = expf(key_value((uint32_t)(mine >> 32)) - l0);
        float z = group_sum<G>(ex);
        if (sub < k) {
            ids[t * k + sub] = (int32_t)(~(uint32_t)mine);
            w[t * k + sub] = ex / z;
        }
    }
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
    if (E <= 8) return go<8, 1>(logits, T, E, k, ids, w, s);
    if (E <= 16) return go<16, 1>(logits, T, E, k, ids, w, s);
    if (E <= 32) return go<32, 1>(logits, T, E, k, ids, w, s);
    if (E <= 64) return go<64, 1>(logits, T, E, k, ids, w, s);
    if (E <= 128) return go<64, 2>(logits, T, E, k, ids, w, s);
    if (E <= 256) return go<64, 4>(logits, T, E, k, ids, w, s);
    if (E <= 512) return go<64, 8>(logits, T, E, k, ids, w, s);
    return go<64, 16>(logits, T, E, k, ids, w, s);
}

}  // namespace moe
