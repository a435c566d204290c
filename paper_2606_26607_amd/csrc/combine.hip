// Combine: unpermute the expert outputs and reduce them with the gate
// weights, one token per block sweep, 8 bf16 (16 bytes) per thread access.
#include "moe_internal.h"

namespace moe {
namespace {

__device__ __forceinline__ void add8(float acc[8], uint4 v, float s)
{
    acc[0] += s * bf16lo(v.x);
    acc[1] += s * bf16hi(v.x);
    acc[2] += s * bf16lo(v.y);
    acc[3] += s * bf16hi(v.y);
    acc[4] += s * bf16lo(v.z);
    acc[5] += s * bf16hi(v.z);
    acc[6] += s * bf16lo(v.w);
    acc[7] += s * bf16hi(v.w);
}

__global__ __launch_bounds__(256) void combine_kernel(const uint16_t *__restrict__ y, int64_t y_rows,
                                                      const int32_t *__restrict__ pair_to_row,
                                                      const float *__restrict__ w, int64_t T, int k,
                                                      int H, const uint16_t *__restrict__ shared_y,
                                                      int64_t sb, int64_t sc, int accumulate,
                                                      uint16_t *__restrict__ out)
{
    __shared__ int32_t rows[MOE_MAX_TOPK];
    __shared__ float wts[MOE_MAX_TOPK];
    const int vecs = H / 8;
    for (int64_t t = blockIdx.x; t < T; t += gridDim.x) {
        if (threadIdx.x < k) {
            int32_t r = pair_to_row[t * k + threadIdx.x];
            rows[threadIdx.x] = (r >= 0 && r < y_rows) ? r : -1;
            wts[threadIdx.x] = w[t * k + threadIdx.x];
        }
        __syncthreads();
        const bool has_shared = shared_y != nullptr && t >= sb && t < sb + sc;
        uint4 *o = reinterpret_cast<uint4 *>(out + t * H);
        for (int i = threadIdx.x; i < vecs; i += blockDim.x) {
            float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
            if (accumulate) add8(acc, o[i], 1.0f);
            if (has_shared)
                add8(acc, reinterpret_cast<const uint4 *>(shared_y + (t - sb) * H)[i], 1.0f);
            for (int j = 0; j < k; ++j) {
                const int32_t r = rows[j];
                if (r >= 0) add8(acc, reinterpret_cast<const uint4 *>(y + (int64_t)r * H)[i], wts[j]);
            }
            uint4 v;
            v.x = pack_bf16(acc[0], acc[1]);
            v.y = pack_bf16(acc[2], acc[3]);
            v.z = pack_bf16(acc[4], acc[5]);
            v.w = pack_bf16(acc[6], acc[7]);
            o[i] = v;
        }
        __syncthreads();
    }
}

}  // namespace

hipError_t launch_combine(const uint16_t *y, int64_t y_rows, const int32_t *pair_to_row,
                          const float *w, int64_t T, int k, int H, const uint16_t *shared_y,
                          int64_t sb, int64_t sc, int accumulate, uint16_t *out, hipStream_t s)
{
    if (T == 0) return hipSuccess;
    KernelTimer timer(MOE_K_COMBINE, s);
    int64_t blocks = T < 8192 ? T : 8192;
    int threads = H / 8 >= 256 ? 256 : ((H / 8 + 63) / 64) * 64;
    combine_kernel<<<dim3((unsigned)blocks), dim3(threads), 0, s>>>(
        y, y_rows, pair_to_row, w, T, k, H, shared_y, sb, sc, accumulate, out);
    return hipGetLastError();
}

}  // namespace moe
