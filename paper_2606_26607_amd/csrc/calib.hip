// Matrix-core reference loop for measurement (not part of the layer): how
// fast the bf16 matrix cores run on this device when nothing else limits
// them.  With random operands the chip lowers its clock under the switching
// activity, so this rate, not the datasheet figure, bounds what any bf16
// GEMM on real data can reach here.
#include "moe_internal.h"

namespace moe {
namespace {

constexpr int CALIB_THREADS = 512;  // 8 waves, two per SIMD, like the grouped GEMM

__device__ __forceinline__ uint32_t mix32(uint32_t x)
{
    x ^= x >> 16;
    x *= 0x7feb352du;
    x ^= x >> 15;
    x *= 0x846ca68bu;
    x ^= x >> 16;
    return x;
}

// Each wave keeps 2 x 4 independent 32x32 accumulators (the grouped GEMM's
// 64 x 128 block) and issues iters rounds of 8 v_mfma_f32_32x32x16_bf16 on
// operands fixed at the start: uniform in [-1, 1) for A, [-0.02, 0.02) for B
// (the layer's activation and weight scales), or zeros.
__global__ __launch_bounds__(CALIB_THREADS) void calib_mfma_kernel(int iters, int zero, float *__restrict__ out)
{
    const int tid = threadIdx.x;
    uint32_t h = (uint32_t)(blockIdx.x * CALIB_THREADS + tid) * 0x9e3779b9u + 1u;
    bf16x8_t a[2], b[4];
    for (int i = 0; i < 2; ++i)
        for (int e = 0; e < 8; ++e) {
            h = mix32(h);
            a[i][e] = (__bf16)(zero ? 0.f : ((float)(int)(h & 0xffffu) - 32768.f) / 32768.f);
        }
    for (int j = 0; j < 4; ++j)
        for (int e = 0; e < 8; ++e) {
            h = mix32(h);
            b[j][e] = (__bf16)(zero ? 0.f : ((float)(int)(h & 0xffffu) - 32768.f) / 32768.f * 0.02f);
        }
    f32x16_t acc[2][4];
    for (int i = 0; i < 2; ++i)
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x16_t{};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    float t = 0.f;
    for (int i = 0; i < 2; ++i)
        for (int j = 0; j < 4; ++j)
            for (int q = 0; q < 16; ++q) t += acc[i][j][q];
    out[(int64_t)blockIdx.x * CALIB_THREADS + tid] = t;
}

}  // namespace

hipError_t launch_calib_mfma(int grid, int iters, int zero, float *out, hipStream_t s)
{
    calib_mfma_kernel<<<dim3((unsigned)grid), dim3(CALIB_THREADS), 0, s>>>(iters, zero, out);
    return hipGetLastError();
}

}  // namespace moe

extern "C" moe_status moe_calib_mfma(int grid, int iters, int zero_operands, float *out, void *stream)
{
    if (out == nullptr) return moe::set_error(MOE_ERR_INVALID_ARG, "moe_calib_mfma: null out");
    if (grid < 1 || grid > 65536 || iters < 1 || iters > (1 << 24))
        return moe::set_error(MOE_ERR_INVALID_ARG, "moe_calib_mfma: grid=%d or iters=%d out of range", grid, iters);
    const hipError_t err = moe::launch_calib_mfma(grid, iters, zero_operands != 0, out, (hipStream_t)stream);
    if (err != hipSuccess) return moe::set_error(MOE_ERR_HIP, "moe_calib_mfma: %s", hipGetErrorString(err));
    return MOE_OK;
}
