// Internal declarations shared by the libmoe host API and its HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/libmoe.h"

namespace moe {

// ---------------------------------------------------------------- bf16
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float bf16_to_f32(uint16_t b)
{
    return __uint_as_float((uint32_t)b << 16);
}

// fp32 -> bf16, round to nearest even; NaN stays a quiet NaN.
__device__ __forceinline__ uint16_t f32_to_bf16(float f)
{
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// Two packed bf16 (little-endian: low half first) <-> two floats.
__device__ __forceinline__ float bf16lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi)
{
    return (uint32_t)f32_to_bf16(lo) | ((uint32_t)f32_to_bf16(hi) << 16);
}

// Records a message for moe_last_error() on the calling thread and returns st.
moe_status set_error(moe_status st, const char *fmt, ...);

// ------------------------------------------------------------- timing
// Record around every kernel launch when timing is enabled (see timing.cpp).
struct KernelTimer {
    int slot;
    hipStream_t s;
    KernelTimer(int kind, hipStream_t stream);
    ~KernelTimer();
};

// ------------------------------------------------------------ launchers
// Every launcher enqueues on `s` and returns hipGetLastError() of the launch.
hipError_t launch_route(const float *logits, int64_t T, int E, int k, int32_t *ids, float *w,
                        hipStream_t s);

int64_t permute_chunks(int64_t T, int k, int El);
// Device address of the current device's permutation scratch array
// (MOE_PERMUTE_SCRATCH_BYTES), looked up once per device.
hipError_t permute_scratch(int32_t **ptr);
hipError_t launch_permute(const int32_t *ids, int64_t T, int k, int e0, int El, int32_t *counts,
                          int32_t *offsets, int32_t *row_to_pair, int32_t *pair_to_row,
                          const uint16_t *x, int H, uint16_t *x_perm, int64_t cap, int32_t *ws,
                          hipStream_t s);

size_t ffn_workspace_bytes(int64_t cap, int El, int H, int Is);
// Whether the 64-wide-K large-tile kernels serve these sizes (x_rows: rows of
// the activation operand; rows: all rows of the call).  A call with a shared
// expert needs them.
bool ffn_large_tiles(int64_t x_rows, int64_t rows, int H, int Is);
// shared_rows = 0: no shared expert (sw13, sw2, shared_y unused).
hipError_t launch_grouped_ffn(const uint16_t *x, int64_t x_rows, const int32_t *row_index, int kdiv,
                              const int32_t *offsets, int El, int64_t cap, int H, int Is,
                              const uint16_t *w13, const uint16_t *w2, uint16_t *y, int64_t shared_begin,
                              int64_t shared_rows, const uint16_t *sw13, const uint16_t *sw2,
                              uint16_t *shared_y, void *ws, hipStream_t s);

// Matrix-core reference loop (calib.hip): grid workgroups of 512 threads,
// out[grid * 512].
hipError_t launch_calib_mfma(int grid, int iters, int zero, float *out, hipStream_t s);

// dir: MOE_EP_TO_TP or MOE_TP_TO_EP; src arrays are host arrays of P device
// pointers (NULL pairs skipped).
hipError_t launch_reshard(int dir, int P, int r, int E, int H, int I, const uint16_t *const *src_w13,
                          const uint16_t *const *src_w2, uint16_t *dst_w13, uint16_t *dst_w2, hipStream_t s);

hipError_t launch_kv_slots(const int32_t *page_table, int64_t stride, const int32_t *first, int n_req,
                           int page_size, int64_t max_tokens, int32_t *slots, hipStream_t s);
hipError_t launch_kv_move(int n_src, const uint16_t *const *sk, const uint16_t *const *sv, const int64_t *s_slots,
                          const int64_t *first, int s_heads, uint16_t *dk, uint16_t *dv, int64_t d_slots, int d_heads,
                          int head_dim, int hs0, int hd0, int nh, const int32_t *src_slot, const int32_t *dst_slot,
                          hipStream_t s);

// The whole layer (moe_layer_forward): routing, permutation (no x_perm)
// and tile schedule in fused launches where layer_fused_prep says so, else
// the separate launches of the four calls; then the GEMMs and the combine.
// ws_perm: moe_permute_workspace_size bytes; ws_ffn: the grouped FFN's.
bool layer_fused_prep(int64_t T, int k, int El, int H, int Is, int64_t sc);
hipError_t launch_layer(const uint16_t *x, const float *logits, int64_t T, int E, int k, int e0, int El, int H,
                        int Is, const uint16_t *w13, const uint16_t *w2, int64_t sb, int64_t sc,
                        const uint16_t *sw13, const uint16_t *sw2, int32_t *ids, float *w, int32_t *counts,
                        int32_t *offsets, int32_t *r2p, int32_t *p2r, uint16_t *y, uint16_t *shared_y,
                        uint16_t *out, int32_t *ws_perm, void *ws_ffn, hipStream_t s);

hipError_t launch_combine(const uint16_t *y, int64_t y_rows, const int32_t *pair_to_row,
                          const float *w, int64_t T, int k, int H, const uint16_t *shared_y,
                          int64_t sb, int64_t sc, int accumulate, uint16_t *out, hipStream_t s);

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

}  // namespace moe
