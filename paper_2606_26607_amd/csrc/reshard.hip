// Expert-weight resharding between the EP and TP views (Sec. 3.1) for one
// destination rank.
//
// EP view of rank q: W13 [E/P, 2I, H], W2 [E/P, H, I] (experts q*E/P ..).
// TP view of rank r: W13 [E, 2I/P, H] (gate rows [r*I/P, (r+1)*I/P) of every
// expert, then the matching up rows) and W2 [E, H, I/P].
//
// A source rank q contributes 1/P of the destination: E/P * 2I/P rows of W13
// (H elements each) and E/P * H runs of W2 (I/P elements each), all
// contiguous in both views.  The kernel walks 16-byte chunks of those rows
// with a grid-stride loop, so every element is read once and written once
// (the bound is HBM).  The source of the destination rank itself is the
// part a switch keeps on the GPU; the other sources are the parts the paper
// moves between GPUs (here any device pointers, e.g. peers' buffers).
#include "moe_internal.h"

namespace moe {
namespace {

struct ReshardArgs {
    const uint16_t *w13[MOE_MAX_RESHARD_RANKS];  // compacted list of the given sources
    const uint16_t *w2[MOE_MAX_RESHARD_RANKS];
    int q[MOE_MAX_RESHARD_RANKS];                // their ranks
    int nsrc;
};

template <int DIR>
__global__ __launch_bounds__(256) void reshard_kernel(ReshardArgs a, int P, int r, int E, int H, int I,
                                                      uint16_t *__restrict__ d13, uint16_t *__restrict__ d2)
{
    const int El = E / P, Is = I / P;
    const int64_t ch_row = H / 8, ch_run = Is / 8;           // 16-byte chunks per W13 row / W2 run
    const int64_t c13 = (int64_t)El * 2 * Is * ch_row;       // W13 chunks per source
    const int64_t c2 = (int64_t)El * H * ch_run;             // W2 chunks per source
    const int64_t per = c13 + c2;
    const int64_t total = per * a.nsrc;
    for (int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; x < total;
         x += (int64_t)gridDim.x * blockDim.x) {
        const int si = (int)(x / per);
        int64_t y = x - (int64_t)si * per;
        const int q = a.q[si];
        const uint16_t *src;
        uint16_t *dst;
        if (y < c13) {
            const int64_t unit = y / ch_row, c = y - unit * ch_row;
            const int l = (int)(unit / (2 * Is)), j = (int)(unit % (2 * Is));
            if (DIR == MOE_EP_TO_TP) {
                // row j of rank r's shard of expert q*El + l: gate row r*Is + j
                // or up row I + r*Is + (j - Is) of the EP source
                const int g = j < Is ? r * Is + j : I + r * Is + (j - Is);
                src = a.w13[si] + ((int64_t)l * 2 * I + g) * H + c * 8;
                dst = d13 + (((int64_t)q * El + l) * 2 * Is + j) * H + c * 8;
            } else {
                // TP source q holds shard q of expert r*El + l
                const int g = j < Is ? q * Is + j : I + q * Is + (j - Is);
                src = a.w13[si] + (((int64_t)r * El + l) * 2 * Is + j) * H + c * 8;
                dst = d13 + ((int64_t)l * 2 * I + g) * H + c * 8;
            }
        } else {
            y -= c13;
            const int64_t unit = y / ch_run, c = y - unit * ch_run;
            const int l = (int)(unit / H), h = (int)(unit % H);
            if (DIR == MOE_EP_TO_TP) {
                src = a.w2[si] + ((int64_t)l * H + h) * I + r * Is + c * 8;
                dst = d2 + (((int64_t)q * El + l) * H + h) * Is + c * 8;
            } else {
                src = a.w2[si] + (((int64_t)r * El + l) * H + h) * Is + c * 8;
                dst = d2 + ((int64_t)l * H + h) * I + q * Is + c * 8;
            }
        }
        typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
        // streamed once: no need to keep either side in the caches
        const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(src));
        __builtin_nontemporal_store(v, reinterpret_cast<u32x4_t *>(dst));
    }
}

}  // namespace

hipError_t launch_reshard(int dir, int P, int r, int E, int H, int I, const uint16_t *const *src_w13,
                          const uint16_t *const *src_w2, uint16_t *dst_w13, uint16_t *dst_w2, hipStream_t s)
{
    ReshardArgs a{};
    for (int q = 0; q < P; ++q) {
        if (!src_w13[q]) continue;
        a.w13[a.nsrc] = src_w13[q];
        a.w2[a.nsrc] = src_w2[q];
        a.q[a.nsrc] = q;
        ++a.nsrc;
    }
    if (a.nsrc == 0) return hipSuccess;
    const int64_t per = (int64_t)(E / P) * (2 * (I / P) * (H / 8) + H * ((I / P) / 8));
    const int64_t total = per * a.nsrc;
    const int64_t blocks = ceil_div(total, 256) < 16384 ? ceil_div(total, 256) : 16384;
    KernelTimer timer(MOE_K_RESHARD, s);
    if (dir == MOE_EP_TO_TP)
        reshard_kernel<MOE_EP_TO_TP><<<dim3((unsigned)blocks), dim3(256), 0, s>>>(a, P, r, E, H, I, dst_w13, dst_w2);
    else
        reshard_kernel<MOE_TP_TO_EP><<<dim3((unsigned)blocks), dim3(256), 0, s>>>(a, P, r, E, H, I, dst_w13, dst_w2);
    return hipGetLastError();
}

}  // namespace moe
