// Grouped SwiGLU expert FFN on bf16 MFMA (gfx950).
//
// Two GEMMs per local expert e over its rows [offsets[e], offsets[e+1]):
//   gate-up: h = silu(X W13_g^T) * (X W13_u^T)  -> bf16 h  [rows, I_s]
//   down:    y = h W2^T                         -> bf16 y  [rows, H]
// Both operands are K-contiguous ("NT"), so every MFMA operand fragment is
// one 16-byte LDS read.  Tiles are listed on the device: a schedule kernel
// turns offsets into per-expert m-tile prefix sums, and a persistent grid
// walks (m-tile, n-tile) pairs, so the host never reads the routing result
// and experts with no rows cost nothing.  The gate-up workgroup owns the
// matching gate and up columns, so SwiGLU is applied in registers before h
// is written.
#include "moe_internal.h"

namespace moe {
namespace {

constexpr int BM = 64, BN = 64, BK = 64;
constexpr int KCH = BK / 8;  // 16-byte chunks per tile row

__device__ __forceinline__ int64_t clamp_row(int32_t v, int64_t cap)
{
    int64_t r = v < 0 ? 0 : v;
    return r > cap ? cap : r;
}

// tile_prefix[e] = m-tiles (of BM rows) of experts before e; [El] = total.
__global__ __launch_bounds__(1024) void schedule_kernel(const int32_t *__restrict__ offsets, int El,
                                                        int64_t cap, int bm,
                                                        int32_t *__restrict__ tile_prefix)
{
    __shared__ int32_t wsum[16];
    const int e = threadIdx.x;
    int32_t mt = 0;
    if (e < El) {
        int64_t a = clamp_row(offsets[e], cap), b = clamp_row(offsets[e + 1], cap);
        mt = b > a ? (int32_t)((b - a + bm - 1) / bm) : 0;
    }
    const int lane = e & 63, wv = e >> 6;
    int32_t incl = mt;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        int32_t o = __shfl_up(incl, off, 64);
        if (lane >= off) incl += o;
    }
    if (lane == 63) wsum[wv] = incl;
    __syncthreads();
    int32_t before = 0;
    for (int i = 0; i < wv; ++i) before += wsum[i];
    if (e < El) tile_prefix[e] = before + incl - mt;
    if (e == 1023) tile_prefix[El] = before + incl;
}

// 256 threads = 4 waves in a 2x2 grid, each wave owns a 32x32 block of the
// BMxBN tile (two accumulators when gated).
template <bool GATED>
__global__ __launch_bounds__(256) void gemm_kernel(const uint16_t *__restrict__ A,
                                                   const int32_t *__restrict__ offsets,
                                                   const int32_t *__restrict__ tile_prefix, int El,
                                                   int64_t cap, int N, int K,
                                                   const uint16_t *__restrict__ W,
                                                   int64_t w_stride, int up_off,
                                                   uint16_t *__restrict__ C)
{
    constexpr int BROWS = GATED ? 2 * BN : BN;
    __shared__ uint4 As[BM * KCH];
    __shared__ uint4 Bs[BROWS * KCH];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int n_tiles = (N + BN - 1) / BN;
    const int64_t total = (int64_t)tile_prefix[El] * n_tiles;

    for (int64_t tile = blockIdx.x; tile < total; tile += gridDim.x) {
        const int mt = (int)(tile / n_tiles), nt = (int)(tile % n_tiles);
        int lo = 0, hi = El - 1;
        while (lo < hi) {
            int mid = (lo + hi + 1) >> 1;
            if (tile_prefix[mid] <= mt) lo = mid; else hi = mid - 1;
        }
        const int e = lo;
        const int64_t r0 = clamp_row(offsets[e], cap) + (int64_t)(mt - tile_prefix[e]) * BM;
        int64_t r1 = clamp_row(offsets[e + 1], cap);
        if (r1 > r0 + BM) r1 = r0 + BM;
        const int n0 = nt * BN;
        const uint16_t *We = W + (int64_t)e * w_stride;

        f32x16_t acc_g = {}, acc_u = {};
        for (int k0 = 0; k0 < K; k0 += BK) {
            for (int c = tid; c < BM * KCH; c += 256) {
                const int row = c / KCH, kc = c % KCH;
                const int64_t gr = r0 + row;
                const int kk = k0 + kc * 8;
                uint4 v = {0u, 0u, 0u, 0u};
                if (gr < r1 && kk < K) v = *reinterpret_cast<const uint4 *>(A + gr * K + kk);
                As[row * KCH + (kc ^ (row & 7))] = v;
            }
            for (int c = tid; c < BROWS * KCH; c += 256) {
                const int row = c / KCH, kc = c % KCH;
                const int n = n0 + (row % BN);
                const int64_t wr = (GATED && row >= BN) ? (int64_t)up_off + n : n;
                const int kk = k0 + kc * 8;
                uint4 v = {0u, 0u, 0u, 0u};
                if (n < N && kk < K) v = *reinterpret_cast<const uint4 *>(We + wr * K + kk);
                Bs[row * KCH + (kc ^ (row & 7))] = v;
            }
            __syncthreads();
#pragma unroll
            for (int ks = 0; ks < BK / 16; ++ks) {
                const int ch = ks * 2 + (lane >> 5);
                const int ar = wm * 32 + (lane & 31);
                const int br = wn * 32 + (lane & 31);
                uint4 av = As[ar * KCH + (ch ^ (ar & 7))];
                uint4 bv = Bs[br * KCH + (ch ^ (br & 7))];
                acc_g = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    *reinterpret_cast<bf16x8_t *>(&av), *reinterpret_cast<bf16x8_t *>(&bv), acc_g, 0, 0, 0);
                if (GATED) {
                    const int ur = BN + br;
                    uint4 uv = Bs[ur * KCH + (ch ^ (ur & 7))];
                    acc_u = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        *reinterpret_cast<bf16x8_t *>(&av), *reinterpret_cast<bf16x8_t *>(&uv), acc_u, 0, 0, 0);
                }
            }
            __syncthreads();
        }
        // epilogue: lane holds column (lane & 31), rows 8*(i/4) + 4*(lane/32) + i%4
        const int col = n0 + wn * 32 + (lane & 31);
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int64_t row = r0 + wm * 32 + 8 * (i / 4) + 4 * (lane >> 5) + (i % 4);
            if (row < r1 && col < N) {
                float v = acc_g[i];
                if (GATED) v = v / (1.0f + expf(-v)) * acc_u[i];
                C[row * N + col] = f32_to_bf16(v);
            }
        }
    }
}

}  // namespace

size_t ffn_workspace_bytes(int64_t cap, int El, int H, int Is)
{
    (void)H;
    return align256((size_t)(El + 1) * sizeof(int32_t)) + align256((size_t)cap * Is * 2);
}

hipError_t launch_grouped_ffn(const uint16_t *x_perm, const int32_t *offsets, int El, int64_t cap,
                              int H, int Is, const uint16_t *w13, const uint16_t *w2, uint16_t *y,
                              void *ws, hipStream_t s)
{
    if (cap == 0) return hipSuccess;
    int32_t *tile_prefix = static_cast<int32_t *>(ws);
    uint16_t *h = reinterpret_cast<uint16_t *>(static_cast<char *>(ws) +
                                               align256((size_t)(El + 1) * sizeof(int32_t)));
    hipError_t err;
    {
        KernelTimer timer(MOE_K_SCHEDULE, s);
        schedule_kernel<<<dim3(1), dim3(1024), 0, s>>>(offsets, El, cap, BM, tile_prefix);
        if ((err = hipGetLastError()) != hipSuccess) return err;
    }
    const int64_t max_mtiles = ceil_div(cap, BM) + El;
    {
        KernelTimer timer(MOE_K_GATE_UP, s);
        int64_t tiles = max_mtiles * ceil_div(Is, BN);
        int64_t grid = tiles < 2048 ? tiles : 2048;
        gemm_kernel<true><<<dim3((unsigned)grid), dim3(256), 0, s>>>(
            x_perm, offsets, tile_prefix, El, cap, Is, H, w13, (int64_t)2 * Is * H, Is, h);
        if ((err = hipGetLastError()) != hipSuccess) return err;
    }
    {
        KernelTimer timer(MOE_K_DOWN, s);
        int64_t tiles = max_mtiles * ceil_div(H, BN);
        int64_t grid = tiles < 2048 ? tiles : 2048;
        gemm_kernel<false><<<dim3((unsigned)grid), dim3(256), 0, s>>>(
            h, offsets, tile_prefix, El, cap, H, Is, w2, (int64_t)H * Is, 0, y);
        if ((err = hipGetLastError()) != hipSuccess) return err;
    }
    return hipSuccess;
}

}  // namespace moe
