// Permutation: stable counting sort of (token, slot) pairs by local expert.
//
// The T*k pairs are cut into chunks of 256 (or 1024 when pairs x experts
// is large, which keeps the per-chunk histograms small), one wavefront per
// chunk:
//   1. count:   per-chunk histogram over local experts (LDS),
//   2. scan:    per expert, exclusive prefix over chunks; per-expert totals
//               and their exclusive prefix over experts give `offsets`, and
//               each (chunk, expert) gets its first output row,
//   3. scatter: each chunk walks its pairs in order, 64 at a time; lanes
//               holding the same expert find each other with ballots over
//               the bits of the expert index, so a pair's row is its chunk
//               base + earlier pairs of that expert in the chunk + its rank
//               among equal lanes.  No global atomics: the result is the
//               unique stable order, identical on every run.
//   4. gather:  optional copy of x rows into permuted order (16-byte moves).
// Small inputs (decode: at most 16384 pairs over at most 64 local experts,
// and a bounded amount of ballot work, see SMALL_WORK) run steps 1-3 in one
// workgroup instead, saving launches; larger ones with at most 64 local
// experts run steps 2 and 3 in one launch.
#include <mutex>

#include "permute_dev.h"

namespace moe {
namespace {

using namespace permute_dev;

template <int ROUNDS>
__global__ __launch_bounds__(64) void count_kernel(const int32_t *__restrict__ ids, int64_t npairs,
                                                   int e0, int El, int32_t *__restrict__ chunk_cnt)
{
    constexpr int CHUNK = ROUNDS * 64;
    extern __shared__ int32_t hist[];
    const int lane = threadIdx.x;
    const int64_t c = blockIdx.x;
    for (int i = lane; i < El; i += 64) hist[i] = 0;
    __syncthreads();
    const int64_t base = c * CHUNK;
    int32_t v[ROUNDS];
#pragma unroll
    for (int r = 0; r < ROUNDS; ++r) {
        int64_t p = base + r * 64 + lane;
        v[r] = p < npairs ? ids[p] : -1;
    }
#pragma unroll
    for (int r = 0; r < ROUNDS; ++r) {
        int le = local_index(v[r], e0, El);
        if (le < El) atomicAdd(&hist[le], 1);
    }
    __syncthreads();
    for (int i = lane; i < El; i += 64) chunk_cnt[c * El + i] = hist[i];
}

// One block of 1024 threads.  chunk_cnt [nchunks, El] is rewritten in place
// with each (chunk, expert)'s first output row.  Each expert gets a group of
// L lanes (L = the largest power of two <= 1024/El, at most 64, so a group
// lies in one wavefront); lane j of the group owns a contiguous run of
// chunks.  Runs are summed, scanned across the group with shuffles, the
// expert totals scanned across the block, and each lane then writes its
// chunks' first rows.
__global__ __launch_bounds__(1024) void scan_kernel(int32_t *__restrict__ chunk_cnt, int64_t nchunks,
                                                    int El, int L, int32_t *__restrict__ counts,
                                                    int32_t *__restrict__ offsets)
{
    __shared__ int32_t tot[1024];
    __shared__ int32_t wsum[16];
    const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
    const int e = t / L, j = t % L;
    const bool active = e < El;
    const int64_t per = (nchunks + L - 1) / L;
    const int64_t c0 = (int64_t)j * per;
    const int64_t c1 = c0 + per < nchunks ? c0 + per : nchunks;
    // the lane's run of chunk counts, loaded UNR at a time (independent
    // loads, one memory round trip per batch)
    constexpr int UNR = 8;
    int32_t run = 0;
    if (active)
        for (int64_t c = c0; c < c1; c += UNR) {
            int32_t v[UNR];
#pragma unroll
            for (int u = 0; u < UNR; ++u) v[u] = c + u < c1 ? chunk_cnt[(c + u) * El + e] : 0;
#pragma unroll
            for (int u = 0; u < UNR; ++u) run += v[u];
        }
    // exclusive scan of the runs over the L lanes of the expert's group
    int32_t incl = run;
    for (int off = 1; off < L; off <<= 1) {
        const int32_t o = __shfl_up(incl, off, L);
        if (j >= off) incl += o;
    }
    const int32_t seg_before = incl - run;
    const int32_t expert_total = __shfl(incl, L - 1, L);
    // exclusive scan of the expert totals over the block: thread e holds
    // expert e's total
    if (active && j == L - 1) tot[e] = expert_total;
    __syncthreads();
    const int32_t mine = t < El ? tot[t] : 0;
    __syncthreads();
    int32_t ein = mine;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int32_t o = __shfl_up(ein, off, 64);
        if (lane >= off) ein += o;
    }
    if (lane == 63) wsum[wv] = ein;
    __syncthreads();
    int32_t before = 0;
    for (int i = 0; i < wv; ++i) before += wsum[i];
    const int32_t eexcl = before + ein - mine;
    if (t < El) {
        counts[t] = mine;
        offsets[t] = eexcl;
        tot[t] = eexcl;
    }
    if (t == 1023) offsets[El] = before + ein;  // total over all experts
    __syncthreads();
    if (active) {
        int32_t row = tot[e] + seg_before;
        for (int64_t c = c0; c < c1; c += UNR) {
            int32_t v[UNR];
#pragma unroll
            for (int u = 0; u < UNR; ++u) v[u] = c + u < c1 ? chunk_cnt[(c + u) * El + e] : 0;
#pragma unroll
            for (int u = 0; u < UNR; ++u)
                if (c + u < c1) {
                    chunk_cnt[(c + u) * El + e] = row;
                    row += v[u];
                }
        }
    }
}

// The scan for at most 64 local experts: lane = expert, each of the 16
// wavefronts owns a contiguous range of chunks and walks its rows (El
// consecutive counts: one coalesced load per row, 8 rows in flight).  Wave
// totals per expert give each wave's starting row; the exclusive scan over
// experts fits one wavefront, so every wave computes it itself.
__global__ __launch_bounds__(1024) void scan_narrow_kernel(int32_t *__restrict__ chunk_cnt, int64_t nchunks,
                                                           int El, int32_t *__restrict__ counts,
                                                           int32_t *__restrict__ offsets)
{
    constexpr int UNR = 8;
    __shared__ int32_t wtot[16][64];
    const int t = threadIdx.x, lane = t & 63, wv = t >> 6, nw = blockDim.x >> 6;
    const bool act = lane < El;
    const int64_t per = (nchunks + nw - 1) / nw;
    const int64_t c0 = wv * per < nchunks ? wv * per : nchunks;
    const int64_t c1 = c0 + per < nchunks ? c0 + per : nchunks;
    int32_t run = 0;
    for (int64_t c = c0; c < c1; c += UNR) {
        int32_t v[UNR];
#pragma unroll
        for (int u = 0; u < UNR; ++u) v[u] = act && c + u < c1 ? chunk_cnt[(c + u) * El + lane] : 0;
#pragma unroll
        for (int u = 0; u < UNR; ++u) run += v[u];
    }
    wtot[wv][lane] = run;
    __syncthreads();
    int32_t before_w = 0, total = 0;
    for (int w = 0; w < nw; ++w) {
        const int32_t x = wtot[w][lane];
        before_w += w < wv ? x : 0;
        total += x;
    }
    // exclusive scan of the expert totals over the lanes (experts)
    int32_t incl = total;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int32_t o = __shfl_up(incl, off, 64);
        if (lane >= off) incl += o;
    }
    const int32_t eexcl = incl - total;
    if (wv == 0 && act) {
        counts[lane] = total;
        offsets[lane] = eexcl;
        if (lane == El - 1) offsets[El] = incl;  // total over all experts
    }
    int32_t row = eexcl + before_w;
    for (int64_t c = c0; c < c1; c += UNR) {
        int32_t v[UNR];
#pragma unroll
        for (int u = 0; u < UNR; ++u) v[u] = act && c + u < c1 ? chunk_cnt[(c + u) * El + lane] : 0;
#pragma unroll
        for (int u = 0; u < UNR; ++u)
            if (act && c + u < c1) {
                chunk_cnt[(c + u) * El + lane] = row;
                row += v[u];
            }
    }
}

__global__ __launch_bounds__(1024) void permute_small_kernel(const int32_t *__restrict__ ids, int64_t npairs,
                                                             int e0, int El, int nbits,
                                                             int32_t *__restrict__ counts,
                                                             int32_t *__restrict__ offsets,
                                                             int32_t *__restrict__ row_to_pair,
                                                             int32_t *__restrict__ pair_to_row)
{
    permute_small_body(ids, npairs, e0, El, nbits, counts, offsets, row_to_pair, pair_to_row);
}

template <int ROUNDS>
__global__ __launch_bounds__(64) void scatter_kernel(const int32_t *__restrict__ ids, int64_t npairs,
                                                     int e0, int El, int nbits,
                                                     const int32_t *__restrict__ chunk_base,
                                                     int32_t *__restrict__ row_to_pair,
                                                     int32_t *__restrict__ pair_to_row)
{
    constexpr int CHUNK = ROUNDS * 64;
    extern __shared__ int32_t next_row[];
    const int lane = threadIdx.x;
    const int64_t c = blockIdx.x;
    for (int i = lane; i < El; i += 64) next_row[i] = chunk_base[c * El + i];
    const int64_t base = c * CHUNK;
    int32_t v[ROUNDS];
#pragma unroll
    for (int r = 0; r < ROUNDS; ++r) {
        int64_t p = base + r * 64 + lane;
        v[r] = p < npairs ? ids[p] : -1;
    }
    __syncthreads();
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    for (int r = 0; r < ROUNDS; ++r) {
        const int64_t p = base + r * 64 + lane;
        const bool valid = p < npairs;
        const int le = valid ? local_index(v[r], e0, El) : El + 1;
        uint64_t peers = ~0ull;
        for (int b = 0; b < nbits; ++b) {
            const bool bit = (le >> b) & 1;
            const uint64_t bal = __ballot(bit);
            peers &= bit ? bal : ~bal;
        }
        const int rank = __popcll(peers & below);
        if (le < El) {
            const int32_t row = next_row[le] + rank;
            row_to_pair[row] = (int32_t)p;
            pair_to_row[p] = row;
        } else if (valid) {
            pair_to_row[p] = -1;
        }
        __syncthreads();
        if (le < El && rank == 0) next_row[le] += __popcll(peers);
        __syncthreads();
    }
}

template <int ROUNDS>
__global__ __launch_bounds__(256) void scan_scatter_kernel(const int32_t *__restrict__ ids, int64_t npairs,
                                                          int e0, int El, int nbits,
                                                          const int32_t *__restrict__ chunk_cnt, int64_t nchunks,
                                                          int32_t *__restrict__ counts,
                                                          int32_t *__restrict__ offsets,
                                                          int32_t *__restrict__ row_to_pair,
                                                          int32_t *__restrict__ pair_to_row)
{
    scan_scatter_body<ROUNDS>(ids, npairs, e0, El, nbits, chunk_cnt, nchunks, counts, offsets, row_to_pair,
                              pair_to_row, blockIdx.x);
}

__global__ __launch_bounds__(256) void gather_kernel(const uint16_t *__restrict__ x, int H, int k,
                                                     const int32_t *__restrict__ row_to_pair,
                                                     const int32_t *__restrict__ offsets, int El,
                                                     int64_t cap, uint16_t *__restrict__ x_perm)
{
    int64_t n = offsets[El];
    if (n > cap) n = cap;
    const int vecs = H / 8;
    for (int64_t r = blockIdx.x; r < n; r += gridDim.x) {
        const int64_t t = row_to_pair[r] / k;
        const uint4 *src = reinterpret_cast<const uint4 *>(x + t * H);
        uint4 *dst = reinterpret_cast<uint4 *>(x_perm + r * H);
        for (int i = threadIdx.x; i < vecs; i += 256) dst[i] = src[i];
    }
}

// Scratch of the allocation-free entry point: the per-chunk histograms that
// the caller's workspace holds otherwise.  Each GPU holds its own copy for
// the life of the process; in host code the name is not a device address,
// so the kernels get it through permute_scratch().
static __device__ __align__(256) int32_t scratch[MOE_PERMUTE_SCRATCH_BYTES / sizeof(int32_t)];

constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mtx;
int32_t *g_scratch[MAX_DEVICES];

}  // namespace

hipError_t permute_scratch(int32_t **ptr)
{
    int dev = 0;
    hipError_t err = hipGetDevice(&dev);
    if (err != hipSuccess) return err;
    if (dev < 0 || dev >= MAX_DEVICES) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mtx);
    if (g_scratch[dev] == nullptr) {
        // once per device, with that device current: the address of this
        // device's copy of the array
        void *p = nullptr;
        err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (err != hipSuccess) return err;
        if (p == nullptr) return hipErrorInvalidSymbol;
        g_scratch[dev] = static_cast<int32_t *>(p);
    }
    *ptr = g_scratch[dev];
    return hipSuccess;
}

int64_t permute_chunks(int64_t T, int k, int El) { return ceil_div(T * k, chunk_pairs(T * k, El)); }

hipError_t launch_permute(const int32_t *ids, int64_t T, int k, int e0, int El, int32_t *counts,
                          int32_t *offsets, int32_t *row_to_pair, int32_t *pair_to_row,
                          const uint16_t *x, int H, uint16_t *x_perm, int64_t cap, int32_t *ws,
                          hipStream_t s)
{
    const int64_t npairs = T * k;
    const int64_t nchunks = permute_chunks(T, k, El);
    const bool short_chunks = chunk_pairs(npairs, El) == 256;
    int nbits = 0;
    while ((1 << nbits) < El + 2) ++nbits;  // distinguishes 0..El+1
    hipError_t err;
    if (npairs > 0 && npairs <= SMALL_PAIRS && El <= 64 && npairs * (nbits + 2) <= SMALL_WORK) {
        KernelTimer timer(MOE_K_PERMUTE, s);
        permute_small_kernel<<<dim3(1), dim3(1024), 0, s>>>(ids, npairs, e0, El, nbits, counts, offsets,
                                                             row_to_pair, pair_to_row);
        if ((err = hipGetLastError()) != hipSuccess) return err;
    } else {
        KernelTimer timer(MOE_K_PERMUTE, s);
        if (nchunks > 0) {
            if (short_chunks)
                count_kernel<4><<<dim3((unsigned)nchunks), dim3(64), El * sizeof(int32_t), s>>>(
                    ids, npairs, e0, El, ws);
            else
                count_kernel<16><<<dim3((unsigned)nchunks), dim3(64), El * sizeof(int32_t), s>>>(
                    ids, npairs, e0, El, ws);
            if ((err = hipGetLastError()) != hipSuccess) return err;
        }
        if (El <= 64 && nchunks > 0 && nchunks <= SCAN_SCATTER_MAX_CHUNKS) {
            // scan and scatter in one launch
            const unsigned blocks = (unsigned)ceil_div(nchunks, 4);
            if (short_chunks)
                scan_scatter_kernel<4><<<dim3(blocks), dim3(256), 0, s>>>(ids, npairs, e0, El, nbits, ws, nchunks,
                                                                          counts, offsets, row_to_pair, pair_to_row);
            else
                scan_scatter_kernel<16><<<dim3(blocks), dim3(256), 0, s>>>(ids, npairs, e0, El, nbits, ws, nchunks,
                                                                           counts, offsets, row_to_pair, pair_to_row);
            if ((err = hipGetLastError()) != hipSuccess) return err;
        } else {
            if (El <= 64) {
                scan_narrow_kernel<<<dim3(1), dim3(1024), 0, s>>>(ws, nchunks, El, counts, offsets);
            } else {
                int L = 1;
                while (L < 64 && 2 * L * El <= 1024) L *= 2;
                scan_kernel<<<dim3(1), dim3(1024), 0, s>>>(ws, nchunks, El, L, counts, offsets);
            }
            if ((err = hipGetLastError()) != hipSuccess) return err;
            if (nchunks > 0) {
                if (short_chunks)
                    scatter_kernel<4><<<dim3((unsigned)nchunks), dim3(64), El * sizeof(int32_t), s>>>(
                        ids, npairs, e0, El, nbits, ws, row_to_pair, pair_to_row);
                else
                    scatter_kernel<16><<<dim3((unsigned)nchunks), dim3(64), El * sizeof(int32_t), s>>>(
                        ids, npairs, e0, El, nbits, ws, row_to_pair, pair_to_row);
                if ((err = hipGetLastError()) != hipSuccess) return err;
            }
        }
    }
    if (x_perm != nullptr && cap > 0) {
        KernelTimer timer(MOE_K_GATHER, s);
        int64_t blocks = cap < 4096 ? cap : 4096;
        gather_kernel<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(x, H, k, row_to_pair, offsets, El,
                                                                   cap, x_perm);
        if ((err = hipGetLastError()) != hipSuccess) return err;
    }
    return hipSuccess;
}

}  // namespace moe
