// Permutation device code shared by the permutation kernels and the fused
// layer kernels (see permute.hip for the overall method).
#pragma once
#include "moe_internal.h"

namespace moe {
namespace permute_dev {

// Chunk size: short chunks give more wavefronts (the scatter walks its
// chunk 64 pairs at a time, in order), long ones fewer histogram rows.
inline int chunk_pairs(int64_t npairs, int El) { return npairs * El <= ((int64_t)1 << 24) ? 256 : 1024; }

__device__ __forceinline__ int local_index(int32_t id, int e0, int El)
{
    int d = id - e0;
    return (d >= 0 && d < El) ? d : El;  // El marks a pair owned elsewhere
}

// The whole permutation in one workgroup, for at most SMALL_PAIRS pairs and
// 64 local experts: each of the 16 wavefronts owns a contiguous run of pairs
// (kept in registers), counts it per expert with the same ballot ranking as
// the scatter, the per-(wave, expert) bases are scanned in LDS, and the
// wavefronts then place their pairs in order.  Same stable result as the
// multi-kernel path.  One workgroup's time grows with the pairs and the
// ballots per pair (bits of the local expert index) while the multi-kernel
// path costs about two launches, so moe_permute's workgroup takes at most
// SMALL_WORK pair-steps (measured: 8192 pairs over 1 local expert and 4096
// over 32 are faster here, 8192 over 8 in two launches).  The layer forward,
// whose two-launch path also routes and schedules, has its own threshold.
constexpr int SMALL_PAIRS = 16 * 1024;
constexpr int64_t SMALL_WORK = 32 * 1024;
// (A device function run by a whole block of 1024 threads.)
__device__ __forceinline__ void permute_small_body(const int32_t *__restrict__ ids, int64_t npairs, int e0,
                                                   int El, int nbits, int32_t *__restrict__ counts,
                                                   int32_t *__restrict__ offsets,
                                                   int32_t *__restrict__ row_to_pair,
                                                   int32_t *__restrict__ pair_to_row)
{
    constexpr int MAXR = SMALL_PAIRS / 1024;  // rounds of 64 pairs per wave, at most
    __shared__ int32_t base[16][64];
    const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
    const int64_t per = ((npairs + 15) / 16 + 63) / 64 * 64;  // pairs per wave, whole rounds
    const int64_t p0 = wv * per;
    const int rounds = (int)((per + 63) / 64);
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    int32_t le[MAXR];
#pragma unroll
    for (int r = 0; r < MAXR; ++r) {
        const int64_t p = p0 + r * 64 + lane;
        le[r] = r < rounds && p < npairs ? local_index(ids[p], e0, El) : El + 1;
    }
    if (lane < El) base[wv][lane] = 0;
    __syncthreads();
    // per-(wave, expert) counts: the first lane of each group of equal
    // experts in a round adds the group's size
    auto peers_of = [&](int x) {
        uint64_t m = ~0ull;
        for (int b = 0; b < nbits; ++b) {
            const bool bit = (x >> b) & 1;
            const uint64_t bal = __ballot(bit);
            m &= bit ? bal : ~bal;
        }
        return m;
    };
#pragma unroll
    for (int r = 0; r < MAXR; ++r) {
        if (r >= rounds) break;
        const uint64_t peers = peers_of(le[r]);
        if (le[r] < El && __popcll(peers & below) == 0) base[wv][le[r]] += __popcll(peers);
    }
    __syncthreads();
    // expert totals, their exclusive scan (one wavefront), and each wave's
    // first row per expert
    if (wv == 0) {
        int32_t total = 0;
        if (lane < El)
            for (int w = 0; w < 16; ++w) total += base[w][lane];
        int32_t incl = total;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int32_t o = __shfl_up(incl, off, 64);
            if (lane >= off) incl += o;
        }
        if (lane < El) {
            counts[lane] = total;
            offsets[lane] = incl - total;
            if (lane == El - 1) offsets[El] = incl;
            int32_t row = incl - total;
            for (int w = 0; w < 16; ++w) {
                const int32_t c = base[w][lane];
                base[w][lane] = row;
                row += c;
            }
        }
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < MAXR; ++r) {
        if (r >= rounds) break;
        const int64_t p = p0 + r * 64 + lane;
        const uint64_t peers = peers_of(le[r]);
        const int rank = __popcll(peers & below);
        if (le[r] < El) {
            const int32_t row = base[wv][le[r]] + rank;
            row_to_pair[row] = (int32_t)p;
            pair_to_row[p] = row;
        } else if (le[r] == El) {
            pair_to_row[p] = -1;
        }
        // a wave's own LDS row: its leaders bump it after every lane read it
        __builtin_amdgcn_wave_barrier();
        if (le[r] < El && rank == 0) base[wv][le[r]] += __popcll(peers);
        __builtin_amdgcn_wave_barrier();
    }
}

// Steps 2 and 3 in one launch (at most 64 local experts and
// SCAN_SCATTER_MAX_CHUNKS chunks): a block of four
// wavefronts scatters four chunks, one each, after rebuilding from the chunk
// histograms what the scan would have handed it: each expert's total (hence
// its first row) and the pairs of that expert in the chunks before its own.
// Every block reads the whole histogram table (a few KB, from L2), which is
// cheaper than a separate single-workgroup scan launch between count and
// scatter.  Block 0 also writes counts and offsets.  The table reads of all
// blocks together grow with the square of the chunk count, so above
// SCAN_SCATTER_MAX_CHUNKS chunks (about 1M pairs in 256-pair chunks, 4M in
// 1024-pair chunks: 4096 chunks x 64 experts x 4 B = 1 MB read by each of
// 1024 blocks) the separate scan and scatter launches take over.
constexpr int64_t SCAN_SCATTER_MAX_CHUNKS = 4096;
// (A device function run by a block of 256 threads as scan block `blk`.)
template <int ROUNDS>
__device__ __forceinline__ void scan_scatter_body(const int32_t *__restrict__ ids, int64_t npairs, int e0,
                                                  int El, int nbits, const int32_t *__restrict__ chunk_cnt,
                                                  int64_t nchunks, int32_t *__restrict__ counts,
                                                  int32_t *__restrict__ offsets,
                                                  int32_t *__restrict__ row_to_pair,
                                                  int32_t *__restrict__ pair_to_row, int64_t blk)
{
    // UNR loads in flight per thread and pass: each pass waits for its
    // loads, so the passes are memory round trips in a row (a 256-chunk
    // histogram of 16 experts is one pass)
    constexpr int CHUNK = ROUNDS * 64, UNR = 16;
    __shared__ int32_t part_tot[256], part_bef[256];
    __shared__ int32_t next_row[4][64];
    const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
    const int64_t c_first = blk * 4;
    // 1. column sums of the histogram table: thread t sums expert t % El over
    //    chunks t / El, t / El + S, ... (S = 256 / El groups), all chunks and
    //    those before this block's first
    const int S = 256 / El;
    int32_t tot = 0, bef = 0;
    if (t < S * El) {
        const int e = t % El;
        for (int64_t c = t / El; c < nchunks; c += (int64_t)S * UNR) {
            int32_t v[UNR];
#pragma unroll
            for (int u = 0; u < UNR; ++u) {
                const int64_t cu = c + (int64_t)u * S;
                v[u] = cu < nchunks ? chunk_cnt[cu * El + e] : 0;
            }
#pragma unroll
            for (int u = 0; u < UNR; ++u) {
                tot += v[u];
                bef += c + (int64_t)u * S < c_first ? v[u] : 0;
            }
        }
    }
    part_tot[t] = tot;
    part_bef[t] = bef;
    __syncthreads();
    // 2. per expert (one lane each): its total, the exclusive scan of the
    //    totals over the experts (its first row), and this block's first row
    if (wv == 0) {
        int32_t total = 0, before = 0;
        if (lane < El)
            for (int g = 0; g < S; ++g) {
                total += part_tot[g * El + lane];
                before += part_bef[g * El + lane];
            }
        int32_t incl = total;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int32_t o = __shfl_up(incl, off, 64);
            if (lane >= off) incl += o;
        }
        const int32_t eexcl = incl - total;
        if (lane < El) {
            if (blk == 0) {
                counts[lane] = total;
                offsets[lane] = eexcl;
                if (lane == El - 1) offsets[El] = incl;  // total over all experts
            }
            next_row[0][lane] = eexcl + before;
        }
    }
    __syncthreads();
    // 3. wave w scatters chunk c_first + w: its first row per expert is the
    //    block's plus the pairs of the block's chunks before it
    int32_t row = lane < El ? next_row[0][lane] : 0;
    __syncthreads();  // every wave has the block's rows before wave 0 reuses its LDS row
    const int64_t c = c_first + wv;
    if (c >= nchunks) return;
    if (lane < El) {
        // the counts of the block's chunks before this one (at most 3),
        // loaded together
        int32_t before[3];
#pragma unroll
        for (int q = 0; q < 3; ++q) before[q] = c_first + q < c ? chunk_cnt[(c_first + q) * El + lane] : 0;
        row += before[0] + before[1] + before[2];
        next_row[wv][lane] = row;
    }
    __builtin_amdgcn_wave_barrier();
    const int64_t base = c * CHUNK;
    int32_t v[ROUNDS];
#pragma unroll
    for (int r = 0; r < ROUNDS; ++r) {
        const int64_t p = base + r * 64 + lane;
        v[r] = p < npairs ? ids[p] : -1;
    }
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
            const int32_t row = next_row[wv][le] + rank;
            row_to_pair[row] = (int32_t)p;
            pair_to_row[p] = row;
        } else if (valid) {
            pair_to_row[p] = -1;
        }
        // the wave's own LDS row: its leaders bump it after every lane read it
        __builtin_amdgcn_wave_barrier();
        if (le < El && rank == 0) next_row[wv][le] += __popcll(peers);
        __builtin_amdgcn_wave_barrier();
    }
}

}  // namespace permute_dev
}  // namespace moe
