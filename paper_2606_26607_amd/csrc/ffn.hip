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
#include <mutex>
#include <type_traits>
#include <vector>

#include "moe_internal.h"
#include "permute_dev.h"
#include "route_dev.h"

namespace moe {
namespace {

constexpr int BM = 64, BN = 64, BK = 64;  // the general kernel (any K multiple of 8)
constexpr int KCH = BK / 8;               // 16-byte chunks per tile row

__device__ __forceinline__ int64_t clamp_row(int32_t v, int64_t cap)
{
    int64_t r = v < 0 ? 0 : v;
    return r > cap ? cap : r;
}

// Row range of expert e in one call's row space: a routed expert e < El holds
// [offsets[e], offsets[e+1]) clamped to [0, cap]; the shared expert (e == El,
// present when the call has shared rows) holds [cap, cap + shared_rows).
__device__ __forceinline__ int64_t expert_begin(const int32_t *__restrict__ offsets, int El, int64_t cap, int e)
{
    return e < El ? clamp_row(offsets[e], cap) : cap;
}

__device__ __forceinline__ int64_t expert_end(const int32_t *__restrict__ offsets, int El, int64_t cap,
                                              int64_t shared_rows, int e)
{
    return e < El ? clamp_row(offsets[e + 1], cap) : cap + shared_rows;
}

// A read of metadata that earlier launches wrote and the grouped GEMM only
// reads (the schedule's tile lists and cuts, the experts' row offsets),
// through the constant address space: it becomes a scalar load, which waits
// on the scalar memory counter.  A vector load would wait on the vector
// counter, which also counts the workgroup's output stores of its previous
// tile, so each lookup at a tile change would wait for those stores to land.
template <class T>
__device__ __forceinline__ T ld_meta(const T *p)
{
    return *(const __attribute__((address_space(4))) T *)p;
}

// SwiGLU of one gate/up pair: silu(g) * u = g / (1 + e^-g) * u, with the
// hardware reciprocal (the result is rounded to bf16).
__device__ __forceinline__ float silu_mul(float g, float u)
{
    return g * __builtin_amdgcn_rcpf(1.0f + __expf(-g)) * u;
}

// Large-tile launches split K only from this many K-slices per tile.
constexpr int SPLIT_MIN_NK = 128;
// The small-row class comes in two heights, chosen per launch by the
// schedule: 64-row tiles (decode: experts of a few rows) and 128-row tiles
// (prefill leftovers of 65-128 rows, which would otherwise take two 64-row
// tiles that each stream the expert's weights).  Each has a largest expert
// it takes whole and the time of one of its K-slices relative to a
// large-tile K-slice, in twentieths: cost_num for a slice of a stream-K
// piece, its share of the piece's partial-sum traffic included, and
// whole_num for a slice of a tile run whole (measured on the prefill
// workloads: a small-row slice is bound by its weight rows, a 256-row one by
// MFMA).  Every tile also pays a prologue (the first operand slices arrive
// from memory) and an epilogue (the output leaves through LDS): about
// LARGE_OVH large slices for a large tile, SMALL_WHOLE_OVH twentieths of one
// for a small-row tile run whole.
constexpr int SMALL_COST_DEN = 20;
struct SmallKind {
    int rows, max_rows, cost_num, whole_num;
};
constexpr SmallKind SMALL64{64, 96, 11, 7};
constexpr SmallKind SMALL128{128, 128, 11, 13};
constexpr int LARGE_OVH = 5, SMALL_WHOLE_OVH = 50;

// Whole small-row tiles of nk K-slices that fit in the time of one large tile
// (nk < 2^25: operands are addressed with 32-bit byte offsets).
__host__ __device__ __forceinline__ int whole_fit(int nk, int whole_num)
{
    return SMALL_COST_DEN * (nk + LARGE_OVH) / (whole_num * nk + SMALL_WHOLE_OVH);
}

// Block-wide exclusive scan of one value per thread (blocks of whole waves,
// at most 1024 threads); returns the exclusive prefix and writes the total
// to *total (last thread).
__device__ __forceinline__ int32_t block_exscan(int32_t v, int32_t *wsum, int32_t *total)
{
    const int e = threadIdx.x, lane = e & 63, wv = e >> 6;
    int32_t incl = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        int32_t o = __shfl_up(incl, off, 64);
        if (lane >= off) incl += o;
    }
    if (lane == 63) wsum[wv] = incl;
    __syncthreads();
    int32_t before = 0;
    for (int i = 0; i < wv; ++i) before += wsum[i];
    if (e == (int)blockDim.x - 1) *total = before + incl;
    __syncthreads();
    return before + incl - v;
}

// The same for N values at once (independent shuffle chains run
// interleaved), in place; totals to tot[0..N-1].
template <int N>
__device__ __forceinline__ void block_exscan_n(int32_t (&v)[N], int32_t (*wsum)[N], int32_t *tot)
{
    const int e = threadIdx.x, lane = e & 63, wv = e >> 6;
    int32_t incl[N];
#pragma unroll
    for (int i = 0; i < N; ++i) incl[i] = v[i];
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        int32_t o[N];
#pragma unroll
        for (int i = 0; i < N; ++i) o[i] = __shfl_up(incl[i], off, 64);
        if (lane >= off) {
#pragma unroll
            for (int i = 0; i < N; ++i) incl[i] += o[i];
        }
    }
    if (lane == 63) {
#pragma unroll
        for (int i = 0; i < N; ++i) wsum[wv][i] = incl[i];
    }
    __syncthreads();
    int32_t before[N];
#pragma unroll
    for (int i = 0; i < N; ++i) before[i] = 0;
    for (int w = 0; w < wv; ++w) {
#pragma unroll
        for (int i = 0; i < N; ++i) before[i] += wsum[w][i];
    }
    if (e == (int)blockDim.x - 1) {
#pragma unroll
        for (int i = 0; i < N; ++i) tot[i] = before[i] + incl[i];
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < N; ++i) v[i] = before[i] + incl[i] - v[i];
}

// Shape of both GEMMs as the schedule's cost model sees it: output tiles per
// m-tile (n_tiles) and K-slices per tile (nk).
struct SchedShape {
    int nt_gu, nk_gu, nt_dn, nk_dn, grid;
    int wfit[2][2];      // [GEMM][64- or 128-row tiles]: whole_fit of the GEMM's nk
    float whole[2][2];   // ... and whole_time
};

// Where a GEMM's ts small-row tiles run next to its tl large tiles on a grid
// of G persistent workgroups:
//   SM_PIECES_IDLE: stream-K over the workgroups the large tiles leave idle
//     in their last round, when its slices (cost_num / SMALL_COST_DEN of a
//     large slice each) add up to at most one large tile per idle workgroup;
//   SM_WHOLE_IDLE: else whole tiles dealt round robin over the idle
//     workgroups, when as many fit there as take one large tile's time each
//     (whole tiles pay no partial sums);
//   SM_WHOLE_ALL: else, with at most one tile per workgroup, whole tiles
//     dealt over all workgroups (the idle ones first) after their large
//     tiles, when one whole tile takes less than a stream-K share plus the
//     fixed cost of a stream-K piece (prologue and partial sums);
//   SM_PIECES_ALL: else stream-K over all workgroups after their large tiles;
//   SM_PIECES_PAIR: with no idle workgroups and at most G/2 tiles, stream-K
//     over 2 * ts workgroups (spread over the dies) after their large tiles,
//     so that each tile is cut into two halves of K, when that is the
//     cheapest of the three (two pieces pay the fixed cost of a piece and
//     one partial each, PAIR_OVH large slices in all).
// extra = what the small-row work adds to the large tiles' rounds, in units
// of one large-tile K-slice.
enum SmallMode { SM_PIECES_IDLE, SM_WHOLE_IDLE, SM_WHOLE_ALL, SM_PIECES_ALL, SM_PIECES_PAIR };

// x / g (rounded down) for 0 <= x < 2^53 and g >= 1, in 32 bits whenever x
// fits (it always does in practice).  A wider x takes a double-precision
// quotient, exact in its integer part to within one, corrected to the
// floor: an integer 64-bit division expands to about a hundred instructions
// at every use, and the schedule's code runs once per launch from a cold
// instruction cache.
__device__ __forceinline__ int64_t div_g(int64_t x, int g)
{
    if (x <= 0x7fffffff) return (int64_t)((uint32_t)x / (uint32_t)g);
    int64_t q = (int64_t)((double)x / (double)g);
    q -= q * g > x ? 1 : 0;
    q += (q + 1) * g <= x ? 1 : 0;
    return q;
}
constexpr float PIECE_OVH = 8.0f;  // fixed cost of a stream-K piece, in large slices
constexpr float PAIR_OVH = 3.0f;   // fixed cost of splitting a whole small-row tile in two, in large slices
struct SmallPlan {
    SmallMode mode;
    int idle;
    float extra;
};

// Time of one whole small-row tile of nk K-slices, in large slices.
__host__ __device__ __forceinline__ float whole_time(int nk, int whole_num)
{
    return (float)(whole_num * nk + SMALL_WHOLE_OVH) / (float)SMALL_COST_DEN;
}

// The per-GEMM constants of the plan: wfit = whole_fit(nk, kind.whole_num),
// whole = whole_time(nk, kind.whole_num) (worked out once, on the host for
// the schedule).
__device__ __forceinline__ SmallPlan small_plan(int64_t tl, int64_t ts, int nk, int G, int cost_num, int wfit,
                                                float whole)
{
    const bool large_dp = !(tl < G && nk >= SPLIT_MIN_NK);
    const int rest = (int)(tl - div_g(tl, G) * G);
    const int idle = (large_dp && rest) ? G - rest : 0;
    if (ts == 0) return SmallPlan{SM_PIECES_ALL, idle, 0.f};
    if (idle && (int64_t)cost_num * ts <= (int64_t)SMALL_COST_DEN * idle) return SmallPlan{SM_PIECES_IDLE, idle, 0.f};
    if (idle && ts <= (int64_t)idle * wfit) return SmallPlan{SM_WHOLE_IDLE, idle, 0.f};
    const float pieces = (float)cost_num / (float)SMALL_COST_DEN * (float)ts * (float)nk / (float)G;
    const float pair = 0.5f * whole + PAIR_OVH;
    if (idle == 0 && 2 * ts <= G && pair < whole && pair < pieces + PIECE_OVH)
        return SmallPlan{SM_PIECES_PAIR, idle, pair};
    if (ts <= G && whole < pieces + PIECE_OVH) return SmallPlan{SM_WHOLE_ALL, idle, ts > idle ? whole : 0.f};
    return SmallPlan{SM_PIECES_ALL, idle, pieces};
}

// Estimated time of one GEMM, in units of one large-tile K-slice on one
// workgroup, for tl large and ts small-row tiles of nk K-slices: rounds of
// large tiles (or their stream-K share, with its partial-sum traffic, when
// there are fewer tiles than workgroups and K is long) ...
__device__ __forceinline__ float large_cost(int64_t tl, int nk, int grid)
{
    const float t = (float)tl, g = (float)grid;
    const bool split = tl < grid && nk >= SPLIT_MIN_NK;
    const int64_t rounds = div_g(tl, grid);
    const int rest = (int)(tl - rounds * grid);
    float c = 0.f;
    if (tl > 0 && split) {
        c = 1.25f * t * (float)nk / g;
    } else if (tl > 0) {
        // a last round with a fraction f of the workgroups busy takes about
        // 0.6 + 0.4 f of a full one (less contention for L2 and HBM)
        c = (float)rounds * (float)nk;
        if (rest) c += (0.6f + 0.4f * (float)rest / g) * (float)nk;
    }
    return c;
}

// ... plus what its small-row work adds (small_plan); c = large_cost(tl, ...).
__device__ __forceinline__ float gemm_cost(float c, int64_t tl, int64_t ts, int nk, int grid, int cost_num,
                                           int wfit, float whole, bool tall)
{
    const SmallPlan p = small_plan(tl, ts, nk, grid, cost_num, wfit, whole);
    // 128-row tiles not in stream-K pieces over the whole grid: there the
    // last contributor of each tile reads back larger partials alone
    // (measured slower than 64-row tiles)
    if (tall && ts > 0 && p.mode == SM_PIECES_ALL) return 3.0e38f;
    return c + p.extra;
}

constexpr int NC_SCHED = 10;  // base candidates: smax 96 or 128 x leftover threshold 0 .. 128
constexpr int ND_SCHED = 8;   // ... each also with up to 7 more m-tiles of the largest expert moved

// Tile schedule of the grouped FFN, chosen for each GEMM on its own.  An
// expert's rows [a, b) are cut at split[e]: rows [a, split) go to the
// large-tile class (m-tiles of bm rows), rows [split, b) to the small-row
// class.  An expert with at most smax rows (96 or 128) is all small.  A
// larger one may give its leftover rows after whole large tiles to the small
// class (none, or those of at most 32, 64, 96 or 128 rows): a nearly empty
// large tile costs as much as a full one, while small-row work fits where the
// large tiles leave workgroups idle.  The largest expert may also give its
// last D = 1 .. 7 large m-tiles, only where that saves a round of large
// tiles (a sparse last round costs about as much as a full one): the fewest
// such D is a candidate beside D = 0.  Each GEMM takes the candidate (smax,
// threshold, D) and small tile height (64 or 128 rows) of the lowest
// estimated time (gemm_cost); small = false disables the small class.
//   pre_l[g][e] / pre_s[g][e] = m-tiles of the large / small class of GEMM g
//   (0 gate-up, 1 down) for the experts before e, [ne] = totals (ne experts:
//   the routed ones, then the shared one if the call has shared rows),
//   pre_s[g][ne + 1] = the GEMM's small tile height; split[g][e] its cut.
// Also clears the split-K tile counters (no memset node is needed, so the
// chain stays graph-capturable).
struct SchedOut {
    int32_t *pre_l[2], *pre_s[2], *split[2];
    int4 *mt[2];  // per small m-tile: expert, first row, end row
};

// (A device function run by one block: one thread per expert, at least four
// waves, whole waves; NE_MAX bounds the experts, the shared one included.
// offsets may point to LDS.)
template <int NE_MAX>
__device__ __forceinline__ void schedule_body(const int32_t *__restrict__ offsets, int El, int64_t cap,
                                              int64_t shared_rows, int bm, bool small, const SchedShape &sh,
                                              const SchedOut &out, int32_t *__restrict__ counters,
                                              int64_t n_counters)
{
    constexpr int NT = NC_SCHED / 2;  // leftover thresholds 0, 32, 64, 96, 128
    constexpr int NC = NC_SCHED;
    __shared__ int32_t wsum[16][4];
    __shared__ int32_t vals[NE_MAX][3 * NC + 1];  // per expert: its tiles of every base candidate, its rows
    __shared__ int32_t tot[3 * NC];
    __shared__ int32_t ptot[4];
    __shared__ int32_t big[2];  // the largest expert and its rows
    __shared__ unsigned long long kmin[4];
    // one thread per expert, at least four waves, whole waves (the launch
    // sizes the block)
    const int e = threadIdx.x, lane = e & 63, wv = e >> 6;
    // experts: the El routed ones, then the shared one when there are shared
    // rows; rows fit int32 (cap + shared rows < 2^31 is checked on the host)
    const int ne = El + (shared_rows > 0 ? 1 : 0);
    int32_t a = 0, n = 0;
    if (e < ne) {
        a = (int32_t)expert_begin(offsets, El, cap, e);
        const int32_t b = (int32_t)expert_end(offsets, El, cap, shared_rows, e);
        n = b > a ? b - a : 0;
    }
    // for base candidate c (smax = c / NT ? 128 : 96, threshold 32 * (c % NT)):
    // large m-tiles (x) and the rows that go to the small class (y)
    auto rows_for = [&](int32_t rows, int c) {
        const int32_t whole = rows / bm, rest = rows - whole * bm;
        const int smax = c / NT ? SMALL128.max_rows : SMALL64.max_rows;
        const int th = 32 * (c % NT);
        int2 r = make_int2(0, 0);
        if (rows > 0 && small && rows <= smax) {
            r.y = rows;
        } else if (rows > 0) {
            if (small && rest > 0 && rest <= th) {
                r.x = whole;
                r.y = rest;
            } else {
                r.x = whole + (rest > 0);
            }
        }
        return r;
    };
    // ... and with D more m-tiles of the largest expert moved
    auto rows_moved = [&](int32_t rows, int2 r, int D) {
        if (D > 0 && r.x > 0) {
            r.x = r.x > D ? r.x - D : 0;
            r.y = rows - r.x * bm;
        }
        return r;
    };
    int cand[2] = {0, 0}, kinds = 0, L = -1;
    if (small) {
        // class totals of every base candidate: large m-tiles, small m-tiles
        // of 64 and of 128 rows; each expert writes its row, one thread per
        // column sums it (a few dozen experts typically: cheaper than
        // shuffle trees)
        if (e < NE_MAX) {  // rows of threads past the experts are never read
#pragma unroll
            for (int c = 0; c < NC; ++c) {
                const int2 r = rows_for(n, c);
                vals[e][3 * c] = r.x;
                vals[e][3 * c + 1] = (r.y + 63) / 64;
                vals[e][3 * c + 2] = (r.y + 127) / 128;
            }
            vals[e][3 * NC] = n;
        }
        __syncthreads();
        if (e < 3 * NC) {
            int32_t sum = 0;
            for (int i = 0; i < ne; ++i) sum += vals[i][e];
            tot[e] = sum;
        } else if (e == 3 * NC) {
            // the largest expert (ties: the lowest index), none when no
            // expert has rows
            int32_t m = 0, at = -1;
            for (int i = 0; i < ne; ++i) {
                const int32_t r = vals[i][3 * NC];
                if (r > m) {
                    m = r;
                    at = i;
                }
            }
            big[0] = at;
            big[1] = m;
        }
        __syncthreads();
        L = big[0];
        // Candidates of GEMM gi with small tile height tall ? 128 : 64 rows
        // on lanes 0 .. 19 of wave 2 * gi + tall: base candidate c = t / 2
        // (t = lane) with D = 0 (even t) or with the fewest moves D that
        // save a round of large tiles (odd t; none where that takes more
        // than ND_SCHED - 1 moves or more m-tiles than the largest expert
        // has).  Its key is the cost's bits (non-negative floats order as
        // integers), then the candidate as c * ND_SCHED + D, then the height
        // bit, so the least key over both waves of a GEMM is its cheapest
        // candidate and height (ties: smax 96, then fewer moves, then 64
        // rows).  One height per wave halves each lane's work (the costing
        // is a divergent chain of divisions and branches).  The wave index
        // is made uniform and the GEMM's shape selected field by field, so
        // the shape stays in scalar registers: indexed by a per-lane value,
        // it was read with vector loads from the argument segment, a memory
        // round trip in the costing's chain.
        unsigned long long key = ~0ull;
        const int wvu = __builtin_amdgcn_readfirstlane(wv);
        const int gi = wvu >> 1, tall = wvu & 1, t = lane;
        if (wvu < 4 && t < 2 * NC) {
            const int c = t / 2;
            const int nt = gi ? sh.nt_dn : sh.nt_gu, nk = gi ? sh.nk_dn : sh.nk_gu, g = sh.grid;
            const int wf = gi ? (tall ? sh.wfit[1][1] : sh.wfit[1][0]) : (tall ? sh.wfit[0][1] : sh.wfit[0][0]);
            const float wh = gi ? (tall ? sh.whole[1][1] : sh.whole[1][0]) : (tall ? sh.whole[0][1] : sh.whole[0][0]);
            const int64_t tl0 = tot[3 * c];
            int64_t tl = tl0, ts = tot[3 * c + 1 + tall];
            int D = 0;
            bool valid = true;
            if (t & 1) {
                const int64_t r0 = div_g(tl0 * nt + g - 1, g);  // rounds of large tiles
                const int xl = L >= 0 ? vals[L][3 * c] : 0;
                const int64_t dmin = r0 >= 1 ? tl0 - div_g((r0 - 1) * g, nt) : 0;
                valid = dmin >= 1 && dmin < ND_SCHED && dmin <= xl;
                if (valid) {
                    D = (int)dmin;
                    const int2 r = rows_moved(big[1], make_int2(xl, 0), D);
                    tl += r.x - xl;
                    ts += (r.y + (tall ? 127 : 63)) / (tall ? 128 : 64) - vals[L][3 * c + 1 + tall];
                }
            }
            if (valid) {
                // one inlined copy of the cost model for both heights
                const int cnum = tall ? SMALL128.cost_num : SMALL64.cost_num;
                const float cl = large_cost(tl * nt, nk, g);
                const float cost = gemm_cost(cl, tl * nt, ts * nt, nk, g, cnum, wf, wh, tall != 0);
                key = ((unsigned long long)__float_as_uint(cost) << 32) | ((unsigned)(c * ND_SCHED + D) << 1) |
                      (unsigned)tall;
            }
        }
        // the cheapest of each wave: a minimum over lanes 0 .. 31 (DPP within
        // rows, then the rows' results; the whole wave is active), then the
        // lesser of the GEMM's two waves
        if (wvu < 4) {
            key = route_dev::group_reduce<32>(key, [](unsigned long long a, unsigned long long b) { return a < b ? a : b; });
            if (t == 0) kmin[wvu] = key;
        }
        __syncthreads();
        for (int i = 0; i < 2; ++i) {
            const unsigned long long km = kmin[2 * i] < kmin[2 * i + 1] ? kmin[2 * i] : kmin[2 * i + 1];
            cand[i] = (int)((km & 0xffffffffu) >> 1);
            kinds |= (int)(km & 1) << i;
        }
    }
    int32_t v[4];
    int h[2], ms[2];
    int32_t cut[2];
    for (int gi = 0; gi < 2; ++gi) {
        int2 r = rows_for(n, cand[gi] / ND_SCHED);
        if (e == L) r = rows_moved(n, r, cand[gi] % ND_SCHED);
        cut[gi] = a + (n - r.y);
        if (small && e < ne) out.split[gi][e] = cut[gi];
        h[gi] = kinds & (1 << gi) ? SMALL128.rows : SMALL64.rows;
        v[2 * gi] = r.x;
        v[2 * gi + 1] = ms[gi] = (r.y + h[gi] - 1) / h[gi];
    }
    // prefixes of both GEMMs' large and small m-tiles
    block_exscan_n<4>(v, wsum, ptot);
    for (int gi = 0; gi < 2; ++gi) {
        if (e < ne) out.pre_l[gi][e] = v[2 * gi];
        if (e == 0) out.pre_l[gi][ne] = ptot[2 * gi];
        if (small) {
            if (e < ne) {
                out.pre_s[gi][e] = v[2 * gi + 1];
                // this expert's small m-tiles: rows [cut, end) in runs of h
                for (int j = 0; j < ms[gi]; ++j) {
                    const int32_t r0 = cut[gi] + j * h[gi], r1 = r0 + h[gi] < a + n ? r0 + h[gi] : a + n;
                    out.mt[gi][v[2 * gi + 1] + j] = make_int4(e, r0, r1, 0);
                }
            }
            if (e == 0) {
                out.pre_s[gi][ne] = ptot[2 * gi + 1];
                out.pre_s[gi][ne + 1] = h[gi];
            }
        }
    }
    // the GEMMs' split-K tile counters, cleared last: before a barrier,
    // the barrier's fence would wait for these stores to land
    for (int64_t i = e; i < n_counters; i += blockDim.x) counters[i] = 0;
}

__global__ __launch_bounds__(1024) void schedule_kernel(const int32_t *__restrict__ offsets, int El,
                                                        int64_t cap, int64_t shared_rows, int bm, bool small,
                                                        SchedShape sh, SchedOut out,
                                                        int32_t *__restrict__ counters, int64_t n_counters)
{
    schedule_body<1024>(offsets, El, cap, shared_rows, bm, small, sh, out, counters, n_counters);
}

// 256 threads = 4 waves in a 2x2 grid, each wave owns a 32x32 block of the
// BMxBN tile (two accumulators when gated).
template <bool GATED>
__global__ __launch_bounds__(256) void gemm_kernel(const uint16_t *__restrict__ A,
                                                   const int32_t *__restrict__ row_index, int kdiv,
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
                if (gr < r1 && kk < K) {
                    const int64_t src_row = row_index ? (int64_t)(row_index[gr] / kdiv) : gr;
                    v = *reinterpret_cast<const uint4 *>(A + src_row * K + kk);
                }
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
                if (GATED) v = silu_mul(v, acc_u[i]);
                C[row * N + col] = f32_to_bf16(v);
            }
        }
    }
}


// ---------------------------------------------------------------------------
// Large-tile kernel (K a multiple of 64, at least 128): BMxBN tiles (BN counts
// weight rows; a gated tile holds BN/2 gate rows and the BN/2 matching up
// rows), 8 waves (two per SIMD) in a WM x (8/WM) grid, each wave owning
// (BM/WM)x(BN*WM/8) of 32x32x16 MFMA blocks, accumulators in AGPRs.
//
// Operands move L2 -> LDS with buffer loads that write LDS directly (no VGPR
// staging) in BK=64 slices (128-byte row segments: whole L2 lines).  A
// (activations, mostly L2 hits) and B (weights, more misses) have separate
// rings: 2 A slots and 3 B slots fill the 160 KB of LDS, so while slice s is
// consumed the loads of A(s+1) and B(s+2) are in flight.  The loads are issued
// one per four MFMAs (A under k-steps 0-1, B under k-steps 2-3): a burst would
// stall the wave's in-order instruction stream behind the memory pipeline.
// Fragments of k-step kk+1 are read while the MFMAs of kk run, and the
// barrier that hands over to slice s+1 sits before the last k-step, so the
// next slice's first fragments are read under MFMAs too.  Buffer range
// checking returns zeros for rows past the expert's last row or past N.
// LDS rows are 128 bytes; 16-byte chunk c of row r sits at c ^ swz(r), so
// each 16-row (and 8-row) group read by one ds_read_b128 covers distinct
// banks.  The epilogue stages the bf16 tile in LDS and writes it with
// coalesced 16-byte stores.
// ---------------------------------------------------------------------------
constexpr int BIG_BK = 64;        // K per slice
constexpr int CPR = BIG_BK / 8;   // 16-byte chunks per LDS row
constexpr int RPI = 64 / CPR;     // rows per DMA instruction
static_assert(RPI == 8, "a lane's DMA row is lane / 8");

// RPI consecutive row indices from a 4-byte aligned address, as one scalar
// load (a read of metadata like ld_meta's).
typedef int32_t rows_t __attribute__((ext_vector_type(RPI), aligned(4)));
__device__ __forceinline__ rows_t ld_rows(const int32_t *p)
{
    return *(const __attribute__((address_space(4))) rows_t *)p;
}
constexpr int A_SLOTS = 2, B_SLOTS = 3;        // large tiles: A(s+1), B(s+2) in flight
constexpr int SA_SLOTS = 3, SB_SLOTS = 4;      // small-row tiles: A(s+2), B(s+3) in flight
constexpr int BIG_RING_CHUNKS = (A_SLOTS * 256 + B_SLOTS * 256) * CPR;  // 160 KB of 16-byte chunks
constexpr int GEMM_WAVES = 8;                  // waves per workgroup: two per SIMD
constexpr int GEMM_THREADS = GEMM_WAVES * 64;

__device__ __forceinline__ int swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

typedef __attribute__((address_space(3))) void *lds_ptr_t;
typedef int i32x4_t __attribute__((ext_vector_type(4)));

// Workgroup barrier without the memory fence of __syncthreads(): that fence
// would also wait for the slices still in flight.  The ordering the rings
// need is explicit: each wave waits (vmcnt) for its own loads of a slice to
// land in LDS, and (lgkmcnt) for its own reads of a slot, before the barrier
// that publishes the slice or frees the slot.
__device__ __forceinline__ void lds_barrier()
{
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Raw buffer descriptor: base, no stride, num_records bytes (reads past it
// return zero), default data format for untyped loads.
__device__ __forceinline__ i32x4_t buffer_desc(const void *base, int64_t bytes)
{
    const uint64_t b = reinterpret_cast<uint64_t>(base);
    i32x4_t d;
    d.x = __builtin_amdgcn_readfirstlane((int)(uint32_t)b);
    d.y = __builtin_amdgcn_readfirstlane((int)(uint32_t)((b >> 32) & 0xffffu));
    d.z = __builtin_amdgcn_readfirstlane((int)bytes);
    d.w = 0x00020000;
    return d;
}

// 16 bytes per lane from global memory straight into LDS: lane i's data lands
// at LDS byte address lds + 16*i.  Written as inline asm so that the
// compiler does not track it as a pending LDS write (it would otherwise wait
// for every such load before any LDS read); the rings wait explicitly.
__device__ __forceinline__ void dma16(i32x4_t desc, uint32_t lds, uint32_t voff, uint32_t soff)
{
    asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
                 :: "s"(lds), "v"(voff), "s"(desc), "s"(soff) : "memory");
}

// The same with the non-temporal hint, for weights that are streamed
// through once per launch.
__device__ __forceinline__ void dma16_nt(i32x4_t desc, uint32_t lds, uint32_t voff, uint32_t soff)
{
    asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen nt lds"
                 :: "s"(lds), "v"(voff), "s"(desc), "s"(soff) : "memory");
}

// The same with an agent-coherent (sc1) load, for data another workgroup
// (possibly on another die, behind another L2) stored with sc1.
__device__ __forceinline__ void dma16_sc1(i32x4_t desc, uint32_t lds, uint32_t voff, uint32_t soff)
{
    asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen sc1 lds"
                 :: "s"(lds), "v"(voff), "s"(desc), "s"(soff) : "memory");
}

__device__ __forceinline__ uint32_t lds_addr(const void *p)
{
    return (uint32_t)(uintptr_t)(lds_ptr_t)(const_cast<void *>(p));
}

// Per-tile DMA sources.  Every row offset is in the per-lane VGPR offset,
// never in the SGPR offset: the buffer range check covers the VGPR offset,
// so a row past the expert's end (A) or past N (B) is given the offset
// num_records and reads as zeros instead of touching memory beyond the
// operand.  The SGPR offset carries only the slice's K position within a row.
struct SliceSrc {
    i32x4_t ra, rb;
    uint32_t voa[8], vob[8];  // per DMA instruction q: this lane's row/chunk byte offset
    int wave;
};

// DMA instruction q of this wave for one BK-slice of A (or of B) into a ring
// slot.  Instruction g of the operand tile fills LDS rows RPI*g .. RPI*g+RPI-1;
// lane i carries row RPI*g + i/CPR at LDS position i%CPR, holding global
// chunk (i%CPR) ^ swz(row).
template <int BMt>
__device__ __forceinline__ void issue_a(const SliceSrc &a, uint32_t slot, int k0, int q)
{
    constexpr int A_INS = BMt / RPI / GEMM_WAVES;
    dma16(a.ra, slot + (a.wave * A_INS + q) * 1024, a.voa[q], (uint32_t)k0 * 2u);
}

template <int BNt, bool NT>
__device__ __forceinline__ void issue_b(const SliceSrc &a, uint32_t slot, int k0, int q)
{
    constexpr int B_INS = BNt / RPI / GEMM_WAVES;
    if constexpr (NT) dma16_nt(a.rb, slot + (a.wave * B_INS + q) * 1024, a.vob[q], (uint32_t)k0 * 2u);
    else dma16(a.rb, slot + (a.wave * B_INS + q) * 1024, a.vob[q], (uint32_t)k0 * 2u);
}

// Instruction q of this wave's run of NI instructions of one operand (A or
// B, whichever the wave loads; its descriptor in a.ra, its offsets in
// a.voa), into a ring slot: operand rows RPI * (a.wave * NI + q) onwards.
template <int NI>
__device__ __forceinline__ void issue_own(const SliceSrc &a, uint32_t slot, int k0, int q)
{
    dma16(a.ra, slot + (a.wave * NI + q) * 1024, a.voa[q], (uint32_t)k0 * 2u);
}

template <int MB, int NB>
struct Frags {
    bf16x8_t a[2][MB], b[2][NB];
};

template <int MB, int NB>
__device__ __forceinline__ void load_frags(Frags<MB, NB> &f, int sl, const uint4 *sa, const uint4 *sb, int kk,
                                           const int (&arow)[MB], const int (&brow)[NB])
{
    const int ch = kk * 2 + ((threadIdx.x & 63) >> 5);
#pragma unroll
    for (int i = 0; i < MB; ++i) {
        uint4 v = sa[arow[i] * CPR + (ch ^ swz(arow[i]))];
        f.a[sl][i] = *reinterpret_cast<bf16x8_t *>(&v);
    }
#pragma unroll
    for (int j = 0; j < NB; ++j) {
        uint4 v = sb[brow[j] * CPR + (ch ^ swz(brow[j]))];
        f.b[sl][j] = *reinterpret_cast<bf16x8_t *>(&v);
    }
}

// The MFMAs of one k-step (MB x NB blocks) with NQ loads of A (IS_B = 0) or
// B (IS_B = 1), numbered q0 .. q0+NQ-1, spread evenly between them (B with
// the non-temporal hint when NTB).
template <int IS_B, int NQ, int MB, int NB, int BMt, int BNt, bool NTB>
__device__ __forceinline__ void mfma_step(f32x16_t (&acc)[MB][NB], const Frags<MB, NB> &f, int sl,
                                          const SliceSrc &src, uint32_t slot, int k0, int q0)
{
    constexpr int TOT = MB * NB;
#pragma unroll
    for (int t = 0; t < TOT; ++t) {
        const int i = t / NB, j = t % NB;
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[sl][i], f.b[sl][j], acc[i][j], 0, 0, 0);
        constexpr int dummy = 0;
        (void)dummy;
        if constexpr (NQ > 0) {
            const int qa = t * NQ / TOT, qb = (t + 1) * NQ / TOT;
            if (qb > qa) {
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int q = qa; q < qb; ++q) {
                    if (IS_B) issue_b<BNt, NTB>(src, slot, k0, q0 + q);
                    else issue_a<BMt>(src, slot, k0, q0 + q);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    }
}

// The MFMAs of one k-step with NQ of this wave's own-operand loads
// (issue_own, numbered q0 .. q0+NQ-1) spread evenly between them, issued
// only when `on` (uniform over the wave).
template <int NI, int NQ, int MB, int NB>
__device__ __forceinline__ void mfma_step_own(f32x16_t (&acc)[MB][NB], const Frags<MB, NB> &f, int sl,
                                              const SliceSrc &src, uint32_t slot, int k0, int q0, bool on)
{
    constexpr int TOT = MB * NB;
#pragma unroll
    for (int t = 0; t < TOT; ++t) {
        const int i = t / NB, j = t % NB;
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[sl][i], f.b[sl][j], acc[i][j], 0, 0, 0);
        if constexpr (NQ > 0) {
            const int qa = t * NQ / TOT, qb = (t + 1) * NQ / TOT;
            if (qb > qa) {
                __builtin_amdgcn_sched_barrier(0);
                if (on) {
#pragma unroll
                    for (int q = qa; q < qb; ++q) issue_own<NI>(src, slot, k0, q0 + q);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    }
}

__device__ __forceinline__ uint16_t bf16_bits(float f)
{
    __bf16 h = static_cast<__bf16>(f);  // round to nearest even
    return *reinterpret_cast<uint16_t *>(&h);
}

// Coordinates of tile `tile` of a tile class: expert e, rows [r0, r1) and
// output columns [n0, n0 + nvalid).  Large tiles are numbered expert by
// expert (ne experts), then by n-tile, with m-tiles innermost, so a die's
// run of tiles shares weight panels.  Small-row tiles are numbered n-tile by
// n-tile, every expert's m-tiles within one: an expert with more rows (a
// shared expert's decode rows) costs more per slice, and numbered this way
// its tiles fall into many workgroups' stream-K runs instead of filling the
// runs of a few.  The class's rows of expert e are [begin(e), split[e]) for
// the large class and [split[e], end(e)) for the tail class.
struct TileCoord {
    int e;
    int64_t r0, r1;
    int n0, nvalid;
};

template <int BMt, int OUTN, bool TAIL>
__device__ __forceinline__ TileCoord tile_coord(int64_t tile, const int32_t *__restrict__ tile_prefix,
                                                const int4 *__restrict__ mtile, int ne,
                                                int n_tiles, const int32_t *__restrict__ offsets, int El,
                                                int64_t shared_rows, const int32_t *__restrict__ split,
                                                int64_t cap, int N)
{
    TileCoord c;
    if constexpr (TAIL) {
        // the class has fewer than 2^31 tiles (checked on the host); its
        // m-tiles are listed by the schedule, so one load finds the expert
        const uint32_t ms = (uint32_t)ld_meta(tile_prefix + ne);
        const int nt = (int)((uint32_t)tile / ms);
        const int32_t *m = reinterpret_cast<const int32_t *>(mtile + ((uint32_t)tile - (uint32_t)nt * ms));
        c.e = ld_meta(m);
        c.r0 = ld_meta(m + 1);
        c.r1 = ld_meta(m + 2);
        c.n0 = nt * OUTN;
        c.nvalid = N - c.n0 < OUTN ? N - c.n0 : OUTN;
        return c;
    } else {
        int lo = 0, hi = ne - 1;
        while (lo < hi) {
            int mid = (lo + hi + 1) >> 1;
            if ((int64_t)ld_meta(tile_prefix + mid) * n_tiles <= tile) lo = mid; else hi = mid - 1;
        }
        const int32_t p0 = ld_meta(tile_prefix + lo), p1 = ld_meta(tile_prefix + lo + 1);
        const int64_t local = tile - (int64_t)p0 * n_tiles;
        const int mte = p1 - p0;
        const int64_t nt64 = div_g(local, mte);
        const int nt = (int)nt64, mt = (int)(local - nt64 * mte);
        c.e = lo;
        const int64_t rb = lo < El ? clamp_row(ld_meta(offsets + lo), cap) : cap;
        const int64_t re = ld_meta(split + lo);
        c.r0 = rb + (int64_t)mt * BMt;
        c.r1 = re < c.r0 + BMt ? re : c.r0 + BMt;
        c.n0 = nt * OUTN;
        c.nvalid = N - c.n0 < OUTN ? N - c.n0 : OUTN;
        return c;
    }
}

// A partial accumulator slot holds one fp32 value per accumulator register
// of each of the 256 threads, stored register-major so each access is a
// coalesced 16-byte vector per lane.

// Work split of one launch over G persistent workgroups.  Tiles [0, dp) are
// handed out whole: large tiles each die a contiguous run dealt round robin
// over its workgroups (workgroups on one die then walk K in near lockstep
// over shared panels, which is what keeps the die's L2 effective), small-row
// tiles round robin over the class's group.
// The K-slices of tiles [dp, T) are cut into G contiguous runs
// ("stream-K"), so every workgroup gets the same number of slices; partial
// sums are combined by the last contributor of each tile (small-row tiles,
// whose partials are small) or by a separate reduction kernel (large tiles:
// one workgroup reading several 256 KB partials would be bound by what one
// CU can pull from memory).  Stream-K takes the weight-streaming small-row
// tiles unless they run whole, and large tiles only in a launch of fewer
// tiles than workgroups with a long K (e.g. one expert's down projection).
enum SplitMode { SPLIT_AUTO, SPLIT_ALWAYS, SPLIT_NEVER };
struct WorkSplit {
    int64_t T, dp, iters;  // tiles, whole tiles, K-slices in the stream-K part
    int nk, G, Gsk;        // slices per tile, workgroups, workgroups in the stream-K part
    __device__ WorkSplit(int64_t total, int nk_, int g, SplitMode mode) : T(total), nk(nk_), G(g)
    {
        // splitting pays only when a tile has many slices and there are too
        // few tiles to fill the grid: each split piece moves its fp32 partial
        // sums through memory, and split pieces lose the lockstep walk over K
        const bool split = mode == SPLIT_ALWAYS || (mode == SPLIT_AUTO && T < G && nk >= SPLIT_MIN_NK);
        dp = split ? 0 : T;
        iters = (T - dp) * nk;
        // every stream-K workgroup gets at least one slice, so the workgroups
        // that meet a tile are exactly a consecutive range
        Gsk = iters < G ? (int)iters : G;
    }
    // first stream-K slice of workgroup v (v <= Gsk)
    __device__ int64_t begin(int v) const { return (int64_t)v * iters / Gsk; }
    // workgroup whose stream-K run holds slice x
    __device__ int owner(int64_t x) const
    {
        int v = (int)(x * Gsk / iters);
        while (v + 1 < Gsk && begin(v + 1) <= x) ++v;
        while (v > 0 && begin(v) > x) --v;
        return v;
    }
};

// Operands of one grouped GEMM launch (both tile classes).
struct GemmArgs {
    const uint16_t *A;          // activations: token matrix (with row_index) or permuted rows
    const int32_t *row_index;   // row -> pair index (divided by kdiv gives the token), or null
    int kdiv;
    int64_t a_rows;             // rows of A when row_index is given
    const int32_t *offsets;     // [El+1] routed experts' row ranges
    const int32_t *split;       // [ne] cut of each expert's rows between the tile classes
    int El, ne;                 // routed experts; all experts (+1 with a shared expert)
    int64_t cap;                // routed rows; the shared expert's rows follow at cap
    int64_t shared_rows, shared_begin;  // shared expert: rows, first token
    int N, K;                   // output columns (per part when gated), reduction length
    const uint16_t *W;          // [El] weight blocks of w_stride elements, rows K-contiguous
    int64_t w_stride;
    const uint16_t *Wsh;        // the shared expert's weight block
    int up_off;                 // first up row when gated
    uint16_t *C;                // [cap, N] bf16 out (routed rows)
    uint16_t *Csh;              // [shared_rows, N] bf16 out (shared rows)
};

// Per tile class: its m-tile prefix over experts, split-K tile counters and
// partial slots.  split[e] cuts expert e's rows between the classes: the
// large class takes [offsets[e], split[e]), the small (tail) class
// [split[e], offsets[e+1]).
struct TileClass {
    const int32_t *tile_prefix;
    const int4 *mtile;  // small class: the schedule's list of its m-tiles
    int32_t *tile_cnt;
    float *partials;
};

// One tile class (BMt x BNt tiles, WM x (8/WM) waves) of a grouped GEMM,
// processed by every workgroup of the persistent grid; `ring` is the
// workgroup's LDS (at least the class's ring size).  Pointers are restrict
// parameters so that the inlined body keeps the no-alias facts of kernel
// arguments (its loads are not reordered around the stores it makes).
template <int BMt, int BNt, bool GATED, int WM, bool TAIL, int ASL, int BSL, bool STREAM>
__device__ __forceinline__ void gemm_class(uint4 *ring, const uint16_t *__restrict__ A,
                                           const int32_t *__restrict__ row_index, int kdiv, int64_t a_rows,
                                           const int32_t *__restrict__ offsets,
                                           const int32_t *__restrict__ split,
                                           const int32_t *__restrict__ tile_prefix,
                                           const int4 *__restrict__ mtile, int El, int ne,
                                           int64_t cap, int64_t shared_rows, int64_t shared_begin,
                                           int N, int K, const uint16_t *__restrict__ W, int64_t w_stride,
                                           const uint16_t *__restrict__ Wsh, int up_off,
                                           uint16_t *__restrict__ C, uint16_t *__restrict__ Csh,
                                           int32_t *__restrict__ tile_cnt, float *__restrict__ partials,
                                           int v, int grp_size, bool deal)
{
    constexpr int A_STAGE = BMt * CPR, B_STAGE = BNt * CPR;  // 16-byte chunks per slot
    constexpr int A_INS = BMt / RPI / GEMM_WAVES, B_INS = BNt / RPI / GEMM_WAVES;
    constexpr int WN = GEMM_WAVES / WM;             // waves in a WM x WN grid
    constexpr int MB = BMt / WM / 32;               // 32-row blocks per wave
    constexpr int NB = BNt / WN / 32;               // 32-col blocks per wave (gate+up when gated)
    constexpr int OUTN = GATED ? BNt / 2 : BNt;     // output columns per tile
    static_assert(MB >= 1 && NB >= (GATED ? 2 : 1), "tile too small for the wave grid");
    // ring slots: ASL for A, BSL for B; under slice s go out A(s+LA) and
    // B(s+LA+1)
    constexpr int LA = ASL - 1;
    static_assert(BSL == ASL + 1 && (LA == 1 || LA == 2), "ring depths");
    constexpr int RING = ASL * A_STAGE + BSL * B_STAGE;
    static_assert(RING <= BIG_RING_CHUNKS, "rings exceed the workgroup's LDS");
    static_assert(A_INS >= 1 && B_INS >= 2 && B_INS % 2 == 0, "DMA instruction split");
    // Large tiles split the loads by operand: waves 0-3 load all of A, waves
    // 4-7 all of B, NI instructions each (see do_work).
    constexpr bool ROLES = !TAIL;
    constexpr int NI = 2 * A_INS;
    static_assert(!ROLES || (2 * B_INS == NI && NI <= 8 && LA == 1 && GEMM_WAVES == 8), "operand roles");
    static_assert(BMt * OUTN * 2 <= RING * 16, "epilogue staging must fit the rings");
    constexpr int SLOT = MB * NB * 16 * GEMM_THREADS;  // floats per partial slot

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform per wave
    const int wm = wave / WN, wn = wave % WN;
    const int n_tiles = (N + OUTN - 1) / OUTN;
    const int nk = K / BIG_BK;
    // the class runs on grp_size workgroups; this one is number v of them
    // (negative: not one of them).  deal (small-row class only): whole tiles
    // dealt round robin over the group instead of stream-K
    const WorkSplit ws((int64_t)tile_prefix[ne] * n_tiles, nk, grp_size,
                       TAIL ? (deal ? SPLIT_NEVER : SPLIT_ALWAYS) : SPLIT_AUTO);
    if (ws.T == 0 || v < 0 || v >= grp_size) return;
    const uint32_t ring_base = lds_addr(ring);
    const uint4 *const a_ring = ring;
    const uint4 *const b_ring = ring + ASL * A_STAGE;

    // this lane's LDS rows for its MFMA fragments
    int arow[MB], brow[NB];
#pragma unroll
    for (int i = 0; i < MB; ++i) arow[i] = wm * (BMt / WM) + i * 32 + (lane & 31);
#pragma unroll
    for (int j = 0; j < NB; ++j) {
        if (GATED) {
            // first NB/2 blocks: gate rows; last NB/2: the matching up rows
            const int jj = j % (NB / 2);
            brow[j] = (j < NB / 2 ? 0 : BNt / 2) + wn * (BNt / 2 / WN) + jj * 32 + (lane & 31);
        } else {
            brow[j] = wn * (BNt / WN) + j * 32 + (lane & 31);
        }
    }

    // Write the staged bf16 tile [BM][OUTN] from LDS with 16-byte stores to
    // rows [r0, r1), whose first row is at Cb.
    auto store_staged = [&](uint16_t *Cb, int64_t r0, int64_t r1, int n0, int nvalid) {
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        lds_barrier();
        const uint4 *so = ring;
        constexpr int CH_ROW = OUTN / 8;
        const int rows = (int)(r1 - r0);
        for (int c = tid; c < BMt * CH_ROW; c += GEMM_THREADS) {
            const int row = c / CH_ROW, cc = c % CH_ROW;
            if (row < rows && cc * 8 < nvalid)
                *reinterpret_cast<uint4 *>(Cb + row * N + n0 + cc * 8) = so[c];
        }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        lds_barrier();  // staging reads done before the next piece's loads
    };

    // One piece of work: K-slices [klo, khi) of tile `tile`.
    auto do_work = [&](int64_t tile, int klo, int khi) {
        const TileCoord tc = tile_coord<BMt, OUTN, TAIL>(tile, tile_prefix, mtile, ne, n_tiles, offsets, El, shared_rows,
                                                         split, cap, N);
        const int e = tc.e;
        const int64_t r0 = tc.r0, r1 = tc.r1;
        const int n0 = tc.n0, nvalid = tc.nvalid;
        // the shared expert (e == El) has its own weights and output rows
        const uint16_t *We = e < El ? W + (int64_t)e * w_stride : Wsh;
        uint16_t *Cb = e < El ? C + r0 * N : Csh + (r0 - cap) * N;

        // Which operand rows this wave loads.  Large tiles: waves 0-3 load
        // all of A and waves 4-7 all of B.  A SIMD runs waves i and i + 4,
        // and the first wins the MFMA arbitration: it finishes each slice
        // ahead of the second and waits at the barrier, while the second
        // reaches its loads (spread over its MFMAs) later; with the loads
        // split evenly, the second then waited for its share of the next A
        // slice while the SIMD's MFMAs stood idle.  So the early waves load
        // the next slice's A and the late ones B two slices ahead, which has
        // landed by the time they need it.  Small-row tiles: every wave loads
        // A_INS instructions of A and B_INS of B.
        const bool loads_a = !ROLES || wave < GEMM_WAVES / 2;  // uniform over the wave
        const int wb = ROLES ? wave - GEMM_WAVES / 2 : wave;   // index among the B loaders
        const int b_ins = ROLES ? NI : B_INS;
        // this wave's B rows lie in one part (gate or up) when gated
        const int bpart = GATED ? ((wb * b_ins * RPI) / (BNt / 2)) : 0;
        const int brow0 = wb * b_ins * RPI - bpart * (BNt / 2);  // first B row of this wave in its part
        SliceSrc src;
        src.wave = ROLES && !loads_a ? wb : wave;
        // A rows come from the permuted buffer (rows r0.. contiguous) or, with
        // row_index, straight from the token matrix (the fused row gather)
        const int64_t a_bytes = row_index ? a_rows * K * 2 : (r1 - r0) * K * 2;
        const i32x4_t desc_a = buffer_desc(row_index ? A : A + r0 * K, a_bytes);
        const int64_t b_bytes = (int64_t)nvalid * K * 2;
        const i32x4_t desc_b = buffer_desc(We + (int64_t)((GATED && bpart) ? up_off + n0 : n0) * K, b_bytes);
        // K, kdiv and the lane pass through empty asm statements so that the
        // offsets below are computed per tile: hoisted out of the tile loop,
        // their tile-independent parts would be kept in spilled registers
        // and reloaded from scratch at every tile, each reload waiting
        // (vector memory counter) for the previous tile's output stores.
        int Kt = K, kd = kdiv, ln = lane;
        asm volatile("" : "+s"(Kt), "+s"(kd), "+v"(ln));
        const int lr = ln >> 3;  // this lane's row within a DMA instruction
        // this lane's byte offset in A instruction g (LDS rows RPI*g ..)
        // ... given ri, the row index of this lane's row of instruction g
        // (gathered rows; unused otherwise)
        auto a_off_ri = [&](int g, int32_t ri) -> uint32_t {
            const int trow = g * RPI + lr;                       // row of the tile
            const int kc = (ln & 7) ^ lr ^ (g & 1);                // position ^ swz(row)
            const int64_t r = r0 + trow;
            int64_t off;
            if (r >= r1) off = a_bytes;                            // past the expert: zeros
            else if (row_index) {
                // the shared expert's rows are tokens shared_begin, ...
                const int64_t tok = r < cap ? (int64_t)(ri / kd) : shared_begin + (r - cap);
                off = (tok * Kt + kc * 8) * 2;
            }
            else off = ((int64_t)trow * Kt + kc * 8) * 2;
            return (uint32_t)off;
        };
        // This lane's row index in RPI indices read as one scalar load.
        auto pick = [&](const rows_t &vj) -> int32_t {
            int32_t ri = 0;
#pragma unroll
            for (int j = 0; j < RPI; ++j) ri = lr == j ? vj[j] : ri;
            return ri;
        };
        auto a_off = [&](int g) -> uint32_t {
            // Gathered rows: the RPI row indices of this instruction's rows
            // are read with scalar loads (the rows are the same for the whole
            // wave), so they do not wait for the output stores of the
            // workgroup's previous tile; each lane takes its own.  Rows at or
            // past cap (the shared expert's) take none, and the indices read
            // are clamped into the array.
            int32_t ri = 0;
            const int64_t rb = r0 + (int64_t)g * RPI;
            if (row_index != nullptr && rb + RPI <= cap) {
                ri = pick(ld_rows(row_index + rb));
            } else if (row_index != nullptr && rb < cap) {
#pragma unroll
                for (int j = 0; j < RPI; ++j) {
                    const int32_t vj = ld_meta(row_index + (rb + j < cap ? rb + j : cap - 1));
                    ri = lr == j ? vj : ri;
                }
            }
            return a_off_ri(g, ri);
        };
        // ... in this wave's B instruction q, instruction g of the operand
        auto b_off = [&](int q, int g) -> uint32_t {
            const int prow = brow0 + q * RPI + lr;                 // row within its part
            const int kc = (ln & 7) ^ lr ^ (g & 1);                // LDS row g*RPI+lr
            return prow < nvalid ? (uint32_t)(((int64_t)prow * Kt + kc * 8) * 2) : (uint32_t)b_bytes;
        };
        if constexpr (ROLES) {
            // one descriptor and one set of offsets: the operand this wave loads
            src.ra = loads_a ? desc_a : desc_b;
            if (loads_a) {
                const int64_t gb = r0 + (int64_t)wave * NI * RPI;  // first row of this wave's instructions
                // (only the gate-up GEMM gathers its rows: the down GEMM's code
                // keeps its register allocation)
                if (GATED && row_index != nullptr && gb + NI * RPI <= cap) {
                    // every instruction's rows are routed rows: issue all NI
                    // index loads before using any, so the prologue waits for
                    // one scalar-load latency instead of NI in a row
                    rows_t vr[NI];
#pragma unroll
                    for (int q = 0; q < NI; ++q) vr[q] = ld_rows(row_index + gb + q * RPI);
#pragma unroll
                    for (int q = 0; q < NI; ++q) src.voa[q] = a_off_ri(wave * NI + q, pick(vr[q]));
                } else {
#pragma unroll
                    for (int q = 0; q < NI; ++q) src.voa[q] = a_off(wave * NI + q);
                }
            } else {
#pragma unroll
                for (int q = 0; q < NI; ++q) src.voa[q] = b_off(q, wb * NI + q);
            }
        } else {
            src.ra = desc_a;
            src.rb = desc_b;
#pragma unroll
            for (int q = 0; q < A_INS; ++q) src.voa[q] = a_off(wave * A_INS + q);
#pragma unroll
            for (int q = 0; q < B_INS; ++q) src.vob[q] = b_off(q, wave * B_INS + q);
        }

        f32x16_t acc[MB][NB];
#pragma unroll
        for (int i = 0; i < MB; ++i)
#pragma unroll
            for (int j = 0; j < NB; ++j) acc[i][j] = f32x16_t{};
        Frags<MB, NB> f;

        // Slices klo..khi-1 (local index j): A(j) in A slot j % ASL, B(j) in
        // B slot j % BSL.  Loads go out in pairs (A(t), B(t+1)) after B(0):
        // the prologue issues pairs t < LA, slice s issues pair s+LA (A under
        // k-steps 0-1, B under k-steps 2-3) into the slots slice s-1 freed.
        const int ns = khi - klo;  // slices in this piece (>= 1)
        auto kof = [&](int j) { return (klo + j) * BIG_BK; };
        auto a_slot = [&](int j) { return ring_base + (uint32_t)((j % ASL) * A_STAGE * 16); };
        auto b_slot = [&](int j) { return ring_base + (uint32_t)((ASL * A_STAGE + (j % BSL) * B_STAGE) * 16); };
        auto a_ptr = [&](int j) { return a_ring + (j % ASL) * A_STAGE; };
        auto b_ptr = [&](int j) { return b_ring + (j % BSL) * B_STAGE; };
        using T_ = std::true_type;
        using F_ = std::false_type;
        if constexpr (ROLES) {
            // prologue: A(0) on the A loaders, B(0) and B(1) on the B loaders
            if (loads_a) {
#pragma unroll
                for (int q = 0; q < NI; ++q) issue_own<NI>(src, a_slot(0), kof(0), q);
                asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
            } else {
#pragma unroll
                for (int q = 0; q < NI; ++q) issue_own<NI>(src, b_slot(0), kof(0), q);
                if (ns > 1) {
#pragma unroll
                    for (int q = 0; q < NI; ++q) issue_own<NI>(src, b_slot(1), kof(1), q);
                    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)" ::"n"(NI) : "memory");
                } else {
                    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
                }
            }
            lds_barrier();
            load_frags(f, 0, a_ptr(0), b_ptr(0), 0, arow, brow);

            // One slice: under k-steps 0-1 the A loaders issue A(s+1) (HA: it
            // exists) and the B loaders B(s+2) (HB: it exists).
            auto slice = [&](int s, auto has_a, auto has_b) {
                constexpr bool HA = decltype(has_a)::value, HB = decltype(has_b)::value;
                constexpr int NQ = HA || HB ? NI / 2 : 0;
                const bool on = loads_a ? HA : HB;
                const uint32_t dst = loads_a ? a_slot(s + 1) : b_slot(s + 2);
                const int kn = loads_a ? kof(s + 1) : kof(s + 2);
                const uint4 *sa = a_ptr(s), *sb = b_ptr(s);
                load_frags(f, 1, sa, sb, 1, arow, brow);
                __builtin_amdgcn_sched_barrier(0);
                mfma_step_own<NI, NQ>(acc, f, 0, src, dst, kn, 0, on);
                __builtin_amdgcn_sched_barrier(0);
                load_frags(f, 0, sa, sb, 2, arow, brow);
                __builtin_amdgcn_sched_barrier(0);
                mfma_step_own<NI, NQ>(acc, f, 1, src, dst, kn, NI / 2, on);
                __builtin_amdgcn_sched_barrier(0);
                load_frags(f, 1, sa, sb, 3, arow, brow);
                __builtin_amdgcn_sched_barrier(0);
                mfma_step_own<NI, 0>(acc, f, 0, src, dst, kn, 0, false);
                __builtin_amdgcn_sched_barrier(0);
                if (s + 1 < ns) {
                    // hand over to slice s+1 once this wave's loads of it
                    // have landed: A(s+1), issued under this slice, or
                    // B(s+1), issued under the last one (B(s+2) may still be
                    // in flight)
                    if (!loads_a && HB) asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)" ::"n"(NI) : "memory");
                    else asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
                    lds_barrier();
                    load_frags(f, 0, a_ptr(s + 1), b_ptr(s + 1), 0, arow, brow);
                    __builtin_amdgcn_sched_barrier(0);
                }
                mfma_step_own<NI, 0>(acc, f, 1, src, dst, kn, 0, false);
                __builtin_amdgcn_sched_barrier(0);
            };
            int s = 0;
            for (; s + 2 < ns; ++s) slice(s, T_{}, T_{});
            for (; s + 1 < ns; ++s) slice(s, T_{}, F_{});
            for (; s < ns; ++s) slice(s, F_{}, F_{});
        } else {
            // prologue: B(0), then (A(t), B(t+1)) for t < LA; wait for A(0), B(0)
    #pragma unroll
            for (int q = 0; q < B_INS; ++q) issue_b<BNt, STREAM>(src, b_slot(0), kof(0), q);
    #pragma unroll
            for (int t = 0; t < LA; ++t) {
                if (t < ns) {
    #pragma unroll
                    for (int q = 0; q < A_INS; ++q) issue_a<BMt>(src, a_slot(t), kof(t), q);
                }
                if (t + 1 < ns) {
    #pragma unroll
                    for (int q = 0; q < B_INS; ++q) issue_b<BNt, STREAM>(src, b_slot(t + 1), kof(t + 1), q);
                }
            }
            // issued after A(0): B(1), then the pairs 1 .. LA-1
            if (ns > LA) asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)" ::"n"(B_INS + (LA - 1) * (A_INS + B_INS)) : "memory");
            else asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
            lds_barrier();
            load_frags(f, 0, a_ptr(0), b_ptr(0), 0, arow, brow);

            // One slice.  HAVE_A: A(s+LA) exists; HAVE_B: B(s+LA+1) exists; loads
            // absent at the tail keep the MFMA runs free of branches.
            auto slice = [&](int s, auto have_a, auto have_b) {
                constexpr bool HA = decltype(have_a)::value, HB = decltype(have_b)::value;
                // loads issued after A(s+1) when this slice hands over: B(s+2) ..
                // B(s+LA), A(s+2) .. A(s+LA) and the first half of B(s+LA+1)
                constexpr int AFTER = HA ? (LA - 1) * (A_INS + B_INS) + (HB ? B_INS / 2 : 0) : 0;
                const uint4 *sa = a_ptr(s), *sb = b_ptr(s);
                load_frags(f, 1, sa, sb, 1, arow, brow);
                __builtin_amdgcn_sched_barrier(0);
                mfma_step<0, HA ? A_INS / 2 : 0, MB, NB, BMt, BNt, STREAM>(acc, f, 0, src, a_slot(s + LA), kof(s + LA), 0);
                __builtin_amdgcn_sched_barrier(0);
                load_frags(f, 0, sa, sb, 2, arow, brow);
                __builtin_amdgcn_sched_barrier(0);
                mfma_step<0, HA ? A_INS - A_INS / 2 : 0, MB, NB, BMt, BNt, STREAM>(acc, f, 1, src, a_slot(s + LA),
                                                                       kof(s + LA), A_INS / 2);
                __builtin_amdgcn_sched_barrier(0);
                load_frags(f, 1, sa, sb, 3, arow, brow);
                __builtin_amdgcn_sched_barrier(0);
                mfma_step<1, HB ? B_INS / 2 : 0, MB, NB, BMt, BNt, STREAM>(acc, f, 0, src, b_slot(s + LA + 1), kof(s + LA + 1),
                                                               0);
                __builtin_amdgcn_sched_barrier(0);
                if (HA || s + 1 < ns) {
                    // hand over to slice s+1 once A(s+1) (and B(s+1), issued before
                    // it) have landed
                    if (AFTER > 0) asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)" ::"n"(AFTER) : "memory");
                    else asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
                    lds_barrier();
                    load_frags(f, 0, a_ptr(s + 1), b_ptr(s + 1), 0, arow, brow);
                    __builtin_amdgcn_sched_barrier(0);
                }
                mfma_step<1, HB ? B_INS - B_INS / 2 : 0, MB, NB, BMt, BNt, STREAM>(acc, f, 1, src, b_slot(s + LA + 1),
                                                                       kof(s + LA + 1), B_INS / 2);
                __builtin_amdgcn_sched_barrier(0);
            };
            int s = 0;
            for (; s + LA + 1 < ns; ++s) slice(s, T_{}, T_{});
            for (; s + LA < ns; ++s) slice(s, T_{}, F_{});
            for (; s < ns; ++s) slice(s, F_{}, F_{});
        }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        lds_barrier();  // every wave is done with the ring before it is reused

        if (klo != 0 || khi != nk) {
            // Part of a stream-K tile.  Contributors are the workgroups whose
            // runs meet the tile's slices; each stores its partial, and the
            // last to arrive sums all of them in contributor order (the same
            // order whoever arrives last) and writes the tile.
            const int64_t tb = (tile - ws.dp) * nk;  // first stream-K slice of the tile
            const int vfirst = ws.owner(tb), vlast = ws.owner(tb + nk - 1);
            auto slot_of = [&](int u) {  // slot 0: u's run starts in this tile; 1: it ends here
                return (int64_t)u * 2 + (ws.begin(u) >= tb ? 0 : 1);
            };
            // Partials move with agent-coherent (sc1) stores and loads, so no
            // L2-wide write-back/invalidate fence is needed: a fence would
            // flush the operand panels other workgroups on the die are reusing.
            typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
            const __amdgpu_buffer_rsrc_t pr = __builtin_amdgcn_make_buffer_rsrc(
                partials, (short)0, (int)((int64_t)2 * ws.G * SLOT * 4), 0x00020000);
            constexpr int SC1 = 0x10;
            // Small-row tiles move only the 8-row groups of a wave that hold
            // rows of the tile (decode tiles are mostly padding); the group
            // test is uniform over the wave, so writer and reader agree.
            // Large tiles move everything (splitk_reduce reads whole slots).
            const int nrows = (int)(r1 - r0);
            auto live = [&](int i, int q) { return !TAIL || wm * (BMt / WM) + i * 32 + 8 * q < nrows; };
            {
                const uint32_t base_b = (uint32_t)(slot_of(v) * SLOT * 4);
#pragma unroll
                for (int i = 0; i < MB; ++i)
#pragma unroll
                    for (int j = 0; j < NB; ++j)
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            if (!live(i, q)) continue;
                            float4 pv = make_float4(acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                                                    acc[i][j][4 * q + 3]);
                            __builtin_amdgcn_raw_buffer_store_b128(
                                *reinterpret_cast<u32x4_t *>(&pv), pr,
                                base_b + (uint32_t)((((i * NB + j) * 4 + q) * GEMM_THREADS + tid) * 16), 0, SC1);
                        }
            }
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // partial is visible device-wide
            lds_barrier();
            if constexpr (!TAIL) return;  // large tiles: splitk_reduce combines the partials
            int *flag = reinterpret_cast<int *>(ring);
            if (tid == 0) {
                const int old = __hip_atomic_fetch_add(&tile_cnt[tile], 1, __ATOMIC_RELAXED,
                                                       __HIP_MEMORY_SCOPE_AGENT);
                *flag = old == vlast - vfirst;
            }
            asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
            lds_barrier();
            const bool last = *flag != 0;
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            lds_barrier();
            if (!last) return;
            // Stream contributor c's partial into the accumulators (assign:
            // acc = partial, else acc += partial) through LDS: one block row
            // (NB*4 DMA instructions per wave, 1 KB each) per chunk, two
            // chunks in flight.  Each wave reads back only what its own loads
            // wrote, so waiting for its own loads (vmcnt) is enough.
            const i32x4_t pdesc = buffer_desc(partials, (int64_t)2 * ws.G * SLOT * 4);
            auto add_partial = [&](int c, bool assign) {
                constexpr int CH = NB * 4;
                const uint32_t base_c = (uint32_t)(slot_of(c) * SLOT * 4);
                constexpr int JQ = GEMM_THREADS * 16;  // bytes of one (j, q) chunk of the slot
                auto issue = [&](int i) {
                    const uint32_t buf = ring_base + (uint32_t)((i & 1) * CH * JQ);
#pragma unroll
                    for (int jq = 0; jq < CH; ++jq)
                        if (live(i, jq % 4))
                            dma16_sc1(pdesc, buf + jq * JQ + wave * 1024, (uint32_t)(jq * JQ + tid * 16),
                                      base_c + (uint32_t)(i * CH * JQ));
                };
                issue(0);
#pragma unroll
                for (int i = 0; i < MB; ++i) {
                    if (i + 1 < MB) {
                        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // chunk i-1 read out
                        issue(i + 1);
                        // with groups skipped the count of chunk i+1 varies
                        if (TAIL) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
                        else asm volatile("s_waitcnt vmcnt(%0)" ::"n"(CH) : "memory");
                    } else {
                        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
                    }
                    const uint4 *bp = ring + (i & 1) * CH * GEMM_THREADS;
#pragma unroll
                    for (int j = 0; j < NB; ++j)
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            if (!live(i, q)) continue;  // rows past the tile: never stored
                            const uint4 w = bp[(j * 4 + q) * GEMM_THREADS + tid];
                            const float pv[4] = {__uint_as_float(w.x), __uint_as_float(w.y),
                                                 __uint_as_float(w.z), __uint_as_float(w.w)};
#pragma unroll
                            for (int r = 0; r < 4; ++r)
                                acc[i][j][4 * q + r] = assign ? pv[r] : acc[i][j][4 * q + r] + pv[r];
                        }
                }
                asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            };
            if (vlast - vfirst == 1) {
                // Two contributors: add the other one's partial (fp32
                // addition commutes, so the sum does not depend on which of
                // the two arrived last).
                add_partial(v == vfirst ? vlast : vfirst, false);
            } else {
                // Three or more: rebuild the sum in contributor order from the
                // stored partials, this workgroup's own included, so the
                // result does not depend on which contributor arrived last.
                for (int c = vfirst; c <= vlast; ++c) add_partial(c, c == vfirst);
            }
            lds_barrier();  // LDS free again for the epilogue's staging
        }

        // epilogue: block (i, j) lane holds column (lane & 31), rows
        // 8*(v/4) + 4*(lane/32) + v%4; stage the bf16 tile [BM][OUTN] in LDS
        uint16_t *stage_out = reinterpret_cast<uint16_t *>(ring);
#pragma unroll
        for (int i = 0; i < MB; ++i) {
#pragma unroll
            for (int j = 0; j < (GATED ? NB / 2 : NB); ++j) {
                const int col = wn * (OUTN / WN) + j * 32 + (lane & 31);
#pragma unroll
                for (int q = 0; q < 16; ++q) {
                    const int row = wm * (BMt / WM) + i * 32 + 8 * (q / 4) + 4 * (lane >> 5) + (q % 4);
                    float o = acc[i][j][q];
                    if (GATED) o = silu_mul(o, acc[i][j + NB / 2][q]);
                    stage_out[row * OUTN + col] = bf16_bits(o);
                }
            }
        }
        store_staged(Cb, r0, r1, n0, nvalid);
    };

    // This workgroup's work items, in order: its whole tiles, then its
    // stream-K run.  Whole tiles: the group is 8 runs of G/8 ids, one per die
    // (die-major numbering, see gemm_grouped); die d takes the contiguous
    // tiles [dp*d/8, dp*(d+1)/8), dealt round robin over its workgroups, so
    // each die walks a run of consecutive tiles (m-tiles innermost: shared B
    // panels in its L2) and every die gets the same number of tiles (the
    // workgroups idle in the last round are spread over all dies); small-row
    // tiles dealt whole form one run over the whole group.  One call site
    // keeps the kernel's register allocation to a single copy of the
    // pipeline.
    constexpr int NDIE = TAIL ? 1 : 8;
    int64_t n_dp = 0, t0 = 0;
    const int P = grp_size / NDIE;
    if (ws.dp > 0) {
        const int d = v / P, u = v % P;
        const int64_t lo = ws.dp * d / NDIE, hi = ws.dp * (d + 1) / NDIE;
        n_dp = u < hi - lo ? (hi - lo - 1 - u) / P + 1 : 0;
        t0 = lo + u;
    }
    const bool has_sk = ws.iters > 0 && v < ws.Gsk;
    int64_t sk_i = has_sk ? ws.begin(v) : 0;
    const int64_t sk_end = has_sk ? ws.begin(v + 1) : 0;
    for (int64_t w = 0;; ++w) {
        int64_t tile;
        int klo, khi;
        if (w < n_dp) {
            tile = t0 + w * P;
            klo = 0;
            khi = nk;
        } else if (sk_i < sk_end) {
            tile = ws.dp + sk_i / nk;
            klo = (int)(sk_i % nk);
            khi = (int)(klo + (sk_end - sk_i) < nk ? klo + (sk_end - sk_i) : nk);
            sk_i += khi - klo;
        } else {
            break;
        }
        do_work(tile, klo, khi);
    }
}

constexpr int BIGM = 256, BIGN = 256;  // large tiles: 256 rows x 256 weight rows
constexpr int BIG_WM = 4;              // ... 4 x 2 waves of 64 x 128
// small-row tiles: 64 or 128 rows x 256 weight rows, 2 x 4 waves of 32 x 64
// or 64 x 64; the 128-row rings are shallower (A(s+1), B(s+2) in flight)
constexpr int SMALL_WM = 2;
constexpr int S128_ASL = 2, S128_BSL = 3;
constexpr int REDUCE_GRID = 2048;      // workgroups of the split-K reduction
constexpr int BIG_RING = BIG_RING_CHUNKS;
// floats per partial slot of each class (one per accumulator register; the
// small class's slots fit either height)
constexpr int SLOT_SMALL = (SMALL128.rows / SMALL_WM / 32) * (BIGN / (GEMM_WAVES / SMALL_WM) / 32) * 16 *
                           GEMM_THREADS;
constexpr int SLOT_BIG = (BIGM / BIG_WM / 32) * (BIGN / (GEMM_WAVES / BIG_WM) / 32) * 16 * GEMM_THREADS;

// The small-row class's group of workgroups under small_plan: the idle ones
// (SM_PIECES_IDLE, SM_WHOLE_IDLE), or all of them (SM_WHOLE_ALL with the
// idle ones numbered first, SM_PIECES_ALL in die-major order).  The
// workgroups the large tiles leave idle in their last round are found from
// the large tiles' die-balanced deal.  Stream-K members are numbered die by
// die (consecutive slices of a tile then share a die's L2); members that are
// dealt whole tiles are numbered across the dies in turn, so that fewer tiles
// than members still spread over all dies (on a few dies they would pull
// every weight panel through those dies' links).  vx is this workgroup's
// die-major id (G/8 consecutive ids per die).  Returns this workgroup's
// number in the group (negative: not in it), the group size and whether
// whole tiles are dealt round robin (else stream-K).
struct SmallGroup {
    int v, size;
    bool deal;
};

__device__ __forceinline__ SmallGroup small_group(int64_t tl, int64_t ts, int nk, int G, SmallKind kind, int vx)
{
    const SmallPlan p = small_plan(tl, ts, nk, G, kind.cost_num, whole_fit(nk, kind.whole_num),
                                   whole_time(nk, kind.whole_num));
    const bool deal = p.mode == SM_WHOLE_IDLE || p.mode == SM_WHOLE_ALL;
    if (p.mode == SM_PIECES_ALL) return SmallGroup{vx, G, false};
    if (p.mode == SM_PIECES_PAIR) {
        // the first 2 * ts workgroups in (workgroup within die, die) order
        const int P = G / 8, size = (int)(2 * ts);
        const int v = (vx % P) * 8 + vx / P;
        return SmallGroup{v < size ? v : -1, size, false};
    }
    // die d holds c_d = tl*(d+1)/8 - tl*d/8 whole tiles; with R rounds (the
    // busiest die's), its workgroups u < c_d - (R-1)*P are busy in the last
    // round and the others idle (G - tl % G of them in all; none, and all
    // counted busy, when the last round is full or there are no large tiles)
    const int P = G / 8, d = vx / P, u = vx % P;
    const int64_t R = ((tl + 7) / 8 + P - 1) / P;
    int busy[8];
    int n_idle = 0;
    for (int dd = 0; dd < 8; ++dd) {
        const int64_t c = tl * (dd + 1) / 8 - tl * dd / 8;
        const int64_t b64 = p.idle ? c - (R - 1) * P : P;
        busy[dd] = b64 < 0 ? 0 : (b64 > P ? P : (int)b64);
        n_idle += P - busy[dd];
    }
    const bool idle = u >= busy[d];
    const int j = idle ? u - busy[d] : u;  // index among the die's idle (busy) workgroups
    int v = 0;
    for (int dd = 0; dd < 8; ++dd) {
        const int cnt = idle ? P - busy[dd] : busy[dd];
        if (deal) v += (cnt < j ? cnt : j) + (dd < d && cnt > j);  // (j, die) order
        else if (dd < d) v += cnt;                                 // (die, j) order
    }
    v += deal ? 0 : j;
    if (!idle) v = p.mode == SM_WHOLE_ALL ? n_idle + v : -1;
    return SmallGroup{v, p.mode == SM_WHOLE_ALL ? G : n_idle, deal};
}

// Device-side launch timestamps (moe_timing_device_*): per slot, the
// earliest workgroup start and the latest workgroup end of one launch, in
// ticks of the 100 MHz constant clock.  A launch takes a slot on the host
// (at capture time when it is captured), so launches replayed from a HIP
// graph, where no event can be recorded between kernels, are timed too.
// Each die keeps its own start and end (workgroup b runs on die b % 8, as
// the hardware deals workgroups to the dies round robin), which spreads the
// atomics over eight words; the dies' counters agree to well under a
// microsecond, so a launch's duration is its earliest start on any die to
// its latest end on any die.
constexpr int DEV_TS_SLOTS = 4096;
__device__ unsigned long long g_dev_ts[2][8][DEV_TS_SLOTS];  // [0]: start (min), [1]: end (max), per die

// One grouped GEMM launch: the large-tile class (256-row tiles) and the
// small-row class (64- or 128-row tiles as the schedule chose, K-split over
// its workgroups: these stream weights, and spreading them over many CUs is
// what reaches HBM bandwidth) in the same persistent grid.  The classes
// cover disjoint rows, so a workgroup goes from its large tiles to its
// small-row share without waiting for anyone.  STREAM: the small-row class
// loads its weights with the non-temporal hint (launches whose weights
// cannot stay in the last-level cache from one step to the next).
template <bool GATED, bool STREAM>
__global__ __attribute__((amdgpu_flat_work_group_size(GEMM_THREADS, GEMM_THREADS), amdgpu_waves_per_eu(2, 2)))
void gemm_grouped(GemmArgs g, TileClass small, TileClass large, int tslot)
{
    __shared__ uint4 ring[BIG_RING];
    if (tslot >= 0 && threadIdx.x == 0) atomicMin(&g_dev_ts[0][blockIdx.x & 7][tslot], __builtin_amdgcn_s_memrealtime());
    constexpr int OUTN = GATED ? BIGN / 2 : BIGN;
    // die-major id: the hardware deals workgroups to the 8 dies round robin
    const int vx = (blockIdx.x & 7) * (gridDim.x >> 3) + (blockIdx.x >> 3);
    gemm_class<BIGM, BIGN, GATED, BIG_WM, false, A_SLOTS, B_SLOTS, false>(
        ring, g.A, g.row_index, g.kdiv, g.a_rows, g.offsets, g.split, large.tile_prefix, nullptr, g.El, g.ne, g.cap,
        g.shared_rows, g.shared_begin, g.N, g.K, g.W, g.w_stride, g.Wsh, g.up_off, g.C, g.Csh, large.tile_cnt,
        large.partials, vx, gridDim.x, false);
    // the small class's group, worked out only now (a compiler barrier keeps
    // its loads here, so nothing of it stays live through the large tiles)
    asm volatile("" ::: "memory");
    const int64_t n_tiles = (g.N + OUTN - 1) / OUTN;
    const bool tall = small.tile_prefix[g.ne + 1] == SMALL128.rows;  // uniform
    const SmallGroup sg = small_group((int64_t)large.tile_prefix[g.ne] * n_tiles,
                                      (int64_t)small.tile_prefix[g.ne] * n_tiles, g.K / BIG_BK, gridDim.x,
                                      tall ? SMALL128 : SMALL64, vx);
    if (tall)
        gemm_class<SMALL128.rows, BIGN, GATED, SMALL_WM, true, S128_ASL, S128_BSL, STREAM>(
            ring, g.A, g.row_index, g.kdiv, g.a_rows, g.offsets, g.split, small.tile_prefix, small.mtile, g.El, g.ne, g.cap,
            g.shared_rows, g.shared_begin, g.N, g.K, g.W, g.w_stride, g.Wsh, g.up_off, g.C, g.Csh,
            small.tile_cnt, small.partials, sg.v, sg.size, sg.deal);
    else
        gemm_class<SMALL64.rows, BIGN, GATED, SMALL_WM, true, SA_SLOTS, SB_SLOTS, STREAM>(
            ring, g.A, g.row_index, g.kdiv, g.a_rows, g.offsets, g.split, small.tile_prefix, small.mtile, g.El, g.ne, g.cap,
            g.shared_rows, g.shared_begin, g.N, g.K, g.W, g.w_stride, g.Wsh, g.up_off, g.C, g.Csh,
            small.tile_cnt, small.partials, sg.v, sg.size, sg.deal);
    if (tslot >= 0) {
        __syncthreads();  // every wave of the workgroup is done
        if (threadIdx.x == 0) atomicMax(&g_dev_ts[1][blockIdx.x & 7][tslot], __builtin_amdgcn_s_memrealtime());
    }
}

// Combines the split-K partials of the large-tile class after its GEMM
// launch (G persistent workgroups, the same work split): for every split
// tile, every block of 32x32 outputs of every wave position is one work
// item, so all CUs share the partial traffic.  Each partial is summed in
// contributor order (deterministic), then the epilogue of the GEMM is
// applied (SwiGLU when gated) and the bf16 result written.
template <bool GATED>
__global__ __launch_bounds__(GEMM_THREADS) void splitk_reduce(const int32_t *__restrict__ offsets,
                                                     const int32_t *__restrict__ split,
                                                     const int32_t *__restrict__ tile_prefix, int El, int ne,
                                                     int64_t cap, int64_t shared_rows, int N, int K, int G,
                                                     const float *__restrict__ partials,
                                                     uint16_t *__restrict__ C, uint16_t *__restrict__ Csh)
{
    constexpr int WM = BIG_WM, WN = GEMM_WAVES / BIG_WM;
    constexpr int MB = BIGM / WM / 32, NB = BIGN / WN / 32;
    constexpr int OUTN = GATED ? BIGN / 2 : BIGN;
    constexpr int JJ = GATED ? NB / 2 : NB;  // output blocks per wave row
    const int n_tiles = (N + OUTN - 1) / OUTN;
    const int nk = K / BIG_BK;
    const WorkSplit ws((int64_t)tile_prefix[ne] * n_tiles, nk, G, SPLIT_AUTO);
    const int64_t items = (ws.T - ws.dp) * MB * JJ;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;
    for (int64_t it = blockIdx.x; it < items; it += gridDim.x) {
        const int64_t tile = ws.dp + it / (MB * JJ);
        const int i = (int)((it / JJ) % MB), j = (int)(it % JJ);
        const TileCoord tc = tile_coord<BIGM, OUTN, false>(tile, tile_prefix, nullptr, ne, n_tiles, offsets, El, shared_rows,
                                                           split, cap, N);
        uint16_t *Cb = tc.e < El ? C + tc.r0 * N : Csh + (tc.r0 - cap) * N;
        const int64_t tb = (tile - ws.dp) * nk;
        const int vfirst = ws.owner(tb), vlast = ws.owner(tb + nk - 1);
        float g[16], u[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) g[r] = u[r] = 0.f;
        for (int c = vfirst; c <= vlast; ++c) {
            const float4 *slot = reinterpret_cast<const float4 *>(
                partials + (c * 2 + (ws.begin(c) >= tb ? 0 : 1)) * (int64_t)SLOT_BIG);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float4 pg = slot[((i * NB + j) * 4 + q) * GEMM_THREADS + tid];
                g[4 * q] += pg.x; g[4 * q + 1] += pg.y; g[4 * q + 2] += pg.z; g[4 * q + 3] += pg.w;
                if (GATED) {
                    const float4 pu = slot[((i * NB + j + NB / 2) * 4 + q) * GEMM_THREADS + tid];
                    u[4 * q] += pu.x; u[4 * q + 1] += pu.y; u[4 * q + 2] += pu.z; u[4 * q + 3] += pu.w;
                }
            }
        }
        const int col = wn * (OUTN / WN) + j * 32 + (lane & 31);
        if (col >= tc.nvalid) continue;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int64_t row = wm * (BIGM / WM) + i * 32 + 8 * (r / 4) + 4 * (lane >> 5) + (r % 4);
            if (tc.r0 + row >= tc.r1) continue;
            float o = g[r];
            if (GATED) o = silu_mul(o, u[r]);
            Cb[row * N + tc.n0 + col] = bf16_bits(o);
        }
    }
}

// ---------------------------------------------------------------------------
// The layer's first launches, fused (moe_layer_forward): routing, the
// permutation and the grouped FFN's tile schedule, in one launch for small
// inputs and two for larger ones, instead of a routing launch, one or two
// permutation launches and a schedule launch.  Each piece computes exactly
// what its own launch computes.
// ---------------------------------------------------------------------------
constexpr int LAYER_NE_MAX = 128;  // experts of the fused schedule (local ones + shared), at most
// The layer's one-workgroup permutation takes at most this many pair-steps
// (pairs x (index bits + 2)); larger inputs take the two fused launches.
// Measured (same-box A/B of the layer step): 4096 pairs over 32 local
// experts (32768 pair-steps: the 512-token decode slice) 0.4971 -> 0.4952 ms
// and 8192 pairs over one expert (32768: the Mixtral EP slice) 0.4440 ->
// 0.4407 ms in two launches; 512 pairs over 32 experts (4096: the 64-token
// decode slice) 0.4102 ms in one workgroup against 0.4115 in two.  The
// threshold lies between the measured points.
constexpr int64_t LAYER_SMALL_WORK = 16 * 1024;

// Small inputs (the one-workgroup permutation), after the routing launch:
// one block of 1024 threads permutes the pairs, then schedules the FFN's
// tiles.  (Routing stays a launch of its own: over many workgroups its
// memory round trips overlap, in one they would follow each other.)
__global__ __launch_bounds__(1024) void layer_perm_sched_kernel(const int32_t *__restrict__ ids, int64_t npairs,
                                                                int e0, int El, int nbits,
                                                                int32_t *__restrict__ counts,
                                                                int32_t *__restrict__ offsets,
                                                                int32_t *__restrict__ row_to_pair,
                                                                int32_t *__restrict__ pair_to_row, int64_t cap,
                                                                int64_t sc, SchedShape sh, SchedOut so,
                                                                int32_t *__restrict__ counters, int64_t n_counters)
{
    permute_dev::permute_small_body(ids, npairs, e0, El, nbits, counts, offsets, row_to_pair, pair_to_row);
    __syncthreads();  // the offsets are visible to the block
    schedule_body<LAYER_NE_MAX>(offsets, El, cap, sc, BIGM, true, sh, so, counters, n_counters);
}

// Larger inputs, at most 64 local experts: block c routes the tokens that
// have a pair in chunk c of the pairs (CH = ROUNDS * 64 pairs, the
// permutation's chunks), writes those whose first pair lies in the chunk
// (every token once over the grid) and counts the chunk's pairs per local
// expert (the permutation's histogram row c).
constexpr int RC_THREADS = 512;  // route/count block: 512 / G tokens routed at once
template <int G, int S, int ROUNDS>
__global__ __launch_bounds__(RC_THREADS) void layer_route_count_kernel(const float *__restrict__ logits, int64_t T, int E,
                                                                int k, int e0, int El, int32_t *__restrict__ ids,
                                                                float *__restrict__ w,
                                                                int32_t *__restrict__ chunk_cnt)
{
    constexpr int CH = ROUNDS * 64;
    __shared__ int32_t lid[CH + 2 * MOE_MAX_TOPK];
    __shared__ float lw[CH + 2 * MOE_MAX_TOPK];
    __shared__ int32_t hist[64];
    const int tid = threadIdx.x;
    const int64_t npairs = T * k, p0 = (int64_t)blockIdx.x * CH;
    const int64_t p1 = p0 + CH < npairs ? p0 + CH : npairs;
    const int64_t ta = p0 / k, tb = (p1 + k - 1) / k;  // tokens [ta, tb) have pairs in the chunk
    const int sub = tid % G;
    for (int64_t t = ta + tid / G; t < tb; t += RC_THREADS / G)
        route_dev::route_token<G, S>(logits + t * E, E, k, sub, lid + (t - ta) * k, lw + (t - ta) * k);
    if (tid < 64) hist[tid] = 0;
    __syncthreads();
    const int64_t tw = (p0 + k - 1) / k;  // the first token whose first pair lies in the chunk
    for (int64_t q = tw * k + tid; q < tb * k; q += RC_THREADS) {
        ids[q] = lid[q - ta * k];
        w[q] = lw[q - ta * k];
    }
    for (int64_t p = p0 + tid; p < p1; p += RC_THREADS) {
        const int le = permute_dev::local_index(lid[p - ta * k], e0, El);
        if (le < El) atomicAdd(&hist[le], 1);
    }
    __syncthreads();
    if (tid < El) chunk_cnt[(int64_t)blockIdx.x * El + tid] = hist[tid];
}

// Then blocks 0 .. nb-1 (nb = ceil(nchunks / 4)) scan and scatter the
// permutation, four chunks each, and block nb schedules the FFN's tiles from
// the expert totals of the histogram (it does not wait for the scatter).
template <int ROUNDS>
__global__ __launch_bounds__(256) void layer_scan_sched_kernel(const int32_t *__restrict__ ids, int64_t npairs,
                                                               int e0, int El, int nbits,
                                                               const int32_t *__restrict__ chunk_cnt, int64_t nchunks,
                                                               int32_t *__restrict__ counts,
                                                               int32_t *__restrict__ offsets,
                                                               int32_t *__restrict__ row_to_pair,
                                                               int32_t *__restrict__ pair_to_row, int64_t cap,
                                                               int64_t sc, SchedShape sh, SchedOut so,
                                                               int32_t *__restrict__ counters, int64_t n_counters)
{
    const int64_t nb = (nchunks + 3) / 4;
    if ((int64_t)blockIdx.x < nb) {
        permute_dev::scan_scatter_body<ROUNDS>(ids, npairs, e0, El, nbits, chunk_cnt, nchunks, counts, offsets,
                                               row_to_pair, pair_to_row, blockIdx.x);
        return;
    }
    // expert totals: thread t sums expert t % El over chunks t / El, + S, ...
    // (S = 256 / El column groups), then one lane per expert adds the groups
    // and the lanes scan the totals into the experts' first rows
    constexpr int UNR = 16;  // loads in flight per thread and pass (one pass for 256 chunks of 16 experts)
    __shared__ int32_t part[256];
    __shared__ int32_t soff[64 + 1];
    const int t = threadIdx.x, S = 256 / El;
    int32_t tot = 0;
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
            for (int u = 0; u < UNR; ++u) tot += v[u];
        }
    }
    part[t] = tot;
    __syncthreads();
    if (t < 64) {
        int32_t total = 0;
        if (t < El)
            for (int g = 0; g < S; ++g) total += part[g * El + t];
        int32_t incl = total;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int32_t o = __shfl_up(incl, off, 64);
            if (t >= off) incl += o;
        }
        if (t < El) soff[t] = incl - total;
        if (t == El - 1) soff[El] = incl;
    }
    __syncthreads();
    schedule_body<LAYER_NE_MAX>(soff, El, cap, sc, BIGM, true, sh, so, counters, n_counters);
}

}  // namespace

namespace {

std::mutex g_dts_mu;
bool g_dts_on = false;
std::vector<int> g_dts_kind;  // slot -> kernel kind

// The next device-timestamp slot for a launch of `kind`, or -1 when device
// timing is off or the table is full.
int device_ts_slot(int kind)
{
    std::lock_guard<std::mutex> lk(g_dts_mu);
    if (!g_dts_on || g_dts_kind.size() >= (size_t)DEV_TS_SLOTS) return -1;
    g_dts_kind.push_back(kind);
    return (int)g_dts_kind.size() - 1;
}

// Whether a grouped GEMM launch streams its weights: when the local
// experts' weights of the GEMM (elems bf16 values) exceed half of the 256 MB
// last-level cache, they do not stay cached from one step to the next, and
// the small-row tiles (the decode path, one reader per weight panel) load
// them with the non-temporal hint.  Measured on the DeepSeek-V3-shaped
// decode slices: gate-up 285 -> 252 us (T = 64), 343 -> 301 us (T = 512),
// down 155 -> 137 us and 188 -> 169 us.  Below the threshold the weights
// are re-read from the cache in the next step (the Qwen-shaped slice's
// 100 MB, prefill tail tiles sharing panels with large tiles), and the hint
// made those launches 1-10% slower.
constexpr int64_t STREAM_WEIGHT_BYTES = (int64_t)128 << 20;
bool weights_streamed(int64_t elems)
{
    return elems * 2 > STREAM_WEIGHT_BYTES;
}

int device_cus()
{
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
        cus = 256;
    return (cus + 7) / 8 * 8;  // whole rounds over the 8 dies
}

// Shape of both GEMMs for the schedule, with the per-GEMM constants of its
// small-row plans.
SchedShape sched_shape(int H, int Is, int grid)
{
    SchedShape sh{(int)ceil_div(Is, BIGN / 2), H / BIG_BK, (int)ceil_div(H, BIGN), Is / BIG_BK, grid, {}, {}};
    const int nk[2] = {sh.nk_gu, sh.nk_dn};
    const SmallKind kinds[2] = {SMALL64, SMALL128};
    for (int gi = 0; gi < 2; ++gi)
        for (int k = 0; k < 2; ++k) {
            sh.wfit[gi][k] = whole_fit(nk[gi], kinds[k].whole_num);
            sh.whole[gi][k] = whole_time(nk[gi], kinds[k].whole_num);
        }
    return sh;
}

// Workspace layout of the grouped FFN (every part 256-byte aligned):
//   prefix large, gate-up and down [El+1] each | prefix small, gate-up and
//   down [El+1] + small tile height each | class cut, gate-up and down [El] each |
//   small m-tiles (expert, first row, end row), gate-up and down [mts] each |
//   tile counters: large gate-up, large down, small gate-up, small down |
//   split-K partial slots: small [2*G][SLOT_SMALL], large [2*G][SLOT_BIG] fp32 |
//   h [cap, I_s] bf16
// The two GEMMs run one after the other on the stream and share the partial
// slots; each keeps its own tile counters.
struct FfnLayout {
    bool big;
    int64_t t_gu, t_dn, ts_gu, ts_dn;  // tile-count bounds per class and GEMM
    int grid;                          // persistent workgroups of a large-tile launch
    size_t off_pre_ld, off_pre_s, off_pre_sd, off_split, off_split_d, off_mt, off_mt_d, off_cnt, off_part_s, off_part,
        off_h, total;
    FfnLayout(int64_t cap, int El, int H, int Is)
    {
        big = (H % BIG_BK == 0) && (Is % BIG_BK == 0) && H >= 2 * BIG_BK && Is >= 2 * BIG_BK;
        const int bm = big ? BIGM : BM;
        const int64_t mt = ceil_div(cap, bm) + El;
        t_gu = mt * ceil_div(Is, big ? BIGN / 2 : BN);
        t_dn = mt * ceil_div(H, big ? BIGN : BN);
        // a small-row expert or leftover has at most max_rows rows: at most
        // two m-tiles of either height; the largest expert may add up to
        // ND_SCHED - 1 large m-tiles (4 small m-tiles each at most)
        static_assert(SMALL64.max_rows <= 2 * SMALL64.rows && SMALL128.max_rows <= 2 * SMALL128.rows, "");
        const int64_t mts = big ? (int64_t)El * 2 + (ND_SCHED - 1) * (BIGM / SMALL64.rows) : 0;
        ts_gu = mts * ceil_div(Is, BIGN / 2);
        ts_dn = mts * ceil_div(H, BIGN);
        grid = device_cus();
        const size_t slots = big ? 2 * (size_t)grid : 0;
        off_pre_ld = align256((size_t)(El + 1) * sizeof(int32_t));
        off_pre_s = off_pre_ld + align256((size_t)(El + 1) * sizeof(int32_t));
        off_pre_sd = off_pre_s + align256((size_t)(El + 2) * sizeof(int32_t));
        off_split = off_pre_sd + align256((size_t)(El + 2) * sizeof(int32_t));
        off_split_d = off_split + align256((size_t)El * sizeof(int32_t));
        off_mt = off_split_d + align256((size_t)El * sizeof(int32_t));
        off_mt_d = off_mt + align256((size_t)mts * sizeof(int4));
        off_cnt = off_mt_d + align256((size_t)mts * sizeof(int4));
        off_part_s = off_cnt + align256((size_t)(t_gu + t_dn + ts_gu + ts_dn) * sizeof(int32_t));
        off_part = off_part_s + align256(slots * SLOT_SMALL * sizeof(float));
        off_h = off_part + align256(slots * SLOT_BIG * sizeof(float));
        total = off_h + align256((size_t)cap * Is * 2);
    }
};

}  // namespace

size_t ffn_workspace_bytes(int64_t cap, int El, int H, int Is)
{
    return FfnLayout(cap, El, H, Is).total;
}

bool ffn_large_tiles(int64_t x_rows, int64_t rows, int H, int Is)
{
    // K a multiple of 64 with at least two slices, every operand
    // addressable with 32-bit buffer offsets, and small-row tile numbers
    // below 2^31 (at most 2 * 1025 + 28 m-tiles, with a shared expert, of
    // 2^26 / 128 + 1 n-tiles)
    if (H % BIG_BK || Is % BIG_BK || H < 2 * BIG_BK || Is < 2 * BIG_BK) return false;
    if (H > (1 << 26) || Is > (1 << 26)) return false;
    const int64_t lim = ((int64_t)1 << 32) - 4 * (int64_t)(H > Is ? H : Is);
    return x_rows * (int64_t)H * 2 < lim && rows * (int64_t)H * 2 < lim && rows * (int64_t)Is * 2 < lim;
}

namespace {

// One grouped-FFN call: its row space (the routed rows [0, cap), then the
// shared expert's rows), the workspace parts and the schedule's arguments.
struct FfnCall {
    FfnLayout L;
    int El, ne, H, Is;
    int64_t cap, sc, rows, n_cnt;
    bool big;
    int32_t *pre, *pre_ld, *pre_s, *pre_sd, *split, *split_d, *cnt;
    int4 *mt_g, *mt_d;
    float *part_s, *part;
    uint16_t *h, *h_sh;
    SchedShape sh;
    SchedOut so;
    FfnCall(int64_t x_rows, bool gather, int El_, int64_t cap_, int H_, int Is_, int64_t sc_, void *ws)
        : L(cap_ + sc_, El_ + (sc_ > 0 ? 1 : 0), H_, Is_), El(El_), ne(El_ + (sc_ > 0 ? 1 : 0)), H(H_), Is(Is_),
          cap(cap_), sc(sc_), rows(cap_ + sc_)
    {
        char *base = static_cast<char *>(ws);
        pre = reinterpret_cast<int32_t *>(base);                     // large class, gate-up
        pre_ld = reinterpret_cast<int32_t *>(base + L.off_pre_ld);  // large class, down
        pre_s = reinterpret_cast<int32_t *>(base + L.off_pre_s);    // small class, gate-up
        pre_sd = reinterpret_cast<int32_t *>(base + L.off_pre_sd);  // small class, down
        split = reinterpret_cast<int32_t *>(base + L.off_split);    // class cut, gate-up
        split_d = reinterpret_cast<int32_t *>(base + L.off_split_d);
        mt_g = reinterpret_cast<int4 *>(base + L.off_mt);  // small m-tiles, gate-up
        mt_d = reinterpret_cast<int4 *>(base + L.off_mt_d);
        cnt = reinterpret_cast<int32_t *>(base + L.off_cnt);
        part_s = reinterpret_cast<float *>(base + L.off_part_s);
        part = reinterpret_cast<float *>(base + L.off_part);
        h = reinterpret_cast<uint16_t *>(base + L.off_h);
        h_sh = h + cap * Is;  // the shared expert's h rows
        big = ffn_large_tiles(gather ? x_rows : rows, rows, H, Is);
        n_cnt = big ? L.t_gu + L.t_dn + L.ts_gu + L.ts_dn : 0;
        sh = sched_shape(H, Is, L.grid);
        so = SchedOut{{pre, pre_ld}, {pre_s, pre_sd}, {split, split_d}, {mt_g, mt_d}};
    }
    int bm() const { return big ? BIGM : BM; }
};

// The GEMM launches of a call whose schedule is already in the workspace.
hipError_t launch_gemms(const FfnCall &c, const uint16_t *x, int64_t x_rows, const int32_t *row_index, int kdiv,
                        const int32_t *offsets, const uint16_t *w13, const uint16_t *w2, uint16_t *y,
                        int64_t shared_begin, const uint16_t *sw13, const uint16_t *sw2, uint16_t *shared_y,
                        hipStream_t s)
{
    const FfnLayout &L = c.L;
    const int El = c.El, ne = c.ne, H = c.H, Is = c.Is;
    const int64_t cap = c.cap, sc = c.sc, rows = c.rows;
    hipError_t err;
    if (c.big) {
        int32_t *c_gu = c.cnt, *c_dn = c.cnt + L.t_gu, *cs_gu = c_dn + L.t_dn, *cs_dn = cs_gu + L.ts_gu;
        {
            KernelTimer timer(MOE_K_GATE_UP, s);
            const GemmArgs g{x,   row_index, kdiv, x_rows, offsets, c.split, El, ne, cap, sc, shared_begin,
                             Is,  H,         w13,  (int64_t)2 * Is * H, sw13, Is, c.h, c.h_sh};
            const TileClass sm{c.pre_s, c.mt_g, cs_gu, c.part_s}, lg{c.pre, nullptr, c_gu, c.part};
            if (weights_streamed((int64_t)El * 2 * Is * H))
                gemm_grouped<true, true><<<dim3((unsigned)L.grid), dim3(GEMM_THREADS), 0, s>>>(
                    g, sm, lg, device_ts_slot(MOE_K_GATE_UP));
            else
                gemm_grouped<true, false><<<dim3((unsigned)L.grid), dim3(GEMM_THREADS), 0, s>>>(
                    g, sm, lg, device_ts_slot(MOE_K_GATE_UP));
            if ((err = hipGetLastError()) != hipSuccess) return err;
        }
        if (H / BIG_BK >= SPLIT_MIN_NK) {  // the large tiles may have been split over K
            KernelTimer timer(MOE_K_SPLITK_REDUCE, s);
            splitk_reduce<true><<<dim3(REDUCE_GRID), dim3(GEMM_THREADS), 0, s>>>(
                offsets, c.split, c.pre, El, ne, cap, sc, Is, H, L.grid, c.part, c.h, c.h_sh);
            if ((err = hipGetLastError()) != hipSuccess) return err;
        }
        {
            KernelTimer timer(MOE_K_DOWN, s);
            const GemmArgs g{c.h, nullptr, 1, rows, offsets, c.split_d, El, ne, cap, sc, shared_begin,
                             H,   Is,      w2, (int64_t)H * Is, sw2, 0, y, shared_y};
            const TileClass sm{c.pre_sd, c.mt_d, cs_dn, c.part_s}, lg{c.pre_ld, nullptr, c_dn, c.part};
            if (weights_streamed((int64_t)El * H * Is))
                gemm_grouped<false, true><<<dim3((unsigned)L.grid), dim3(GEMM_THREADS), 0, s>>>(
                    g, sm, lg, device_ts_slot(MOE_K_DOWN));
            else
                gemm_grouped<false, false><<<dim3((unsigned)L.grid), dim3(GEMM_THREADS), 0, s>>>(
                    g, sm, lg, device_ts_slot(MOE_K_DOWN));
            if ((err = hipGetLastError()) != hipSuccess) return err;
        }
        if (Is / BIG_BK >= SPLIT_MIN_NK) {
            KernelTimer timer(MOE_K_SPLITK_REDUCE, s);
            splitk_reduce<false><<<dim3(REDUCE_GRID), dim3(GEMM_THREADS), 0, s>>>(
                offsets, c.split_d, c.pre_ld, El, ne, cap, sc, H, Is, L.grid, c.part, y, shared_y);
            if ((err = hipGetLastError()) != hipSuccess) return err;
        }
        return hipSuccess;
    }
    // general path: tiles of BM rows (the layout sized the tile counters with
    // the large tiles, which is an upper bound here too)
    const int64_t mt = ceil_div(cap, BM) + El;
    {
        KernelTimer timer(MOE_K_GATE_UP, s);
        int64_t tiles = mt * ceil_div(Is, BN);
        int64_t grid = tiles < 2048 ? tiles : 2048;
        gemm_kernel<true><<<dim3((unsigned)grid), dim3(256), 0, s>>>(
            x, row_index, kdiv, offsets, c.pre, El, cap, Is, H, w13, (int64_t)2 * Is * H, Is, c.h);
        if ((err = hipGetLastError()) != hipSuccess) return err;
    }
    {
        KernelTimer timer(MOE_K_DOWN, s);
        int64_t tiles = mt * ceil_div(H, BN);
        int64_t grid = tiles < 2048 ? tiles : 2048;
        gemm_kernel<false><<<dim3((unsigned)grid), dim3(256), 0, s>>>(
            c.h, nullptr, 1, offsets, c.pre, El, cap, H, Is, w2, (int64_t)H * Is, 0, y);
        if ((err = hipGetLastError()) != hipSuccess) return err;
    }
    return hipSuccess;
}

}  // namespace

hipError_t launch_grouped_ffn(const uint16_t *x, int64_t x_rows, const int32_t *row_index, int kdiv,
                              const int32_t *offsets, int El, int64_t cap, int H, int Is,
                              const uint16_t *w13, const uint16_t *w2, uint16_t *y, int64_t shared_begin,
                              int64_t shared_rows, const uint16_t *sw13, const uint16_t *sw2,
                              uint16_t *shared_y, void *ws, hipStream_t s)
{
    if (cap + shared_rows == 0) return hipSuccess;
    const FfnCall c(x_rows, row_index != nullptr, El, cap, H, Is, shared_rows, ws);
    if (shared_rows > 0 && !c.big) return hipErrorNotSupported;  // the host API checks this first
    {
        KernelTimer timer(MOE_K_SCHEDULE, s);
        const unsigned threads = (unsigned)(ceil_div(c.ne > 256 ? c.ne : 256, 64) * 64);
        schedule_kernel<<<dim3(1), dim3(threads), 0, s>>>(offsets, El, cap, shared_rows, c.bm(), c.big, c.sh, c.so,
                                                          c.cnt, c.n_cnt);
        hipError_t err = hipGetLastError();
        if (err != hipSuccess) return err;
    }
    return launch_gemms(c, x, x_rows, row_index, kdiv, offsets, w13, w2, y, shared_begin, sw13, sw2, shared_y, s);
}

namespace {

// The token group of the fused routing: 16 lanes per token, each holding
// E / 16 logits (64 lanes above 512 experts), so a block of 256 threads
// routes 16 tokens at a time.  (The weights do not depend on the group
// width: route_token sums them in rank order.)
template <template <int, int> class F, typename... A>
hipError_t by_experts(int E, A... a)
{
    if (E <= 8) return F<8, 1>::go(a...);
    if (E <= 16) return F<16, 1>::go(a...);
    if (E <= 32) return F<16, 2>::go(a...);
    if (E <= 64) return F<16, 4>::go(a...);
    if (E <= 128) return F<16, 8>::go(a...);
    if (E <= 256) return F<16, 16>::go(a...);
    if (E <= 512) return F<16, 32>::go(a...);
    return F<64, 16>::go(a...);
}

template <int G, int S>
struct LaunchRouteCount {
    static hipError_t go(const float *logits, int64_t T, int E, int k, int e0, int El, int32_t *ids, float *w,
                         int32_t *chunk_cnt, int64_t nchunks, bool short_chunks, hipStream_t s)
    {
        if (short_chunks)
            layer_route_count_kernel<G, S, 4><<<dim3((unsigned)nchunks), dim3(RC_THREADS), 0, s>>>(
                logits, T, E, k, e0, El, ids, w, chunk_cnt);
        else
            layer_route_count_kernel<G, S, 16><<<dim3((unsigned)nchunks), dim3(RC_THREADS), 0, s>>>(
                logits, T, E, k, e0, El, ids, w, chunk_cnt);
        return hipGetLastError();
    }
};

}  // namespace

bool layer_fused_prep(int64_t T, int k, int El, int H, int Is, int64_t sc)
{
    const int64_t npairs = T * k, cap = T * (k < El ? k : El);
    int nbits = 0;
    while ((1 << nbits) < El + 2) ++nbits;
    const bool fuse = npairs > 0 && El <= 64 && El + (sc > 0 ? 1 : 0) <= LAYER_NE_MAX &&
                      ffn_large_tiles(T, cap + sc, H, Is);
    const bool small = npairs <= permute_dev::SMALL_PAIRS && npairs * (nbits + 2) <= LAYER_SMALL_WORK;
    return fuse && (small || permute_chunks(T, k, El) <= permute_dev::SCAN_SCATTER_MAX_CHUNKS);
}

hipError_t launch_layer(const uint16_t *x, const float *logits, int64_t T, int E, int k, int e0, int El, int H,
                        int Is, const uint16_t *w13, const uint16_t *w2, int64_t sb, int64_t sc,
                        const uint16_t *sw13, const uint16_t *sw2, int32_t *ids, float *w, int32_t *counts,
                        int32_t *offsets, int32_t *r2p, int32_t *p2r, uint16_t *y, uint16_t *shared_y,
                        uint16_t *out, int32_t *ws_perm, void *ws_ffn, hipStream_t s)
{
    const int64_t npairs = T * k, cap = T * (k < El ? k : El);
    hipError_t err;
    if (!layer_fused_prep(T, k, El, H, Is, sc)) {
        // the separate launches of the four calls
        if ((err = launch_route(logits, T, E, k, ids, w, s)) != hipSuccess) return err;
        if ((err = launch_permute(ids, T, k, e0, El, counts, offsets, r2p, p2r, nullptr, 0, nullptr, cap, ws_perm,
                                  s)) != hipSuccess)
            return err;
        if ((err = launch_grouped_ffn(x, T, r2p, k, offsets, El, cap, H, Is, w13, w2, y, sb, sc, sw13, sw2,
                                      shared_y, ws_ffn, s)) != hipSuccess)
            return err;
        return launch_combine(y, cap, p2r, w, T, k, H, sc > 0 ? shared_y : nullptr, sb, sc, 0, out, s);
    }
    const FfnCall c(T, true, El, cap, H, Is, sc, ws_ffn);
    int nbits = 0;
    while ((1 << nbits) < El + 2) ++nbits;
    const bool small = npairs <= permute_dev::SMALL_PAIRS && npairs * (nbits + 2) <= LAYER_SMALL_WORK;
    if (small && (err = launch_route(logits, T, E, k, ids, w, s)) != hipSuccess) return err;
    {
        KernelTimer timer(MOE_K_LAYER_PREP, s);
        if (small) {
            layer_perm_sched_kernel<<<dim3(1), dim3(1024), 0, s>>>(ids, npairs, e0, El, nbits, counts, offsets, r2p,
                                                                    p2r, cap, sc, c.sh, c.so, c.cnt, c.n_cnt);
            err = hipGetLastError();
        } else {
            const int64_t nchunks = permute_chunks(T, k, El);
            const bool short_chunks = permute_dev::chunk_pairs(npairs, El) == 256;
            err = by_experts<LaunchRouteCount>(E, logits, T, E, k, e0, El, ids, w, ws_perm, nchunks, short_chunks, s);
            if (err != hipSuccess) return err;
            const unsigned blocks = (unsigned)(ceil_div(nchunks, 4) + 1);
            if (short_chunks)
                layer_scan_sched_kernel<4><<<dim3(blocks), dim3(256), 0, s>>>(
                    ids, npairs, e0, El, nbits, ws_perm, nchunks, counts, offsets, r2p, p2r, cap, sc, c.sh, c.so, c.cnt,
                    c.n_cnt);
            else
                layer_scan_sched_kernel<16><<<dim3(blocks), dim3(256), 0, s>>>(
                    ids, npairs, e0, El, nbits, ws_perm, nchunks, counts, offsets, r2p, p2r, cap, sc, c.sh, c.so, c.cnt,
                    c.n_cnt);
            err = hipGetLastError();
        }
        if (err != hipSuccess) return err;
    }
    if ((err = launch_gemms(c, x, T, r2p, k, offsets, w13, w2, y, sb, sw13, sw2, shared_y, s)) != hipSuccess)
        return err;
    return launch_combine(y, cap, p2r, w, T, k, H, sc > 0 ? shared_y : nullptr, sb, sc, 0, out, s);
}

}  // namespace moe

// Device-side timestamps of the grouped GEMM launches (see include/libmoe.h).
extern "C" moe_status moe_timing_device_enable(int enable)
{
    std::lock_guard<std::mutex> lk(moe::g_dts_mu);
    moe::g_dts_on = enable != 0;
    return MOE_OK;
}

extern "C" moe_status moe_timing_device_clear(void)
{
    std::lock_guard<std::mutex> lk(moe::g_dts_mu);
    moe::g_dts_kind.clear();
    return MOE_OK;
}

extern "C" moe_status moe_timing_device_reset(void)
{
    void *p = nullptr;
    hipError_t err = hipGetSymbolAddress(&p, HIP_SYMBOL(moe::g_dev_ts));
    if (err == hipSuccess) err = hipDeviceSynchronize();
    const size_t half = sizeof(unsigned long long) * 8 * moe::DEV_TS_SLOTS;
    if (err == hipSuccess) err = hipMemset(p, 0xff, half);                             // starts: max
    if (err == hipSuccess) err = hipMemset(static_cast<char *>(p) + half, 0, half);  // ends: 0
    if (err == hipSuccess) err = hipDeviceSynchronize();
    if (err != hipSuccess) return moe::set_error(MOE_ERR_HIP, "moe_timing_device_reset: %s", hipGetErrorString(err));
    return MOE_OK;
}

extern "C" moe_status moe_timing_device_read(int kind, double *total_ms, int64_t *launches)
{
    if (total_ms == nullptr || launches == nullptr || kind < 0 || kind >= MOE_K_COUNT)
        return moe::set_error(MOE_ERR_INVALID_ARG, "moe_timing_device_read: bad kind %d or null output", kind);
    std::vector<unsigned long long> ts(2 * 8 * moe::DEV_TS_SLOTS);
    hipError_t err = hipDeviceSynchronize();
    if (err == hipSuccess)
        err = hipMemcpyFromSymbol(ts.data(), HIP_SYMBOL(moe::g_dev_ts), ts.size() * sizeof(unsigned long long), 0,
                                  hipMemcpyDeviceToHost);
    if (err != hipSuccess) return moe::set_error(MOE_ERR_HIP, "moe_timing_device_read: %s", hipGetErrorString(err));
    std::lock_guard<std::mutex> lk(moe::g_dts_mu);
    double sum = 0.0;
    int64_t n = 0;
    for (size_t i = 0; i < moe::g_dts_kind.size(); ++i) {
        if (moe::g_dts_kind[i] != kind) continue;
        unsigned long long first = ~0ull, last = 0;  // over the dies
        for (int d = 0; d < 8; ++d) {
            const unsigned long long a = ts[(size_t)d * moe::DEV_TS_SLOTS + i];
            const unsigned long long b = ts[(size_t)(8 + d) * moe::DEV_TS_SLOTS + i];
            if (b == 0 || a == ~0ull || b < a) continue;  // no workgroup of this die ran since the reset
            first = a < first ? a : first;
            last = b > last ? b : last;
        }
        if (last == 0) continue;
        sum += (double)(last - first) * 1e-5;  // 100 MHz ticks -> ms
        ++n;
    }
    *total_ms = sum;
    *launches = n;
    return MOE_OK;
}
