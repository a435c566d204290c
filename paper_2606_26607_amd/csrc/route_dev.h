// Gating device code shared by the routing kernel and the fused layer
// kernels: softmax top-k over router logits, one lane group per token.
//
// A token's E logits are spread over a group of G lanes (G = 8..64, a power
// of two), S logits per lane, G*S >= E.  Each logit becomes
// a 64-bit key whose high word orders floats (with -0.0 folded onto +0.0)
// and whose low word is ~id, so the largest key is the largest logit with
// the lowest expert id.  k rounds of a group-wide max over the keys pick the
// experts in rank order; the weights are exp(l_j - l_0) / sum_i exp(l_i - l_0)
// over the kept logits (the sum taken in rank order), which equals the full
// softmax renormalised over the kept experts.
#pragma once
#include <type_traits>

#include "moe_internal.h"

namespace moe {
namespace route_dev {


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

// Lane exchange inside a row of 16 lanes (DPP, no LDS round trip):
// CTRL 0xB1 swaps neighbours (quad_perm 1,0,3,2), 0x4E swaps pairs
// (quad_perm 2,3,0,1), 0x141 mirrors each half row, 0x140 mirrors the row.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp32(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, CTRL, 0xF, 0xF, true);
}

// Lane `src`'s value of v (a 32- or 64-bit value), the same in every lane.
template <typename T>
__device__ __forceinline__ T read_lane(T v, int src)
{
    if constexpr (sizeof(T) == 8) {
        const uint64_t u = *reinterpret_cast<uint64_t *>(&v);
        const uint64_t o = (uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, src) |
                           ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), src) << 32);
        return *reinterpret_cast<const T *>(&o);
    } else {
        const uint32_t o = (uint32_t)__builtin_amdgcn_readlane((int)*reinterpret_cast<uint32_t *>(&v), src);
        return *reinterpret_cast<const T *>(&o);
    }
}

// The steps that combine a group of G lanes.  Within a row of 16 lanes DPP
// moves: after the two quad swaps every quad agrees, the half-row mirror
// joins the two quads of a half row, the row mirror joins the halves.  Wider
// groups (32 or 64 lanes, the whole wave active) then combine their rows'
// results read from lanes 0, 16, 32 and 48 into scalar registers, instead of
// cross-lane shuffles through the LDS unit, each of which costs a round trip.
template <int G, typename T, typename Op>
__device__ __forceinline__ T group_reduce(T v, Op op)
{
    if constexpr (G == 32 || G == 64) {
        v = group_reduce<16>(v, op);
        const T r0 = read_lane(v, 0), r1 = read_lane(v, 16), r2 = read_lane(v, 32), r3 = read_lane(v, 48);
        if constexpr (G == 64) return op(op(r0, r1), op(r2, r3));
        else return (threadIdx.x & 32) ? op(r2, r3) : op(r0, r1);
    } else if constexpr (G <= 16) {
        auto step = [&](auto ctrl) {
            constexpr int C = decltype(ctrl)::value;
            if constexpr (sizeof(T) == 8) {
                const uint64_t u = *reinterpret_cast<uint64_t *>(&v);
                const uint64_t o = (uint64_t)dpp32<C>((uint32_t)u) | ((uint64_t)dpp32<C>((uint32_t)(u >> 32)) << 32);
                v = op(v, *reinterpret_cast<const T *>(&o));
            } else {
                const uint32_t o = dpp32<C>(*reinterpret_cast<uint32_t *>(&v));
                v = op(v, *reinterpret_cast<const T *>(&o));
            }
        };
        step(std::integral_constant<int, 0xB1>{});
        if constexpr (G >= 4) step(std::integral_constant<int, 0x4E>{});
        if constexpr (G >= 8) step(std::integral_constant<int, 0x141>{});
        if constexpr (G >= 16) step(std::integral_constant<int, 0x140>{});
    } else {
        static_assert(G <= 64, "a lane group lies within one wave");
    }
    return v;
}

template <int G>
__device__ __forceinline__ uint64_t group_max(uint64_t v)
{
    return group_reduce<G>(v, [](uint64_t a, uint64_t b) { return a > b ? a : b; });
}



// Top-k of one token's logits `row` [E] on a group of G lanes (sub = lane
// index in the group, all G lanes active): lanes sub < k write
// ids[sub] and w[sub].
template <int G, int S>
__device__ __forceinline__ void route_token(const float *__restrict__ row, int E, int k, int sub,
                                            int32_t *__restrict__ ids, float *__restrict__ w)
{
    // All S loads go out before the first is used: a lane past E reads
    // logit E-1 (in bounds) and drops it.  Guarded by e < E instead, each
    // load sat in its own branch and waited for its data before the next
    // was issued, S memory round trips in a row.
    float lv[S];
#pragma unroll
    for (int m = 0; m < S; ++m) {
        const int e = sub + m * G;
        lv[m] = row[e < E ? e : E - 1];
    }
    uint64_t key[S];
#pragma unroll
    for (int m = 0; m < S; ++m) {
        const int e = sub + m * G;
        key[m] = e < E ? ((uint64_t)order_key(lv[m]) << 32) | (uint32_t)(~e) : 0ull;
    }
    // round j's winner is known to every lane of the group, so each lane
    // adds exp(l_j - l_0) in rank order: the normalising sum is the same
    // whatever the group width
    uint64_t mine = 0;
    float l0 = 0.f, z = 0.f, ex = 0.f;
    for (int j = 0; j < k; ++j) {
        uint64_t best = 0;
#pragma unroll
        for (int m = 0; m < S; ++m) best = key[m] > best ? key[m] : best;
        uint64_t win = group_max<G>(best);
#pragma unroll
        for (int m = 0; m < S; ++m)
            if (key[m] == win) key[m] = 0;  // ids are unique: exactly one slot matches
        const float l = key_value((uint32_t)(win >> 32));
        if (j == 0) l0 = l;
        const float e = expf(l - l0);
        z += e;
        if (sub == j) {
            mine = win;
            ex = e;
        }
    }
    if (sub < k) {
        ids[sub] = (int32_t)(~(uint32_t)mine);
        w[sub] = ex / z;
    }
}

}  // namespace route_dev
}  // namespace moe
