// libmoe C ABI: host-side argument validation, then kernel launches.
// Validation happens before anything is enqueued, so a rejected call
// touches no buffer; only the grouped-FFN workspace size queries the device
// (its compute unit count).
#include <stdarg.h>
#include <stdio.h>

#include "moe_internal.h"

using namespace moe;

namespace {

thread_local char g_msg[512] = "no error";

moe_status vfail(moe_status st, const char *fmt, va_list ap)
{
    vsnprintf(g_msg, sizeof g_msg, fmt, ap);
    return st;
}

moe_status fail(moe_status st, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vfail(st, fmt, ap);
    va_end(ap);
    return st;
}

moe_status hip_status(hipError_t err, const char *what)
{
    if (err == hipSuccess) return MOE_OK;
    return fail(MOE_ERR_HIP, "%s: %s", what, hipGetErrorString(err));
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

moe_status check_topk(int64_t T, int E, int k)
{
    if (T < 0) return fail(MOE_ERR_INVALID_ARG, "T=%lld is negative", (long long)T);
    if (E < 1) return fail(MOE_ERR_INVALID_ARG, "E=%d must be >= 1", E);
    if (k < 1 || k > E) return fail(MOE_ERR_INVALID_ARG, "k=%d must be in [1, E=%d]", k, E);
    if (E > MOE_MAX_EXPERTS) return fail(MOE_ERR_UNSUPPORTED, "E=%d exceeds %d", E, MOE_MAX_EXPERTS);
    if (k > MOE_MAX_TOPK) return fail(MOE_ERR_UNSUPPORTED, "k=%d exceeds %d", k, MOE_MAX_TOPK);
    if (T * (int64_t)k >= ((int64_t)1 << 31))
        return fail(MOE_ERR_UNSUPPORTED, "T*k=%lld does not fit int32 indices", (long long)(T * k));
    return MOE_OK;
}

moe_status check_width(const char *name, int v)
{
    if (v <= 0) return fail(MOE_ERR_INVALID_ARG, "%s=%d must be positive", name, v);
    if (v % 8) return fail(MOE_ERR_UNSUPPORTED, "%s=%d is not a multiple of 8", name, v);
    return MOE_OK;
}

}  // namespace

moe_status moe::set_error(moe_status st, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vfail(st, fmt, ap);
    va_end(ap);
    return st;
}

extern "C" const char *moe_status_str(int status)
{
    switch (status) {
    case MOE_OK: return "MOE_OK";
    case MOE_ERR_INVALID_ARG: return "MOE_ERR_INVALID_ARG";
    case MOE_ERR_UNSUPPORTED: return "MOE_ERR_UNSUPPORTED";
    case MOE_ERR_WORKSPACE: return "MOE_ERR_WORKSPACE";
    case MOE_ERR_HIP: return "MOE_ERR_HIP";
    default: return "MOE_ERR_UNKNOWN";
    }
}

extern "C" const char *moe_last_error(void) { return g_msg; }

extern "C" int moe_version(void) { return 8; }

extern "C" moe_status moe_route(const float *logits, int64_t T, int E, int k, int32_t *topk_ids,
                                float *topk_w, void *stream)
{
    moe_status st = check_topk(T, E, k);
    if (st != MOE_OK) return st;
    if (T > 0 && (!logits || !topk_ids || !topk_w))
        return fail(MOE_ERR_INVALID_ARG, "moe_route: null pointer");
    return hip_status(launch_route(logits, T, E, k, topk_ids, topk_w, (hipStream_t)stream),
                      "moe_route launch");
}

extern "C" size_t moe_permute_workspace_size(int64_t T, int k, int n_local_experts)
{
    if (T < 0 || k < 1 || n_local_experts < 1) return 0;
    return align256((size_t)(permute_chunks(T, k, n_local_experts) + 1) * (size_t)n_local_experts *
                    sizeof(int32_t));
}

extern "C" moe_status moe_permute(const int32_t *topk_ids, int64_t T, int k, int E, int expert_begin,
                                  int n_local_experts, int32_t *counts, int32_t *offsets,
                                  int32_t *row_to_pair, int32_t *pair_to_row, const uint16_t *x,
                                  int H, uint16_t *x_perm, void *workspace, size_t workspace_bytes,
                                  void *stream)
{
    moe_status st = check_topk(T, E, k);
    if (st != MOE_OK) return st;
    const int El = n_local_experts;
    if (El < 1 || expert_begin < 0 || expert_begin + El > E)
        return fail(MOE_ERR_INVALID_ARG, "local experts [%d, %d+%d) not inside [0, E=%d)",
                    expert_begin, expert_begin, El, E);
    if (!counts || !offsets) return fail(MOE_ERR_INVALID_ARG, "moe_permute: null counts/offsets");
    if (T > 0 && (!topk_ids || !row_to_pair || !pair_to_row))
        return fail(MOE_ERR_INVALID_ARG, "moe_permute: null index array");
    if (x_perm) {
        if ((st = check_width("H", H)) != MOE_OK) return st;
        if (T > 0 && !x) return fail(MOE_ERR_INVALID_ARG, "moe_permute: x_perm given without x");
        if (!aligned16(x) || !aligned16(x_perm))
            return fail(MOE_ERR_INVALID_ARG, "moe_permute: x / x_perm not 16-byte aligned");
    }
    const size_t need = moe_permute_workspace_size(T, k, El);
    if (!workspace || workspace_bytes < need)
        return fail(MOE_ERR_WORKSPACE, "moe_permute: workspace %zu < %zu bytes", workspace_bytes, need);
    const int64_t cap = T * (k < El ? k : El);
    return hip_status(launch_permute(topk_ids, T, k, expert_begin, El, counts, offsets, row_to_pair,
                                     pair_to_row, x, H, x_perm, cap, static_cast<int32_t *>(workspace),
                                     (hipStream_t)stream),
                      "moe_permute launch");
}

extern "C" moe_status moe_permute_noalloc(const int32_t *topk_ids, int64_t T, int k, int E, int expert_begin,
                                          int n_local_experts, int32_t *counts, int32_t *offsets,
                                          int32_t *row_to_pair, int32_t *pair_to_row, const uint16_t *x, int H,
                                          uint16_t *x_perm, void *stream)
{
    // the same checks as moe_permute, then the size bound of the static scratch
    moe_status st = check_topk(T, E, k);
    if (st != MOE_OK) return st;
    const int El = n_local_experts;
    if (El < 1 || expert_begin < 0 || expert_begin + El > E)
        return fail(MOE_ERR_INVALID_ARG, "local experts [%d, %d+%d) not inside [0, E=%d)",
                    expert_begin, expert_begin, El, E);
    if (!counts || !offsets) return fail(MOE_ERR_INVALID_ARG, "moe_permute_noalloc: null counts/offsets");
    if (T > 0 && (!topk_ids || !row_to_pair || !pair_to_row))
        return fail(MOE_ERR_INVALID_ARG, "moe_permute_noalloc: null index array");
    if (x_perm) {
        if ((st = check_width("H", H)) != MOE_OK) return st;
        if (T > 0 && !x) return fail(MOE_ERR_INVALID_ARG, "moe_permute_noalloc: x_perm given without x");
        if (!aligned16(x) || !aligned16(x_perm))
            return fail(MOE_ERR_INVALID_ARG, "moe_permute_noalloc: x / x_perm not 16-byte aligned");
    }
    const size_t need = moe_permute_workspace_size(T, k, El);
    if (need > MOE_PERMUTE_SCRATCH_BYTES)
        return fail(MOE_ERR_UNSUPPORTED,
                    "moe_permute_noalloc: T=%lld, k=%d, %d local experts need %zu bytes of scratch, "
                    "above the static %u (use moe_permute with a workspace)",
                    (long long)T, k, El, need, (unsigned)MOE_PERMUTE_SCRATCH_BYTES);
    int32_t *scratch = nullptr;
    if ((st = hip_status(permute_scratch(&scratch), "moe_permute_noalloc scratch")) != MOE_OK) return st;
    const int64_t cap = T * (k < El ? k : El);
    return hip_status(launch_permute(topk_ids, T, k, expert_begin, El, counts, offsets, row_to_pair, pair_to_row,
                                     x, H, x_perm, cap, scratch, (hipStream_t)stream),
                      "moe_permute_noalloc launch");
}

extern "C" size_t moe_ffn_workspace_size(int64_t cap_rows, int n_local_experts, int H, int I_s)
{
    if (cap_rows < 0 || n_local_experts < 1 || H <= 0 || I_s <= 0) return 0;
    return ffn_workspace_bytes(cap_rows, n_local_experts, H, I_s);
}

namespace {

// Checks shared by both grouped-FFN entry points (the routed experts' part).
moe_status check_ffn(const char *fn, const uint16_t *x, int64_t x_rows, const int32_t *row_to_pair, int k,
                     const int32_t *offsets, int n_local_experts, int64_t cap_rows, int H, int I_s,
                     const uint16_t *w13, const uint16_t *w2, const uint16_t *y)
{
    moe_status st;
    if (n_local_experts < 1) return fail(MOE_ERR_INVALID_ARG, "%s: n_local_experts=%d", fn, n_local_experts);
    if (n_local_experts > MOE_MAX_EXPERTS)
        return fail(MOE_ERR_UNSUPPORTED, "%s: n_local_experts=%d exceeds %d", fn, n_local_experts,
                    MOE_MAX_EXPERTS);
    if (cap_rows < 0) return fail(MOE_ERR_INVALID_ARG, "%s: cap_rows=%lld", fn, (long long)cap_rows);
    if (cap_rows >= ((int64_t)1 << 31)) return fail(MOE_ERR_UNSUPPORTED, "%s: cap_rows too large", fn);
    if (x_rows < 0) return fail(MOE_ERR_INVALID_ARG, "%s: x_rows=%lld", fn, (long long)x_rows);
    if ((st = check_width("H", H)) != MOE_OK) return st;
    if ((st = check_width("I_s", I_s)) != MOE_OK) return st;
    if (!offsets) return fail(MOE_ERR_INVALID_ARG, "%s: null offsets", fn);
    if (row_to_pair) {
        if (k < 1) return fail(MOE_ERR_INVALID_ARG, "%s: k=%d must be >= 1 with row_to_pair", fn, k);
    } else if (x_rows < cap_rows) {
        return fail(MOE_ERR_INVALID_ARG, "%s: x_rows=%lld < cap_rows=%lld for a permuted x", fn,
                    (long long)x_rows, (long long)cap_rows);
    }
    if (cap_rows > 0 && (!x || !w13 || !w2 || !y)) return fail(MOE_ERR_INVALID_ARG, "%s: null pointer", fn);
    if (!aligned16(x) || !aligned16(w13) || !aligned16(w2) || !aligned16(y))
        return fail(MOE_ERR_INVALID_ARG, "%s: tensors must be 16-byte aligned", fn);
    return MOE_OK;
}

moe_status check_workspace(const char *fn, const void *workspace, size_t workspace_bytes, size_t need)
{
    if (!workspace || workspace_bytes < need || (reinterpret_cast<uintptr_t>(workspace) & 255u))
        return fail(MOE_ERR_WORKSPACE, "%s: workspace %zu < %zu bytes or misaligned", fn, workspace_bytes, need);
    return MOE_OK;
}

}  // namespace

extern "C" moe_status moe_grouped_ffn(const uint16_t *x, int64_t x_rows, const int32_t *row_to_pair,
                                      int k, const int32_t *offsets, int n_local_experts,
                                      int64_t cap_rows, int H, int I_s, const uint16_t *w13,
                                      const uint16_t *w2, uint16_t *y, void *workspace,
                                      size_t workspace_bytes, void *stream)
{
    static const char fn[] = "moe_grouped_ffn";
    moe_status st = check_ffn(fn, x, x_rows, row_to_pair, k, offsets, n_local_experts, cap_rows, H, I_s, w13,
                              w2, y);
    if (st != MOE_OK) return st;
    const size_t need = moe_ffn_workspace_size(cap_rows, n_local_experts, H, I_s);
    if ((st = check_workspace(fn, workspace, workspace_bytes, need)) != MOE_OK) return st;
    return hip_status(launch_grouped_ffn(x, x_rows, row_to_pair, k, offsets, n_local_experts, cap_rows, H, I_s,
                                         w13, w2, y, 0, 0, nullptr, nullptr, nullptr, workspace,
                                         (hipStream_t)stream),
                      "moe_grouped_ffn launch");
}

extern "C" moe_status moe_grouped_ffn_shared(const uint16_t *x, int64_t x_rows, const int32_t *row_to_pair,
                                             int k, const int32_t *offsets, int n_local_experts,
                                             int64_t cap_rows, int H, int I_s, const uint16_t *w13,
                                             const uint16_t *w2, uint16_t *y, int64_t shared_begin,
                                             int64_t shared_count, const uint16_t *shared_w13,
                                             const uint16_t *shared_w2, uint16_t *shared_y, void *workspace,
                                             size_t workspace_bytes, void *stream)
{
    static const char fn[] = "moe_grouped_ffn_shared";
    moe_status st = check_ffn(fn, x, x_rows, row_to_pair, k, offsets, n_local_experts, cap_rows, H, I_s, w13,
                              w2, y);
    if (st != MOE_OK) return st;
    if (!row_to_pair) return fail(MOE_ERR_INVALID_ARG, "%s: row_to_pair is required", fn);
    if (shared_begin < 0 || shared_count < 0 || shared_begin + shared_count > x_rows)
        return fail(MOE_ERR_INVALID_ARG, "%s: shared rows [%lld, +%lld) outside the %lld rows of x", fn,
                    (long long)shared_begin, (long long)shared_count, (long long)x_rows);
    if (shared_count > 0) {
        if (!x || !shared_w13 || !shared_w2 || !shared_y) return fail(MOE_ERR_INVALID_ARG, "%s: null pointer", fn);
        if (!aligned16(x) || !aligned16(shared_w13) || !aligned16(shared_w2) || !aligned16(shared_y))
            return fail(MOE_ERR_INVALID_ARG, "%s: tensors must be 16-byte aligned", fn);
        if (n_local_experts + 1 > MOE_MAX_EXPERTS)
            return fail(MOE_ERR_UNSUPPORTED, "%s: n_local_experts + 1 exceeds %d", fn, MOE_MAX_EXPERTS);
        if (cap_rows + shared_count >= ((int64_t)1 << 31))
            return fail(MOE_ERR_UNSUPPORTED, "%s: cap_rows + shared_count too large", fn);
        if (!ffn_large_tiles(x_rows, cap_rows + shared_count, H, I_s))
            return fail(MOE_ERR_UNSUPPORTED,
                        "%s: H=%d and I_s=%d must be multiples of 64, from 128 to 2^26, with operands under 4 GiB",
                        fn, H, I_s);
    }
    const int ne = n_local_experts + (shared_count > 0 ? 1 : 0);
    const size_t need = moe_ffn_workspace_size(cap_rows + shared_count, ne, H, I_s);
    if ((st = check_workspace(fn, workspace, workspace_bytes, need)) != MOE_OK) return st;
    return hip_status(launch_grouped_ffn(x, x_rows, row_to_pair, k, offsets, n_local_experts, cap_rows, H, I_s,
                                         w13, w2, y, shared_begin, shared_count, shared_w13, shared_w2, shared_y,
                                         workspace, (hipStream_t)stream),
                      "moe_grouped_ffn_shared launch");
}

extern "C" size_t moe_layer_workspace_size(int64_t T, int k, int n_local_experts, int H, int I_s,
                                           int64_t shared_count)
{
    if (T < 0 || k < 1 || n_local_experts < 1 || H <= 0 || I_s <= 0 || shared_count < 0) return 0;
    const int64_t cap = T * (k < n_local_experts ? k : n_local_experts);
    const size_t perm = align256(moe_permute_workspace_size(T, k, n_local_experts));
    return perm + moe_ffn_workspace_size(cap + shared_count, n_local_experts + (shared_count > 0 ? 1 : 0), H, I_s);
}

extern "C" moe_status moe_layer_forward(const uint16_t *x, const float *logits, int64_t T, int E, int k,
                                        int expert_begin, int n_local_experts, int H, int I_s, const uint16_t *w13,
                                        const uint16_t *w2, int64_t shared_begin, int64_t shared_count,
                                        const uint16_t *shared_w13, const uint16_t *shared_w2, int32_t *topk_ids,
                                        float *topk_w, int32_t *counts, int32_t *offsets, int32_t *row_to_pair,
                                        int32_t *pair_to_row, uint16_t *y, uint16_t *shared_y, uint16_t *out,
                                        void *workspace, size_t workspace_bytes, void *stream)
{
    static const char fn[] = "moe_layer_forward";
    // what moe_route, moe_permute, moe_grouped_ffn_shared and moe_combine check
    moe_status st = check_topk(T, E, k);
    if (st != MOE_OK) return st;
    const int El = n_local_experts;
    if (El < 1 || expert_begin < 0 || expert_begin + El > E)
        return fail(MOE_ERR_INVALID_ARG, "%s: local experts [%d, %d+%d) not inside [0, E=%d)", fn, expert_begin,
                    expert_begin, El, E);
    const int64_t cap = T * (k < El ? k : El);
    if ((st = check_ffn(fn, x, T, row_to_pair, k, offsets, El, cap, H, I_s, w13, w2, y)) != MOE_OK) return st;
    if (!counts) return fail(MOE_ERR_INVALID_ARG, "%s: null counts", fn);
    if (T > 0 && (!logits || !topk_ids || !topk_w || !row_to_pair || !pair_to_row || !out))
        return fail(MOE_ERR_INVALID_ARG, "%s: null pointer", fn);
    if (!aligned16(out)) return fail(MOE_ERR_INVALID_ARG, "%s: out must be 16-byte aligned", fn);
    if (shared_begin < 0 || shared_count < 0 || shared_begin + shared_count > T)
        return fail(MOE_ERR_INVALID_ARG, "%s: shared rows [%lld, +%lld) outside the %lld tokens", fn,
                    (long long)shared_begin, (long long)shared_count, (long long)T);
    if (shared_count > 0) {
        if (!shared_w13 || !shared_w2 || !shared_y) return fail(MOE_ERR_INVALID_ARG, "%s: null pointer", fn);
        if (!aligned16(shared_w13) || !aligned16(shared_w2) || !aligned16(shared_y))
            return fail(MOE_ERR_INVALID_ARG, "%s: tensors must be 16-byte aligned", fn);
        if (El + 1 > MOE_MAX_EXPERTS)
            return fail(MOE_ERR_UNSUPPORTED, "%s: n_local_experts + 1 exceeds %d", fn, MOE_MAX_EXPERTS);
        if (cap + shared_count >= ((int64_t)1 << 31))
            return fail(MOE_ERR_UNSUPPORTED, "%s: cap_rows + shared_count too large", fn);
        if (!ffn_large_tiles(T, cap + shared_count, H, I_s))
            return fail(MOE_ERR_UNSUPPORTED,
                        "%s: H=%d and I_s=%d must be multiples of 64, from 128 to 2^26, with operands under 4 GiB",
                        fn, H, I_s);
    }
    const size_t need = moe_layer_workspace_size(T, k, El, H, I_s, shared_count);
    if ((st = check_workspace(fn, workspace, workspace_bytes, need)) != MOE_OK) return st;
    char *ws = static_cast<char *>(workspace);
    void *ws_ffn = ws + align256(moe_permute_workspace_size(T, k, El));
    return hip_status(launch_layer(x, logits, T, E, k, expert_begin, El, H, I_s, w13, w2, shared_begin, shared_count,
                                   shared_w13, shared_w2, topk_ids, topk_w, counts, offsets, row_to_pair,
                                   pair_to_row, y, shared_y, out, reinterpret_cast<int32_t *>(ws), ws_ffn,
                                   (hipStream_t)stream),
                      "moe_layer_forward launch");
}

extern "C" moe_status moe_reshard_experts(int direction, int P, int rank, int E, int H, int I,
                                          const uint16_t *const *src_w13, const uint16_t *const *src_w2,
                                          uint16_t *dst_w13, uint16_t *dst_w2, void *stream)
{
    static const char fn[] = "moe_reshard_experts";
    moe_status st;
    if (direction != MOE_EP_TO_TP && direction != MOE_TP_TO_EP)
        return fail(MOE_ERR_INVALID_ARG, "%s: direction=%d", fn, direction);
    if (P < 1) return fail(MOE_ERR_INVALID_ARG, "%s: P=%d", fn, P);
    if (P > MOE_MAX_RESHARD_RANKS) return fail(MOE_ERR_UNSUPPORTED, "%s: P=%d exceeds %d", fn, P, MOE_MAX_RESHARD_RANKS);
    if (rank < 0 || rank >= P) return fail(MOE_ERR_INVALID_ARG, "%s: rank=%d not in [0, %d)", fn, rank, P);
    if (E < P || E % P) return fail(MOE_ERR_INVALID_ARG, "%s: E=%d is not a positive multiple of P=%d", fn, E, P);
    if (I < P || I % P) return fail(MOE_ERR_INVALID_ARG, "%s: I=%d is not a positive multiple of P=%d", fn, I, P);
    if ((st = check_width("H", H)) != MOE_OK) return st;
    if ((I / P) % 8) return fail(MOE_ERR_UNSUPPORTED, "%s: I/P=%d is not a multiple of 8", fn, I / P);
    if (!src_w13 || !src_w2) return fail(MOE_ERR_INVALID_ARG, "%s: null source arrays", fn);
    if (!dst_w13 || !dst_w2) return fail(MOE_ERR_INVALID_ARG, "%s: null destination", fn);
    if (!aligned16(dst_w13) || !aligned16(dst_w2))
        return fail(MOE_ERR_INVALID_ARG, "%s: destination not 16-byte aligned", fn);
    for (int q = 0; q < P; ++q) {
        if (!src_w13[q] != !src_w2[q])
            return fail(MOE_ERR_INVALID_ARG, "%s: source %d has only one of w13, w2", fn, q);
        if (!aligned16(src_w13[q]) || !aligned16(src_w2[q]))
            return fail(MOE_ERR_INVALID_ARG, "%s: source %d not 16-byte aligned", fn, q);
    }
    return hip_status(launch_reshard(direction, P, rank, E, H, I, src_w13, src_w2, dst_w13, dst_w2,
                                     (hipStream_t)stream),
                      "moe_reshard_experts launch");
}

extern "C" moe_status moe_kv_slots(const int32_t *page_table, int64_t pt_stride, const int32_t *first, int n_req,
                                   int page_size, int32_t *slots, int64_t capacity, void *stream)
{
    static const char fn[] = "moe_kv_slots";
    if (n_req < 0 || capacity < 0 || pt_stride < 0)
        return fail(MOE_ERR_INVALID_ARG, "%s: negative n_req, capacity or pt_stride", fn);
    if (page_size < 1) return fail(MOE_ERR_INVALID_ARG, "%s: page_size=%d", fn, page_size);
    if (n_req == 0 || capacity == 0) return MOE_OK;
    if (!page_table || !first || !slots) return fail(MOE_ERR_INVALID_ARG, "%s: null pointer", fn);
    return hip_status(launch_kv_slots(page_table, pt_stride, first, n_req, page_size, capacity, slots,
                                      (hipStream_t)stream),
                      "moe_kv_slots launch");
}

extern "C" moe_status moe_kv_move(int n_src, const uint16_t *const *src_k, const uint16_t *const *src_v,
                                  const int64_t *src_slots, const int64_t *src_first, int src_heads, uint16_t *dst_k,
                                  uint16_t *dst_v, int64_t dst_slots, int dst_heads, int head_dim, int src_head0,
                                  int dst_head0, int n_heads, const int32_t *src_slot, const int32_t *dst_slot,
                                  void *stream)
{
    static const char fn[] = "moe_kv_move";
    moe_status st;
    if (n_src < 1) return fail(MOE_ERR_INVALID_ARG, "%s: n_src=%d", fn, n_src);
    if (n_src > MOE_MAX_KV_SOURCES)
        return fail(MOE_ERR_UNSUPPORTED, "%s: n_src=%d exceeds %d", fn, n_src, MOE_MAX_KV_SOURCES);
    if (!src_k || !src_slots || !src_first) return fail(MOE_ERR_INVALID_ARG, "%s: null source arrays", fn);
    if (dst_slots < 0) return fail(MOE_ERR_INVALID_ARG, "%s: negative dst_slots", fn);
    if ((st = check_width("head_dim", head_dim)) != MOE_OK) return st;
    if (n_heads < 1 || src_heads < 1 || dst_heads < 1 || src_head0 < 0 || dst_head0 < 0 ||
        src_head0 + n_heads > src_heads || dst_head0 + n_heads > dst_heads)
        return fail(MOE_ERR_INVALID_ARG, "%s: head ranges [%d, +%d) / [%d, +%d) outside %d / %d heads", fn,
                    src_head0, n_heads, dst_head0, n_heads, src_heads, dst_heads);
    if (!src_v != !dst_v) return fail(MOE_ERR_INVALID_ARG, "%s: give both V sides or neither", fn);
    if (src_first[0] != 0) return fail(MOE_ERR_INVALID_ARG, "%s: src_first[0] must be 0", fn);
    for (int q = 0; q < n_src; ++q) {
        if (src_first[q + 1] < src_first[q])
            return fail(MOE_ERR_INVALID_ARG, "%s: src_first must not decrease", fn);
        if (src_slots[q] < 0) return fail(MOE_ERR_INVALID_ARG, "%s: negative src_slots[%d]", fn, q);
        if (src_first[q + 1] > src_first[q]) {
            if (!src_k[q] || (src_v && !src_v[q])) return fail(MOE_ERR_INVALID_ARG, "%s: null source pool %d", fn, q);
            if (!aligned16(src_k[q]) || (src_v && !aligned16(src_v[q])))
                return fail(MOE_ERR_INVALID_ARG, "%s: source pool %d not 16-byte aligned", fn, q);
        }
    }
    if (src_first[n_src] == 0) return MOE_OK;
    if (!dst_k || !src_slot || !dst_slot) return fail(MOE_ERR_INVALID_ARG, "%s: null pointer", fn);
    if (!aligned16(dst_k) || !aligned16(dst_v))
        return fail(MOE_ERR_INVALID_ARG, "%s: destination pools must be 16-byte aligned", fn);
    return hip_status(launch_kv_move(n_src, src_k, src_v, src_slots, src_first, src_heads, dst_k, dst_v, dst_slots,
                                     dst_heads, head_dim, src_head0, dst_head0, n_heads, src_slot, dst_slot,
                                     (hipStream_t)stream),
                      "moe_kv_move launch");
}

extern "C" moe_status moe_combine(const uint16_t *y, int64_t y_rows, const int32_t *pair_to_row,
                                  const float *topk_w, int64_t T, int k, int H,
                                  const uint16_t *shared_y, int64_t shared_begin,
                                  int64_t shared_count, int accumulate, uint16_t *out, void *stream)
{
    moe_status st;
    if (T < 0 || y_rows < 0) return fail(MOE_ERR_INVALID_ARG, "negative T or y_rows");
    if (k < 1) return fail(MOE_ERR_INVALID_ARG, "k=%d must be >= 1", k);
    if (k > MOE_MAX_TOPK) return fail(MOE_ERR_UNSUPPORTED, "k=%d exceeds %d", k, MOE_MAX_TOPK);
    if (T * (int64_t)k >= ((int64_t)1 << 31)) return fail(MOE_ERR_UNSUPPORTED, "T*k too large");
    if ((st = check_width("H", H)) != MOE_OK) return st;
    if (T > 0 && (!pair_to_row || !topk_w || !out))
        return fail(MOE_ERR_INVALID_ARG, "moe_combine: null pointer");
    if (y_rows > 0 && !y) return fail(MOE_ERR_INVALID_ARG, "moe_combine: null y with y_rows > 0");
    if (shared_y) {
        if (shared_begin < 0 || shared_count < 0 || shared_begin + shared_count > T)
            return fail(MOE_ERR_INVALID_ARG, "shared rows [%lld, +%lld) outside [0, T)",
                        (long long)shared_begin, (long long)shared_count);
    }
    if (!aligned16(y) || !aligned16(out) || !aligned16(shared_y))
        return fail(MOE_ERR_INVALID_ARG, "moe_combine: tensors must be 16-byte aligned");
    return hip_status(launch_combine(y, y_rows, pair_to_row, topk_w, T, k, H, shared_y,
                                     shared_begin, shared_y ? shared_count : 0, accumulate ? 1 : 0,
                                     out, (hipStream_t)stream),
                      "moe_combine launch");
}
