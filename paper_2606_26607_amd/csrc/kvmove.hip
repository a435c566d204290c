// Paged KV-cache head moves for a layout switch (Sec. 3.2): under EP a rank
// holds every KV head of its own requests, under TP its head shard of every
// request, and a switch moves head slices of every live token between the
// two pools through the page tables.
//
// A pool of one layer is [slots, heads, head_dim] bf16 (a paged pool
// [pages, page_size, heads, head_dim] is the same memory, slot = page *
// page_size + offset).  The page-indexed work descriptors (Sec. 4.3) are one
// slot index per token (kv_slots expands page tables into them); kv_move
// copies, per token, the n_heads * head_dim contiguous elements of a head
// range, for K and V, from up to 16 source pools in one launch.
#include "moe_internal.h"

namespace moe {
namespace {

// slots[first[q] + t] = page_table[q * stride + t / page_size] * page_size +
// t % page_size for the tokens t of request q (first[] is the exclusive
// prefix of the requests' lengths).
// Tokens beyond `capacity`, and tokens whose page lies past the request's
// `stride` page-table entries, are not written / get slot -1 (which kv_move
// skips).
__global__ __launch_bounds__(256) void kv_slots_kernel(const int32_t *__restrict__ page_table, int64_t stride,
                                                       const int32_t *__restrict__ first, int n_req,
                                                       int page_size, int64_t capacity,
                                                       int32_t *__restrict__ slots)
{
    int64_t n = first[n_req];
    if (n > capacity) n = capacity;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        int lo = 0, hi = n_req - 1;  // the request holding token i
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (first[mid] <= i) lo = mid; else hi = mid - 1;
        }
        const int64_t t = i - first[lo];
        const int64_t pg = t / page_size;
        slots[i] = (t < 0 || pg >= stride)
                       ? -1
                       : page_table[(int64_t)lo * stride + pg] * page_size + (int32_t)(t % page_size);
    }
}

// The source pools of one move: tokens [first[q], first[q+1]) come from
// pool q.
struct KvSources {
    const uint16_t *k[MOE_MAX_KV_SOURCES];
    const uint16_t *v[MOE_MAX_KV_SOURCES];
    int64_t slots[MOE_MAX_KV_SOURCES];
    int64_t first[MOE_MAX_KV_SOURCES + 1];
    int n;
};

// Each thread owns one 16-byte chunk position c of a token's head run and
// walks the tokens with a stride of (threads / chunks), so the index maths is
// done once; K and V of a token are loaded before either is stored.  Tokens
// whose source or destination slot lies outside its pool are skipped.
__global__ __launch_bounds__(256) void kv_move_kernel(KvSources src, int s_heads, uint16_t *__restrict__ dk,
                                                      uint16_t *__restrict__ dv, int64_t d_slots, int d_heads,
                                                      int head_dim, int hs0, int hd0, int nh,
                                                      const int32_t *__restrict__ src_slot,
                                                      const int32_t *__restrict__ dst_slot, bool with_v)
{
    typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
    const int64_t n_tokens = src.first[src.n];
    const unsigned chunks = (unsigned)(nh * head_dim / 8);  // per token and tensor
    const unsigned threads = gridDim.x * blockDim.x;
    const unsigned step = threads / chunks;                  // tokens per sweep (>= 1, set by the launch)
    const unsigned g = blockIdx.x * blockDim.x + threadIdx.x;
    if (g >= step * chunks) return;
    const unsigned c = g % chunks;
    int q = 0;
    for (int64_t i = g / chunks; i < n_tokens; i += step) {
        while (q + 1 < src.n && src.first[q + 1] <= i) ++q;  // i only grows
        const int64_t s = src_slot[i], d = dst_slot[i];
        if (s < 0 || s >= src.slots[q] || d < 0 || d >= d_slots) continue;
        const int64_t so = (s * s_heads + hs0) * head_dim + c * 8, dof = (d * d_heads + hd0) * head_dim + c * 8;
        const u32x4_t kx = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(src.k[q] + so));
        if (with_v) {
            const u32x4_t vx = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(src.v[q] + so));
            __builtin_nontemporal_store(kx, reinterpret_cast<u32x4_t *>(dk + dof));
            __builtin_nontemporal_store(vx, reinterpret_cast<u32x4_t *>(dv + dof));
        } else {
            __builtin_nontemporal_store(kx, reinterpret_cast<u32x4_t *>(dk + dof));
        }
    }
}

// Blocks of 256 threads resident at once: 8 per compute unit.
int64_t resident_blocks()
{
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
        cus = 256;
    return 8 * (int64_t)cus;
}

int64_t grid_for(int64_t items)
{
    const int64_t b = ceil_div(items, 256);
    return b < 1 ? 1 : (b > 16384 ? 16384 : b);
}

}  // namespace

hipError_t launch_kv_slots(const int32_t *page_table, int64_t stride, const int32_t *first, int n_req,
                           int page_size, int64_t max_tokens, int32_t *slots, hipStream_t s)
{
    KernelTimer timer(MOE_K_KV_MOVE, s);
    kv_slots_kernel<<<dim3((unsigned)grid_for(max_tokens)), dim3(256), 0, s>>>(page_table, stride, first, n_req,
                                                                              page_size, max_tokens, slots);
    return hipGetLastError();
}

hipError_t launch_kv_move(int n_src, const uint16_t *const *sk, const uint16_t *const *sv, const int64_t *s_slots,
                          const int64_t *first, int s_heads, uint16_t *dk, uint16_t *dv, int64_t d_slots, int d_heads,
                          int head_dim, int hs0, int hd0, int nh, const int32_t *src_slot, const int32_t *dst_slot,
                          hipStream_t s)
{
    KvSources src{};
    src.n = n_src;
    for (int q = 0; q < n_src; ++q) {
        src.k[q] = sk[q];
        src.v[q] = sv ? sv[q] : nullptr;
        src.slots[q] = s_slots[q];
        src.first[q] = first[q];
    }
    src.first[n_src] = first[n_src];
    const int64_t n_tokens = first[n_src];
    if (n_tokens == 0) return hipSuccess;
    const bool with_v = sv != nullptr;
    // one thread per chunk of every token, at most one resident round (8
    // blocks of 256 per CU): a sweep then covers consecutive tokens, whose
    // pages are few, rather than the whole pool at once (measured 1.14x
    // faster than 8x as many blocks on a 250 MB move); at least enough
    // threads for one token's chunks
    const int64_t chunks = (int64_t)nh * head_dim / 8;
    int64_t blocks = ceil_div(n_tokens * chunks, 256);
    if (blocks > resident_blocks()) blocks = resident_blocks();
    if (blocks * 256 < chunks) blocks = ceil_div(chunks, 256);
    KernelTimer timer(MOE_K_KV_MOVE, s);
    kv_move_kernel<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(src, s_heads, dk, dv, d_slots, d_heads, head_dim,
                                                                hs0, hd0, nh, src_slot, dst_slot, with_v);
    return hipGetLastError();
}

}  // namespace moe
