/*
 * libmoe: the Mixture-of-Experts layer forward on one GPU's share of the
 * work, for AMD Instinct MI355X (gfx950).
 *
 * The paper (Sec. 2.1 and Sec. 3.1) runs the expert layer in two layouts:
 *
 *  - tensor parallel (TP): every rank holds one I/P slice of every expert,
 *    W13 (E, 2I/P, H) and W2 (E, H, I/P); all tokens are present and the
 *    rank's output is a partial sum that an all-reduce completes;
 *  - expert parallel (EP): a rank holds E/P whole experts, W13 (E/P, 2I, H)
 *    and W2 (E/P, H, I), and computes only the (token, expert) pairs routed
 *    to them; a combine all-to-all completes the output.
 *
 * W13 stacks the gate projection (rows [0, I_s)) before the up projection
 * (rows [I_s, 2*I_s)) of a SwiGLU MLP; I_s is the rank's intermediate width
 * (I under EP, I/P under TP).  Both layouts compute the same function of the
 * same weights (Sec. 1, Sec. 3), so one library serves both: a TP slice is
 * expert_begin = 0, n_local_experts = E, I_s = I/P; an EP slice is
 * expert_begin = r*E/P, n_local_experts = E/P, I_s = I.
 *
 * The forward is four calls on one stream:
 *   moe_route -> moe_permute -> moe_grouped_ffn -> moe_combine
 * or the same in one call, moe_layer_forward, with fewer launches.
 *
 * Conventions for every call:
 *  - Array arguments are DEVICE pointers owned by the caller, row-major and
 *    contiguous.  bf16 tensors are passed as uint16_t bit patterns.
 *  - The library never allocates, frees or synchronises; scratch memory is
 *    the caller's `workspace` (sizes from the *_workspace_size queries).
 *    Work is enqueued on `stream` (a hipStream_t; NULL = default stream) and
 *    results are valid once that stream has been synchronised.  No call
 *    reads device data back to the host, so the chain can be captured in a
 *    HIP graph.
 *  - Arguments are validated on the host before anything is enqueued; a
 *    rejected call returns MOE_ERR_INVALID_ARG, MOE_ERR_UNSUPPORTED or
 *    MOE_ERR_WORKSPACE, enqueues nothing and leaves every buffer untouched.
 *    Checks of sizes, pointers and limits make no HIP call.  Two lookups do:
 *    the grouped-FFN workspace size depends on the current device's compute
 *    unit count (moe_ffn_workspace_size, and the workspace check of
 *    moe_grouped_ffn / moe_grouped_ffn_shared, query it), and the first
 *    moe_permute_noalloc call on a device looks up its scratch address.
 *    A failed kernel launch returns MOE_ERR_HIP.  moe_last_error() gives a
 *    message for the last non-OK status on the calling thread.
 *  - Sizes: 1 <= E <= 1024, 1 <= k <= min(E, 16), T >= 0, T*k < 2^31,
 *    H and I_s positive multiples of 8.
 */
#ifndef LIBMOE_H
#define LIBMOE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum moe_status {
    MOE_OK = 0,
    MOE_ERR_INVALID_ARG = 1, /* null pointer, negative or inconsistent size */
    MOE_ERR_UNSUPPORTED = 2, /* outside the documented limits */
    MOE_ERR_WORKSPACE = 3,   /* workspace missing or smaller than required */
    MOE_ERR_HIP = 4          /* a HIP runtime call or kernel launch failed */
} moe_status;

#define MOE_MAX_TOPK 16
#define MOE_MAX_EXPERTS 1024
#define MOE_MAX_RESHARD_RANKS 16
#define MOE_MAX_KV_SOURCES 16

/* Static name of a status code ("MOE_OK", ...). */
const char *moe_status_str(int status);

/* Message for the last non-OK status returned on the calling thread. */
const char *moe_last_error(void);

/* Library interface version (incremented on any ABI change). */
int moe_version(void);

/*
 * Gating.  The paper names sparse per-token expert selection (Sec. 1) but
 * not the gating function; libmoe uses softmax top-k renormalised over the
 * kept experts.  For each token t:
 *   - topk_ids[t, 0..k-1]: the k experts with the largest logits, largest
 *     first; equal logits order by ascending expert id, and -0.0 equals +0.0;
 *   - topk_w[t, j] = exp(l_j - l_0) / sum_{i<k} exp(l_i - l_0), the softmax
 *     over all E logits renormalised over the kept k (weights sum to 1).
 * logits   [T, E] fp32, finite (NaN/Inf give unspecified ids and weights)
 * topk_ids [T, k] int32 out;  topk_w [T, k] fp32 out.
 */
moe_status moe_route(const float *logits, int64_t T, int E, int k, int32_t *topk_ids,
                     float *topk_w, void *stream);

/*
 * Permutation (token sort by expert).  Pair p = t*k + j is local when
 * expert_begin <= topk_ids[t, j] < expert_begin + n_local_experts (an EP
 * rank sees only the pairs routed to its experts, Sec. 2.1; a TP rank owns
 * every expert).  Local pairs are ordered by local expert, then by
 * ascending token; this order is unique, so every output is deterministic.
 *   counts      [El]        int32 out: pairs per local expert
 *   offsets     [El + 1]    int32 out: exclusive prefix sum of counts;
 *                           offsets[El] = n, the number of local pairs
 *   row_to_pair [T*min(k,El)] int32 out: rows [0, n) hold the pair index
 *   pair_to_row [T*k]       int32 out: the pair's row, or -1 if not local
 *   x [T, H] bf16 and x_perm [T*min(k,El), H] bf16: when x_perm is not
 *   NULL, row r of x_perm is set to x[row_to_pair[r] / k] for r < n (x may
 *   be NULL when x_perm is NULL).
 * Rows at and beyond n of row_to_pair / x_perm are left untouched.
 * workspace: at least moe_permute_workspace_size(T, k, n_local_experts)
 * bytes, 256-byte aligned.
 */
size_t moe_permute_workspace_size(int64_t T, int k, int n_local_experts);
moe_status moe_permute(const int32_t *topk_ids, int64_t T, int k, int E, int expert_begin,
                       int n_local_experts, int32_t *counts, int32_t *offsets,
                       int32_t *row_to_pair, int32_t *pair_to_row, const uint16_t *x, int H,
                       uint16_t *x_perm, void *workspace, size_t workspace_bytes, void *stream);

/*
 * The permutation without a caller workspace, for callers that cannot
 * allocate device memory: code under HIP graph capture that must not call
 * hipMalloc, tight serving loops, harnesses that forbid allocation.  Same
 * arguments, outputs and errors as moe_permute, minus the workspace: the
 * per-chunk histograms live in a static array of MOE_PERMUTE_SCRATCH_BYTES
 * in the library, one copy per GPU held until the process ends (its address
 * is looked up on the first call on each device).  It allocates nothing and
 * calls no allocating routine.  Calls whose moe_permute_workspace_size(T, k,
 * n_local_experts) exceeds MOE_PERMUTE_SCRATCH_BYTES return
 * MOE_ERR_UNSUPPORTED and enqueue nothing (for 256-pair chunks, T*k*E_l up to
 * 2^24, the need is at most 256 KiB; for larger inputs it is about
 * T*k*E_l/256 bytes).  The scratch of the CURRENT device is used: `stream`
 * must belong to it.  Every call on one GPU shares that GPU's array, so calls
 * that overlap on one GPU (other streams, other threads, other graphs
 * replayed concurrently) race; calls in stream order do not.  Nothing in the
 * array needs to start at zero (each call writes every entry it reads).
 */
#define MOE_PERMUTE_SCRATCH_BYTES (4u << 20)
moe_status moe_permute_noalloc(const int32_t *topk_ids, int64_t T, int k, int E, int expert_begin,
                               int n_local_experts, int32_t *counts, int32_t *offsets, int32_t *row_to_pair,
                               int32_t *pair_to_row, const uint16_t *x, int H, uint16_t *x_perm, void *stream);

/*
 * Grouped SwiGLU expert FFN (Sec. 3.1 weight shapes).  For every local
 * expert e and every row r in [offsets[e], offsets[e+1]), with input row
 *   in_r = x[row_to_pair[r] / k]   when row_to_pair is not NULL (x is the
 *          token matrix [x_rows, H]: the permutation's row gather is done by
 *          the GEMM's operand loads, so no permuted copy is materialised), or
 *   in_r = x[r]                    when row_to_pair is NULL (x is an already
 *          permuted buffer such as moe_permute's x_perm, x_rows >= cap_rows):
 *   g = in_r . W13[e, 0:I_s]^T,   u = in_r . W13[e, I_s:2*I_s]^T
 *   h = silu(g) * u  (fp32, then rounded to bf16)
 *   y[r] = h . W2[e]^T  (fp32 accumulation, rounded to bf16)
 *   offsets [El + 1] int32 (as moe_permute writes them; rows beyond cap_rows
 *   are never touched even if offsets claim them);  row_to_pair [cap_rows]
 *   int32 (entries must lie in [0, x_rows*k));  w13 [El, 2*I_s, H] bf16;
 *   w2 [El, H, I_s] bf16;  y [cap_rows, H] bf16 out (rows >= offsets[El]
 *   untouched).
 * Experts with no rows read none of their weights.
 * workspace: at least moe_ffn_workspace_size(cap_rows, El, H, I_s) bytes,
 * 256-byte aligned (holds the bf16 intermediate h, the tile schedule and the
 * split-K partials; its size depends on the current device's compute unit
 * count, which the query reads with hipGetDevice / hipDeviceGetAttribute).
 */
size_t moe_ffn_workspace_size(int64_t cap_rows, int n_local_experts, int H, int I_s);
moe_status moe_grouped_ffn(const uint16_t *x, int64_t x_rows, const int32_t *row_to_pair, int k,
                           const int32_t *offsets, int n_local_experts, int64_t cap_rows, int H,
                           int I_s, const uint16_t *w13, const uint16_t *w2, uint16_t *y,
                           void *workspace, size_t workspace_bytes, void *stream);

/*
 * Grouped FFN with a shared expert in the same launches (the shared-expert
 * models of Sec. 8: a dense expert every token of the rank's data-parallel
 * share goes through, beside the routed ones).  Computes exactly what
 * moe_grouped_ffn computes for the routed experts (row_to_pair is required
 * here) and, in the same kernels, the SwiGLU FFN of the shared expert on
 * token rows [shared_begin, shared_begin + shared_count) of x:
 *   shared_y[i] = FFN(x[shared_begin + i]; shared_w13, shared_w2)
 *   shared_w13 [2*I_s, H] bf16 (gate rows, then up rows), shared_w2 [H, I_s]
 *   bf16, shared_y [shared_count, H] bf16 out.
 * The shared expert has the routed experts' intermediate width I_s.  One
 * launch per GEMM streams the routed and the shared weights together, which
 * matters in decode, where both are read from HBM once per step.
 * Limits: with shared_count > 0, H and I_s are multiples of 64 and at least
 * 128, n_local_experts + 1 <= 1024 and cap_rows + shared_count < 2^31
 * (MOE_ERR_UNSUPPORTED otherwise); shared_begin + shared_count <= x_rows.
 * workspace: at least moe_ffn_workspace_size(cap_rows + shared_count,
 * n_local_experts + (shared_count > 0), H, I_s) bytes, 256-byte aligned.
 */
moe_status moe_grouped_ffn_shared(const uint16_t *x, int64_t x_rows, const int32_t *row_to_pair, int k,
                                  const int32_t *offsets, int n_local_experts, int64_t cap_rows, int H,
                                  int I_s, const uint16_t *w13, const uint16_t *w2, uint16_t *y,
                                  int64_t shared_begin, int64_t shared_count, const uint16_t *shared_w13,
                                  const uint16_t *shared_w2, uint16_t *shared_y, void *workspace,
                                  size_t workspace_bytes, void *stream);

/*
 * Combine (unpermute and gate-weighted reduce).  For every token t:
 *   out[t] = (accumulate ? out[t] : 0)
 *          + (shared_begin <= t < shared_begin + shared_count ? shared_y[t - shared_begin] : 0)
 *          + sum_{j=0..k-1, pair_to_row[t*k+j] >= 0} topk_w[t, j] * y[pair_to_row[t*k+j]]
 * accumulated in fp32 in that order and rounded once to bf16.  The result
 * is the rank's partial output: the TP partial sum before the all-reduce,
 * or the EP partial before the combine all-to-all (Sec. 1); a token with no
 * local pair gets 0 (or its prior value).  The optional shared term carries
 * a shared expert's output for the rank's own data-parallel token share.
 *   y [y_rows, H] bf16;  pair_to_row [T*k] int32 (rows >= y_rows are
 *   skipped);  topk_w [T, k] fp32;  shared_y [shared_count, H] bf16 or
 *   NULL;  out [T, H] bf16 in/out.
 */
moe_status moe_combine(const uint16_t *y, int64_t y_rows, const int32_t *pair_to_row,
                       const float *topk_w, int64_t T, int k, int H, const uint16_t *shared_y,
                       int64_t shared_begin, int64_t shared_count, int accumulate,
                       uint16_t *out, void *stream);

/*
 * The whole layer forward in one call: exactly
 *   moe_route(logits) -> moe_permute (no x_perm) -> moe_grouped_ffn_shared
 *   (or moe_grouped_ffn without a shared expert; the row gather fused) ->
 *   moe_combine (accumulate = 0, the shared rows added)
 * with every intermediate written to the caller's buffers, bit for bit what
 * those four calls write.  Where the shapes allow it (at most 64 local
 * experts, the large-tile FFN shapes: H and I_s multiples of 64, at least
 * 128), routing, the permutation and the FFN's tile schedule run in fused
 * launches: for small inputs (pairs x (bits of the local expert index + 2)
 * at most 16384, e.g. 2048 pairs over 32 experts) routing, then the
 * permutation with the schedule in one workgroup; for larger ones routing
 * with the permutation's histogram, then its scan and scatter with the
 * schedule: two launches instead of three or four.  Otherwise it runs the
 * four calls' launches.
 *   x [T, H] bf16; logits [T, E] fp32; w13, w2 and shared_w13 [2*I_s, H],
 *   shared_w2 [H, I_s] as for moe_grouped_ffn(_shared) (the shared expert,
 *   on token rows [shared_begin, shared_begin + shared_count), has the
 *   routed experts' width; shared_count = 0 for none);
 *   outputs: topk_ids, topk_w [T, k]; counts [El]; offsets [El+1];
 *   row_to_pair [T*min(k,El)]; pair_to_row [T*k]; y [T*min(k,El), H];
 *   shared_y [shared_count, H]; out [T, H] bf16.
 * workspace: at least moe_layer_workspace_size(T, k, El, H, I_s,
 * shared_count) bytes, 256-byte aligned.  Errors as for the four calls.
 */
size_t moe_layer_workspace_size(int64_t T, int k, int n_local_experts, int H, int I_s, int64_t shared_count);
moe_status moe_layer_forward(const uint16_t *x, const float *logits, int64_t T, int E, int k, int expert_begin,
                             int n_local_experts, int H, int I_s, const uint16_t *w13, const uint16_t *w2,
                             int64_t shared_begin, int64_t shared_count, const uint16_t *shared_w13,
                             const uint16_t *shared_w2, int32_t *topk_ids, float *topk_w, int32_t *counts,
                             int32_t *offsets, int32_t *row_to_pair, int32_t *pair_to_row, uint16_t *y,
                             uint16_t *shared_y, uint16_t *out, void *workspace, size_t workspace_bytes,
                             void *stream);

/*
 * Expert-weight resharding between the EP and TP views (Sec. 3.1; the
 * layout switch of Sec. 4.2-4.3), for one destination rank.  With E experts,
 * P ranks, hidden size H and expert intermediate size I:
 *   EP view of rank q: w13 [E/P, 2I, H] (gate rows [0, I), up rows [I, 2I) of
 *     experts q*E/P ..), w2 [E/P, H, I];
 *   TP view of rank r: w13 [E, 2I/P, H] (for every expert, gate rows
 *     [r*I/P, (r+1)*I/P) then the matching up rows), w2 [E, H, I/P].
 * MOE_EP_TO_TP writes rank `rank`'s TP view from EP views; MOE_TP_TO_EP
 * writes its EP view from TP views.  src_w13 / src_w2 are HOST arrays of P
 * device pointers, the views of ranks 0..P-1 (read during the call only);
 * an entry pair left NULL is skipped, and the part of the destination it
 * would supply is left untouched.  Passing only src[rank] copies the 1/P
 * that stays on the GPU in a switch; passing all P (e.g. peers' buffers
 * mapped into this process) writes the whole destination.  Every element is
 * copied once, bit-exact.  The destination must not overlap a given source
 * (the caller's slot scheme guarantees that: one spare slot per rank, EP
 * layer i in slot i+1, TP layer i in slot i, EP->TP walking layers upward
 * and TP->EP downward).
 * Limits: 1 <= P <= MOE_MAX_RESHARD_RANKS, E and I multiples of P, H and
 * I/P multiples of 8, 16-byte aligned tensors.
 */
typedef enum moe_reshard_dir { MOE_EP_TO_TP = 0, MOE_TP_TO_EP = 1 } moe_reshard_dir;
moe_status moe_reshard_experts(int direction, int P, int rank, int E, int H, int I,
                               const uint16_t *const *src_w13, const uint16_t *const *src_w2,
                               uint16_t *dst_w13, uint16_t *dst_w2, void *stream);

/*
 * Paged KV-cache head moves for a layout switch (Sec. 3.2), driven by
 * page-indexed work descriptors (Sec. 4.3).  Under EP a rank
 * holds every KV head of its own requests; under TP it holds its head shard
 * of every request (a head shared by several ranks when there are fewer KV
 * heads than ranks).  A pool of one layer is [slots, heads, head_dim] bf16
 * (a paged pool [pages, page_size, heads, head_dim] is the same memory, slot
 * = page * page_size + offset); its tokens are found through page tables.
 *
 * moe_kv_slots: one slot per token of n_req requests, in request order:
 *   slots[first[q] + t] = page_table[q * pt_stride + t / page_size] *
 *   page_size + t % page_size  for t < first[q+1] - first[q];
 *   first [n_req + 1] int32 (device): exclusive prefix of the request
 *   lengths; page_table [n_req, pt_stride] int32 (device); slots [capacity]
 *   int32 out.  Tokens at or past `capacity` are not written; a token whose
 *   page index reaches pt_stride gets slot -1.
 *
 * moe_kv_move: copies, for every token i, heads [src_head0, src_head0 +
 *   n_heads) of slot src_slot[i] of its source pool into heads [dst_head0,
 *   dst_head0 + n_heads) of slot dst_slot[i] of the destination pool, for K
 *   and, when src_v / dst_v are given (both or neither), for V.  Tokens
 *   [src_first[q], src_first[q+1]) come from source pool q (q < n_src <=
 *   MOE_MAX_KV_SOURCES), e.g. the pools of the EP ranks whose requests move,
 *   so one launch moves a layer; src_k / src_v / src_slots are HOST arrays
 *   of n_src entries (device pools and their slot counts), src_first a HOST
 *   array of n_src + 1 token offsets (non-decreasing, from 0).  All source
 *   pools have src_heads heads.  src_slot / dst_slot: device int32 slot
 *   vectors of at least src_first[n_src] entries (e.g. from moe_kv_slots).
 *   Entries with a slot outside [0, slots) of their pool are skipped.
 *   Bit-exact copies; destinations of different tokens must not overlap.
 *   A source that supplies no tokens may be NULL; with no tokens at all
 *   nothing is launched.
 * Both calls only read and write the caller's buffers (no allocation) and
 * are asynchronous on `stream`.  Errors: MOE_ERR_INVALID_ARG for null or
 * misaligned pointers, negative sizes, decreasing offsets or head ranges
 * outside the pools; MOE_ERR_UNSUPPORTED for head_dim not a multiple of 8 or
 * n_src above MOE_MAX_KV_SOURCES.
 * Limits: head_dim a positive multiple of 8; 16-byte aligned pools.
 */
moe_status moe_kv_slots(const int32_t *page_table, int64_t pt_stride, const int32_t *first, int n_req,
                        int page_size, int32_t *slots, int64_t capacity, void *stream);
moe_status moe_kv_move(int n_src, const uint16_t *const *src_k, const uint16_t *const *src_v,
                       const int64_t *src_slots, const int64_t *src_first, int src_heads, uint16_t *dst_k,
                       uint16_t *dst_v, int64_t dst_slots, int dst_heads, int head_dim, int src_head0,
                       int dst_head0, int n_heads, const int32_t *src_slot, const int32_t *dst_slot,
                       void *stream);

/*
 * Layout-switch control (host only: arguments are host pointers, no device
 * is touched, nothing is enqueued).  These calls allocate host memory for
 * their own sorting and are safe to call from several threads on distinct
 * policy objects.
 *
 * moe_policy: the switch coordinator's state (Sec. 4.5), owned by the
 *   caller; set it up with moe_policy_init and feed moe_policy_step the
 *   global in-flight request count once per decode iteration, between
 *   steps.  The rule has hysteresis: from TP, one sample above t_high is
 *   enough to request EP; from EP, TP is requested once the average of
 *   the last `window` samples (fewer at start) is under t_low <= t_high.
 *   After a switch, and after a cancelled attempt, no attempt is made for
 *   cooldown_s seconds (times are the caller's clock, e.g. seconds since
 *   start).  target_fits tells whether the other mode can hold the live
 *   KV cache (moe_kv_fits); if not the switch is cancelled (decision
 *   MOE_SWITCH_CANCELLED) and the mode stays.  Paper values: t_high = 256,
 *   cooldown 5 s; interactive serving t_low = 0.8 t_high, window 8;
 *   rollout t_low = t_high, window 1.
 * moe_partition_requests: the deterministic TP->EP ownership (Sec. 3.2):
 *   requests by decreasing length (ties in input order), each placed on the
 *   rank with the least load tokens_r / T + requests_r / N (ties to the
 *   lower rank), in exact integer arithmetic so every rank computes the
 *   same owners.  tokens [n] (>= 0), owner [n] out; rank_tokens [P] and
 *   rank_requests [P] out, optional (NULL).
 * moe_kv_fits: whether every rank's KV pool, `capacity` (page, head) units,
 *   holds the live requests in `mode`: a request of t tokens takes
 *   ceil(t / page_size) pages of every head its rank holds; under EP a rank
 *   holds all n_kv_heads of its own requests (owner [n] required), under TP
 *   max(1, n_kv_heads / P) heads of every request (a head is replicated
 *   over P / n_kv_heads ranks when there are fewer heads than ranks).
 *   n_kv_heads and P must divide one another (else MOE_ERR_UNSUPPORTED).
 * moe_policy_crossover: the initial threshold from decode costs probed in
 *   both modes at n distinct batch sizes (Sec. 4.5): the smallest probed
 *   size from which EP is no slower than TP at every larger probed size;
 *   HUGE_VAL if EP is slower at the largest.
 */
#define MOE_POLICY_MAX_WINDOW 1024
typedef enum moe_mode { MOE_MODE_TP = 0, MOE_MODE_EP = 1 } moe_mode;
typedef enum moe_decision { MOE_STAY = 0, MOE_SWITCH = 1, MOE_SWITCH_CANCELLED = 2 } moe_decision;
typedef struct moe_policy {
    double t_high, t_low, cooldown_s;
    int32_t window, mode;        /* mode: moe_mode, the current layout */
    int32_t n_hist, head;        /* ring of the last `window` counts */
    int32_t has_event, reserved;
    double last_event_s;         /* last switch or cancelled attempt */
    int64_t hist_sum;
    int64_t hist[MOE_POLICY_MAX_WINDOW];
} moe_policy;
moe_status moe_policy_init(moe_policy *pol, double t_high, double t_low, int window, double cooldown_s, int mode);
moe_status moe_policy_step(moe_policy *pol, int64_t in_flight, double now_s, int target_fits, int *decision);
moe_status moe_partition_requests(const int64_t *tokens, int n, int P, int32_t *owner, int64_t *rank_tokens,
                                  int32_t *rank_requests);
moe_status moe_kv_fits(int mode, const int64_t *tokens, int n, const int32_t *owner, int P, int n_kv_heads,
                       int page_size, int64_t capacity, int *fits);
moe_status moe_policy_crossover(const int64_t *batch, const double *tp_cost, const double *ep_cost, int n,
                                double *threshold);

/*
 * Per-kernel timing for measurement.  While enabled, every kernel the
 * library launches is bracketed by HIP events on its own stream (this adds
 * event records to the stream; it never synchronises).  moe_timing_read
 * waits for the recorded events and returns, for one kernel kind, the summed
 * duration in milliseconds and the number of launches since the last reset.
 * Kinds: see enum moe_kernel_kind.  Enabling allocates nothing on the device.
 * Launches on a stream that is being captured into a HIP graph are not
 * timed (a captured event record would not time the replay).
 */
typedef enum moe_kernel_kind {
    MOE_K_ROUTE = 0,
    MOE_K_PERMUTE = 1,   /* count + scan + scatter */
    MOE_K_GATHER = 2,    /* x_perm row gather */
    MOE_K_SCHEDULE = 3,  /* grouped-FFN tile schedule */
    MOE_K_GATE_UP = 4,   /* gate-up GEMM with the SwiGLU epilogue (both tile classes) */
    MOE_K_DOWN = 5,      /* down GEMM (both tile classes, split-K reduction included) */
    MOE_K_COMBINE = 6,
    MOE_K_SPLITK_REDUCE = 7, /* combination of split-K partials of the large tiles (long K only) */
    MOE_K_RESHARD = 8,       /* expert-weight resharding */
    MOE_K_KV_MOVE = 9,       /* paged KV head moves (and their slot expansion) */
    MOE_K_LAYER_PREP = 10,   /* moe_layer_forward: the fused launches of permutation and tile schedule
                                (with routing on larger inputs; on small ones routing is timed as MOE_K_ROUTE) */
    MOE_K_COUNT = 11
} moe_kernel_kind;

/*
 * Device-side timestamps of the grouped GEMM launches (MOE_K_GATE_UP and
 * MOE_K_DOWN of the large-tile path), which also time launches replayed
 * from a HIP graph, where no event can be recorded between kernels.  While
 * enabled, each such launch takes the next slot of a static device table of
 * 4096 slots (a captured launch takes it at capture time, so every replay
 * of it writes that slot) and its workgroups record the earliest start and
 * the latest end, in ticks of the device's 100 MHz constant clock (kept per
 * die to spread the atomics; a launch's duration is from its earliest start
 * on any die to its latest end on any die).
 * moe_timing_device_reset synchronises the device and clears the recorded
 * times (slots stay assigned); moe_timing_device_read synchronises the device
 * and returns, for one kind, the summed duration (ms) and count of the
 * launches that ran since the reset (a slot run several times since then
 * spans from its first start to its last end); moe_timing_device_clear
 * forgets the slots (launches captured before it must not be replayed while
 * device timing is read).  The table is shared by every caller on a device.
 */
moe_status moe_timing_device_enable(int enable);
moe_status moe_timing_device_clear(void);
moe_status moe_timing_device_reset(void);
moe_status moe_timing_device_read(int kind, double *total_ms, int64_t *launches);

moe_status moe_timing_enable(int enable);

/*
 * Matrix-core reference loop for measurement, not part of the layer: the
 * rate at which this device's bf16 matrix cores run with nothing else
 * limiting them.  Launches `grid` workgroups of 8 waves (one per compute
 * unit when grid is the CU count); every wave keeps 2 x 4 independent
 * 32x32 fp32 accumulators and issues `iters` rounds of 8
 * v_mfma_f32_32x32x16_bf16 on operands fixed at its start: hashed uniform
 * values in [-1, 1) and [-0.02, 0.02), or zeros when zero_operands != 0
 * (the same instruction stream without switching activity, so without the
 * clock reduction random operands cause).  Each thread then writes the sum
 * of its accumulators to out[b * 512 + thread] (out: grid * 512 floats,
 * device memory owned by the caller).  One call performs
 * grid * 8 * iters * 8 * 32768 floating-point operations.
 * 1 <= grid <= 65536, 1 <= iters <= 2^24; otherwise MOE_ERR_INVALID_ARG.
 */
moe_status moe_calib_mfma(int grid, int iters, int zero_operands, float *out, void *stream);
/* Time only the kinds whose bit (1 << kind) is set in `kinds` (0 disables);
 * bits at or above MOE_K_COUNT give MOE_ERR_INVALID_ARG. */
moe_status moe_timing_enable_mask(uint32_t kinds);
moe_status moe_timing_reset(void);
moe_status moe_timing_read(int kind, double *total_ms, int64_t *launches);

#ifdef __cplusplus
}
#endif

#endif /* LIBMOE_H */
