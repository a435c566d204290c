// Layout-switch control on the host: the coordinator's policy (Sec. 4.5),
// the deterministic TP->EP request partition (Sec. 3.2), the KV-capacity
// check that gates a switch (Sec. 4.5) and the calibration of the initial
// threshold from probed decode costs (Sec. 4.5).
//
// Every rank must reach the same partition without talking to the others,
// so the partition uses integer arithmetic only: a rank's load
// tokens_r / T + requests_r / N is compared as tokens_r * N + requests_r * T
// in 128 bits.
#include <algorithm>
#include <cmath>
#include <vector>

#include "moe_internal.h"

using moe::set_error;

extern "C" moe_status moe_policy_init(moe_policy *pol, double t_high, double t_low, int window,
                                      double cooldown_s, int mode)
{
    if (!pol) return set_error(MOE_ERR_INVALID_ARG, "moe_policy_init: null policy");
    if (!(t_low <= t_high) || std::isnan(t_low) || std::isnan(t_high))
        return set_error(MOE_ERR_INVALID_ARG, "moe_policy_init: need t_low <= t_high (got %g, %g)", t_low,
                         t_high);
    if (window < 1 || window > MOE_POLICY_MAX_WINDOW)
        return set_error(MOE_ERR_INVALID_ARG, "moe_policy_init: window %d outside [1, %d]", window,
                         MOE_POLICY_MAX_WINDOW);
    if (!(cooldown_s >= 0)) return set_error(MOE_ERR_INVALID_ARG, "moe_policy_init: negative cooldown");
    if (mode != MOE_MODE_TP && mode != MOE_MODE_EP)
        return set_error(MOE_ERR_INVALID_ARG, "moe_policy_init: mode %d", mode);
    *pol = moe_policy{};
    pol->t_high = t_high;
    pol->t_low = t_low;
    pol->cooldown_s = cooldown_s;
    pol->window = window;
    pol->mode = mode;
    return MOE_OK;
}

extern "C" moe_status moe_policy_step(moe_policy *pol, int64_t in_flight, double now_s, int target_fits,
                                      int *decision)
{
    if (!pol || !decision) return set_error(MOE_ERR_INVALID_ARG, "moe_policy_step: null pointer");
    if (pol->window < 1 || pol->window > MOE_POLICY_MAX_WINDOW || pol->n_hist < 0 || pol->n_hist > pol->window ||
        pol->head < 0 || pol->head >= pol->window)
        return set_error(MOE_ERR_INVALID_ARG, "moe_policy_step: policy not initialised");
    if (in_flight < 0) return set_error(MOE_ERR_INVALID_ARG, "moe_policy_step: negative count");
    // the window: the last `window` counts, whatever the mode was
    if (pol->n_hist == pol->window) pol->hist_sum -= pol->hist[pol->head];
    else ++pol->n_hist;
    pol->hist[pol->head] = in_flight;
    pol->hist_sum += in_flight;
    pol->head = (pol->head + 1) % pol->window;

    *decision = MOE_STAY;
    if (pol->has_event && now_s - pol->last_event_s < pol->cooldown_s) return MOE_OK;
    bool want;
    if (pol->mode == MOE_MODE_TP)
        want = (double)in_flight > pol->t_high;                         // a load rise: switch at once
    else
        want = (double)pol->hist_sum / pol->n_hist < pol->t_low;        // a sustained dip only
    if (!want) return MOE_OK;
    pol->has_event = 1;
    pol->last_event_s = now_s;
    if (!target_fits) {
        *decision = MOE_SWITCH_CANCELLED;                               // retried after the cooldown
        return MOE_OK;
    }
    pol->mode = pol->mode == MOE_MODE_TP ? MOE_MODE_EP : MOE_MODE_TP;
    *decision = MOE_SWITCH;
    return MOE_OK;
}

extern "C" moe_status moe_partition_requests(const int64_t *tokens, int n, int P, int32_t *owner,
                                             int64_t *rank_tokens, int32_t *rank_requests)
{
    if (n < 0 || P < 1) return set_error(MOE_ERR_INVALID_ARG, "moe_partition_requests: n=%d P=%d", n, P);
    if (n > 0 && (!tokens || !owner)) return set_error(MOE_ERR_INVALID_ARG, "moe_partition_requests: null pointer");
    __int128 T = 0;
    for (int i = 0; i < n; ++i) {
        if (tokens[i] < 0) return set_error(MOE_ERR_INVALID_ARG, "moe_partition_requests: tokens[%d] < 0", i);
        T += tokens[i];
    }
    if (T >= ((__int128)1 << 62))
        return set_error(MOE_ERR_UNSUPPORTED, "moe_partition_requests: token total too large");
    std::vector<int32_t> order(n);
    for (int i = 0; i < n; ++i) order[i] = i;
    // longest first; equal lengths keep their input order
    std::sort(order.begin(), order.end(), [&](int32_t a, int32_t b) {
        return tokens[a] != tokens[b] ? tokens[a] > tokens[b] : a < b;
    });
    std::vector<int64_t> tok(P, 0);
    std::vector<int32_t> req(P, 0);
    for (int32_t i : order) {
        int best = 0;
        __int128 best_load = 0;
        for (int r = 0; r < P; ++r) {
            // tokens_r / T + requests_r / N, scaled by N * T (requests only when T = 0)
            const __int128 load = T > 0 ? (__int128)tok[r] * n + (__int128)req[r] * T : (__int128)req[r];
            if (r == 0 || load < best_load) {
                best = r;
                best_load = load;
            }
        }
        owner[i] = best;
        tok[best] += tokens[i];
        ++req[best];
    }
    for (int r = 0; r < P; ++r) {
        if (rank_tokens) rank_tokens[r] = tok[r];
        if (rank_requests) rank_requests[r] = req[r];
    }
    return MOE_OK;
}

extern "C" moe_status moe_kv_fits(int mode, const int64_t *tokens, int n, const int32_t *owner, int P,
                                  int n_kv_heads, int page_size, int64_t capacity, int *fits)
{
    static const char fn[] = "moe_kv_fits";
    if (!fits) return set_error(MOE_ERR_INVALID_ARG, "%s: null result", fn);
    if (mode != MOE_MODE_TP && mode != MOE_MODE_EP) return set_error(MOE_ERR_INVALID_ARG, "%s: mode %d", fn, mode);
    if (n < 0 || P < 1 || n_kv_heads < 1 || page_size < 1 || capacity < 0)
        return set_error(MOE_ERR_INVALID_ARG, "%s: n=%d P=%d n_kv_heads=%d page_size=%d capacity=%lld", fn, n, P,
                         n_kv_heads, page_size, (long long)capacity);
    if (n_kv_heads % P != 0 && P % n_kv_heads != 0)
        return set_error(MOE_ERR_UNSUPPORTED, "%s: %d KV heads do not split evenly over %d ranks", fn, n_kv_heads,
                         P);
    if (n > 0 && (!tokens || (mode == MOE_MODE_EP && !owner)))
        return set_error(MOE_ERR_INVALID_ARG, "%s: null pointer", fn);
    std::vector<__int128> use(mode == MOE_MODE_EP ? P : 1, 0);
    for (int i = 0; i < n; ++i) {
        if (tokens[i] < 0) return set_error(MOE_ERR_INVALID_ARG, "%s: tokens[%d] < 0", fn, i);
        const __int128 pages = ((__int128)tokens[i] + page_size - 1) / page_size;
        if (mode == MOE_MODE_TP) {
            use[0] += pages * (n_kv_heads >= P ? n_kv_heads / P : 1);   // every request, the rank's heads
        } else {
            if (owner[i] < 0 || owner[i] >= P)
                return set_error(MOE_ERR_INVALID_ARG, "%s: owner[%d]=%d", fn, i, owner[i]);
            use[owner[i]] += pages * n_kv_heads;                          // own requests, every head
        }
    }
    *fits = *std::max_element(use.begin(), use.end()) <= capacity;
    return MOE_OK;
}

extern "C" moe_status moe_policy_crossover(const int64_t *batch, const double *tp_cost, const double *ep_cost, int n,
                                           double *threshold)
{
    if (n < 1 || !batch || !tp_cost || !ep_cost || !threshold)
        return set_error(MOE_ERR_INVALID_ARG, "moe_policy_crossover: n=%d or null pointer", n);
    std::vector<int> idx(n);
    for (int i = 0; i < n; ++i) {
        if (std::isnan(tp_cost[i]) || std::isnan(ep_cost[i]))
            return set_error(MOE_ERR_INVALID_ARG, "moe_policy_crossover: NaN cost at %d", i);
        idx[i] = i;
    }
    std::sort(idx.begin(), idx.end(), [&](int a, int b) { return batch[a] < batch[b]; });
    for (int i = 1; i < n; ++i)
        if (batch[idx[i]] == batch[idx[i - 1]])
            return set_error(MOE_ERR_INVALID_ARG, "moe_policy_crossover: batch size %lld probed twice",
                             (long long)batch[idx[i]]);
    // the smallest probed size from which EP is never slower
    double th = HUGE_VAL;
    for (int j = n - 1; j >= 0 && ep_cost[idx[j]] <= tp_cost[idx[j]]; --j) th = (double)batch[idx[j]];
    *threshold = th;
    return MOE_OK;
}
