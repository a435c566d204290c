/*
 * CPU oracle for the MoE layer forward on one GPU's share of the work.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg use it.  It shares no code, header, table or helper with
 * the HIP library.
 *
 * It is a plain, slow, obviously correct restatement, in double precision,
 * of what the layer computes.  The paper (Sec. 3.1, "Weights Resharding")
 * fixes the expert shapes: under EP a rank holds E/P whole experts,
 * W13 (E/P, 2I, H) with the gate projection stacked before the up
 * projection, and W2 (E/P, H, I); under TP a rank holds W13 (E, 2I/P, H)
 * and W2 (E, H, I/P), sliced along the intermediate dimension on the output
 * side of gate-up and the input side of down.  Sec. 1 and Sec. 3 state that
 * both layouts compute the same function over the same weights, so the sum
 * of the P partial outputs equals the unsliced layer.
 *
 * The paper does not state the gating function.  The reading used here:
 * softmax over all E router logits, keep the k largest (ties to the lower
 * expert id, -0.0 equal to +0.0), renormalise the kept probabilities to sum
 * to one.  Permuted order inside an expert is ascending token.  Gate weights
 * are applied to each expert's output.  No token is dropped.
 *
 * Parity pins (in tests/, all on the CPU): brute-force sort and softmax from
 * numpy/scipy for routing, a stable library argsort for the permutation, a
 * dense all-experts evaluation with a top-k mask, a torch SwiGLU MLP for
 * E = k = 1, closed forms, and the sum-of-partials identities for both
 * layouts.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* bfloat16 bit pattern -> value (exact: bf16 is the top half of a float). */
static double bf16v(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

int oracle_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void oracle_set_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/*
 * Gating (routing).  For each token t the experts are ordered by logit,
 * largest first, equal logits by ascending expert id; the first k are the
 * token's experts, in that order.  Their weights are the softmax
 * probabilities over all E logits, divided by the sum of the k kept
 * probabilities.
 *   logits [T, E] fp32;  ids [T, k] int32;  w [T, k] double.
 * Logits must be finite.
 */
void oracle_route(const float *logits, int64_t T, int E, int k, int32_t *ids, double *w)
{
    char *taken = (char *)malloc((size_t)E);
    double *p = (double *)malloc((size_t)E * sizeof(double));
    for (int64_t t = 0; t < T; ++t) {
        const float *l = logits + t * E;
        /* selection: k times, the largest remaining logit; strict '>' while
         * scanning ids upward keeps the lowest id among equal logits, and
         * IEEE comparison already treats -0.0 and +0.0 as equal. */
        memset(taken, 0, (size_t)E);
        for (int j = 0; j < k; ++j) {
            int best = -1;
            for (int e = 0; e < E; ++e) {
                if (taken[e]) continue;
                if (best < 0 || l[e] > l[best]) best = e;
            }
            taken[best] = 1;
            ids[t * k + j] = best;
        }
        /* softmax over all E logits (shifted by the max for range) */
        double mx = (double)l[0];
        for (int e = 1; e < E; ++e)
            if ((double)l[e] > mx) mx = (double)l[e];
        double z = 0.0;
        for (int e = 0; e < E; ++e) {
            p[e] = exp((double)l[e] - mx);
            z += p[e];
        }
        for (int e = 0; e < E; ++e) p[e] /= z;
        /* renormalise over the kept experts */
        double s = 0.0;
        for (int j = 0; j < k; ++j) s += p[ids[t * k + j]];
        for (int j = 0; j < k; ++j) w[t * k + j] = p[ids[t * k + j]] / s;
    }
    free(taken);
    free(p);
}

/*
 * Permutation.  A (token, slot) pair p = t*k + j is local when its expert
 * lies in [e0, e0 + El).  Local pairs are listed expert by expert, and
 * inside an expert by ascending token (a token picks an expert at most
 * once).  Row r of the permuted buffer holds pair row_to_pair[r];
 * pair_to_row[p] is that row, or -1 for a non-local pair.  counts[le] is the
 * number of pairs of local expert le and offsets[] its exclusive prefix sum,
 * offsets[El] being the number of local pairs.
 */
void oracle_permute(const int32_t *ids, int64_t T, int k, int e0, int El,
                    int32_t *counts, int32_t *offsets, int32_t *row_to_pair,
                    int32_t *pair_to_row)
{
    int64_t n = 0;
    for (int64_t p = 0; p < T * k; ++p) pair_to_row[p] = -1;
    for (int le = 0; le < El; ++le) {
        offsets[le] = (int32_t)n;
        counts[le] = 0;
        for (int64_t t = 0; t < T; ++t)
            for (int j = 0; j < k; ++j)
                if (ids[t * k + j] == e0 + le) {
                    row_to_pair[n] = (int32_t)(t * k + j);
                    pair_to_row[t * k + j] = (int32_t)n;
                    ++n;
                    ++counts[le];
                }
    }
    offsets[El] = (int32_t)n;
}

/*
 * One expert's SwiGLU FFN on one token row:
 *   g_i = sum_h x_h W13[i][h],  u_i = sum_h x_h W13[I_s + i][h]   (i < I_s)
 *   a_i = silu(g_i) * u_i,  silu(g) = g / (1 + exp(-g))
 *   y_h = sum_i a_i W2[h][i]
 * x [H], w13 [2*I_s, H], w2 [H, I_s] as bf16 bits; y [H] double.
 */
static void expert_ffn_row(const uint16_t *x, const uint16_t *w13, const uint16_t *w2,
                           int H, int Is, double *a, double *y)
{
    for (int i = 0; i < Is; ++i) {
        const uint16_t *gr = w13 + (int64_t)i * H;
        const uint16_t *ur = w13 + (int64_t)(Is + i) * H;
        double g = 0.0, u = 0.0;
        for (int h = 0; h < H; ++h) {
            double xv = bf16v(x[h]);
            g += xv * bf16v(gr[h]);
            u += xv * bf16v(ur[h]);
        }
        a[i] = g / (1.0 + exp(-g)) * u;
    }
    for (int h = 0; h < H; ++h) {
        const uint16_t *dr = w2 + (int64_t)h * Is;
        double s = 0.0;
        for (int i = 0; i < Is; ++i) s += a[i] * bf16v(dr[i]);
        y[h] = s;
    }
}

/*
 * Grouped FFN stage: row r of x_perm, which belongs to local expert le when
 * offsets[le] <= r < offsets[le+1], goes through that expert's FFN.
 *   x_perm [>= offsets[El], H]; w13 [El, 2*I_s, H]; w2 [El, H, I_s];
 *   y [offsets[El], H] double.
 */
void oracle_grouped_ffn(const uint16_t *x_perm, const int32_t *offsets, int El, int H, int Is,
                        const uint16_t *w13, const uint16_t *w2, double *y)
{
    int64_t n = offsets[El];
#pragma omp parallel
    {
        double *a = (double *)malloc((size_t)Is * sizeof(double));
#pragma omp for schedule(dynamic, 1)
        for (int64_t r = 0; r < n; ++r) {
            int le = 0;
            while (!(offsets[le] <= r && r < offsets[le + 1])) ++le;
            expert_ffn_row(x_perm + r * H, w13 + (int64_t)le * 2 * Is * H,
                           w2 + (int64_t)le * H * Is, H, Is, a, y + r * H);
        }
        free(a);
    }
}

/*
 * Combine stage (unpermute and weighted reduce):
 *   out[t] = base[t] + shared[t] + sum over local slots j of w[t,j] * y[pair_to_row[t*k+j]]
 * base[t] is the prior out[t] when accumulate != 0, else 0; shared[t] is
 * shared_y[t - sb] for sb <= t < sb + sc (shared_y may be NULL), else 0.
 * y and shared_y are bf16 bits; w fp32 (as the GPU receives it); out double.
 */
void oracle_combine(const uint16_t *y, const int32_t *pair_to_row, const float *w, int64_t T, int k,
                    int H, const uint16_t *shared_y, int64_t sb, int64_t sc, int accumulate,
                    const uint16_t *prior, double *out)
{
    for (int64_t t = 0; t < T; ++t)
        for (int h = 0; h < H; ++h) {
            double s = accumulate ? bf16v(prior[t * H + h]) : 0.0;
            if (shared_y && t >= sb && t < sb + sc) s += bf16v(shared_y[(t - sb) * H + h]);
            for (int j = 0; j < k; ++j) {
                int32_t r = pair_to_row[t * k + j];
                if (r >= 0) s += (double)w[t * k + j] * bf16v(y[(int64_t)r * H + h]);
            }
            out[t * H + h] = s;
        }
}

/*
 * The whole layer, by definition, on a chosen set of tokens:
 *   out[t] = sum over j with e0 <= ids[t,j] < e0+El of w[t,j] * FFN_{ids[t,j]}(x_t)
 *            + (sb <= t < sb+sc ? FFN_shared(x_t) : 0)
 * ids/w come from oracle_route.  tokens[nt] lists the token indices to
 * evaluate; out [nt, H] double.  sw13/sw2 (shared expert, intermediate
 * Is_sh) may be NULL when sc == 0.
 */
void oracle_layer_tokens(const uint16_t *x, int H, const int32_t *ids, const double *w, int k,
                         int e0, int El, int Is, const uint16_t *w13, const uint16_t *w2,
                         const uint16_t *sw13, const uint16_t *sw2, int Is_sh, int64_t sb,
                         int64_t sc, const int64_t *tokens, int64_t nt, double *out)
{
    int amax = Is > Is_sh ? Is : Is_sh;
#pragma omp parallel
    {
        double *a = (double *)malloc((size_t)(amax > 0 ? amax : 1) * sizeof(double));
        double *y = (double *)malloc((size_t)H * sizeof(double));
#pragma omp for schedule(dynamic, 1)
        for (int64_t q = 0; q < nt; ++q) {
            int64_t t = tokens[q];
            double *o = out + q * H;
            for (int h = 0; h < H; ++h) o[h] = 0.0;
            for (int j = 0; j < k; ++j) {
                int e = ids[t * k + j];
                if (e < e0 || e >= e0 + El) continue;
                int le = e - e0;
                expert_ffn_row(x + t * H, w13 + (int64_t)le * 2 * Is * H,
                               w2 + (int64_t)le * H * Is, H, Is, a, y);
                for (int h = 0; h < H; ++h) o[h] += w[t * k + j] * y[h];
            }
            if (sc > 0 && t >= sb && t < sb + sc) {
                expert_ffn_row(x + t * H, sw13, sw2, H, Is_sh, a, y);
                for (int h = 0; h < H; ++h) o[h] += y[h];
            }
        }
        free(a);
        free(y);
    }
}
