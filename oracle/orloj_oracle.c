/*
 * CPU oracle for scoring candidate batches against latency SLOs
 * (Orloj: "Predictably Serving Unpredictable DNNs", arXiv 2209.00159).
 *
 * TEST INFRASTRUCTURE.  This is the plain, slow, fp64 reference that the
 * HIP library is checked against.  Only the test suite, the smoke check and
 * the benchmark's CPU-baseline leg load it; the product path never does.
 * It shares no code, header, table or helper with the HIP library.
 *
 * The quantity computed is exact under the paper's own model: member
 * latencies are independent (§4.2.2), a padded batch runs as long as its
 * slowest member (§4.2.1, the max of the members), and a histogram bin
 * spreads its mass uniformly over the bin (the per-bin integration behind
 * Eq. (2), §4.1).  The steps below follow the paper's order:
 *
 *   1. empirical CDF of each per-class, per-batch-size histogram at the
 *      grid points (§4.2.1: the CDF is read off the histogram; one
 *      distribution per application, §3.2 "Per-Application Tracking");
 *   2. time left before each deadline, relative to now (§4.4, relative
 *      timestamps);
 *   3. CDF of the batch latency as the product of the members' CDFs: the
 *      law of the maximum of independent variables (§4.2.1 for identical
 *      members, §4.2.2 Eq. (8) for different ones, whose integral over a
 *      bin is exactly the change of this product);
 *   4. expected batch latency, Eq. (5) with the batch histogram;
 *   5. each member's probability of finishing by its deadline (§3.1,
 *      §4.1 cost function);
 *   6. expected number of members finishing in time (scheduler objective,
 *      §4.1);
 *   7. each member's priority, Eq. (1) evaluated through the per-bin closed
 *      form Eq. (2) with L the batch latency (§4.2: L is the execution time
 *      of the whole batch), summed over the batch;
 *   8. the highest-scoring candidate (the scheduler pops the top batch,
 *      §3.2 Algorithm 1).
 *
 * Readings taken where the paper is silent or ambiguous:
 *   - candidates are the prefixes of the deadline-ordered queue of length
 *     n <= min(batch size, queue length); a shorter prefix is padded to the
 *     batch size and uses that size's latency table.  prefix_mode = 1 also
 *     scores n up to the queue length ("what-if"), never selected when
 *     n exceeds the batch size;
 *   - the bin frequency h of Eq. (2) is the bin's probability density
 *     (mass / width), so the priority tends to P / E[L] as b -> 0;
 *   - the second case of Eq. (2) uses the lower edge of the same bin;
 *   - one grid [0, K*w) per model shared by all classes and batch sizes;
 *     a deadline at or beyond K*w finishes with probability 1, one at or
 *     before now with probability 0;
 *   - inside a bin the batch CDF is linear (uniform mass per bin);
 *   - the cost of a miss is c = 1 unless per-request costs are given (the
 *     score then sums c_m p_m; finish probabilities are unweighted);
 *   - selection: the largest score; exact ties go to the larger prefix,
 *     then the smaller batch size; no batch when the best score is <= 0;
 *   - affine mode (Eq. (3)): one histogram per class of the solo latency;
 *     a batch of size k whose slowest member takes l runs c0 + c1 k l, so
 *     its CDF at time t is the members' product at (t - c0) / (c1 k) and
 *     its histogram has the bins of that product stretched by c1 k and
 *     shifted by c0 (Eq. (9), read with the Jacobian 1 / (c1 k) that the
 *     printed form leaves out).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>

enum { ORACLE_OK = 0, ORACLE_E_INVALID = 1, ORACLE_E_DATA = 2, ORACLE_E_NOMEM = 4 };

/* Step 1.  cdf[0] = 0 and cdf[k] = (counts[0] + ... + counts[k-1]) / total
 * for k = 1..n_bins, so cdf[n_bins] = 1.  The running sum is an exact
 * integer; the division is one correctly rounded fp64 division. */
int orloj_oracle_cdf(int32_t n_bins, const uint32_t *counts, double *cdf)
{
    if (n_bins < 1 || !counts || !cdf)
        return ORACLE_E_INVALID;
    uint64_t total = 0;
    for (int32_t k = 0; k < n_bins; ++k)
        total += counts[k];
    if (total == 0)
        return ORACLE_E_DATA;
    uint64_t running = 0;
    cdf[0] = 0.0;
    for (int32_t k = 0; k < n_bins; ++k) {
        running += counts[k];
        cdf[k + 1] = (double)running / (double)total;
    }
    return ORACLE_OK;
}

/* Step 3 for one batch: G[k] = prod_i F_i(x_k) over the members' count
 * rows (rows[i * n_bins ...]).  Exposed for the tests. */
int orloj_oracle_batch_cdf(int32_t n_bins, int32_t n_members, const uint32_t *rows,
                           double *G)
{
    if (n_bins < 1 || n_members < 0 || !G || (n_members > 0 && !rows))
        return ORACLE_E_INVALID;
    double *F = (double *)malloc(sizeof(double) * (size_t)(n_bins + 1));
    if (!F)
        return ORACLE_E_NOMEM;
    for (int32_t k = 0; k <= n_bins; ++k)
        G[k] = 1.0;
    for (int32_t i = 0; i < n_members; ++i) {
        int rc = orloj_oracle_cdf(n_bins, rows + (size_t)i * (size_t)n_bins, F);
        if (rc) {
            free(F);
            return rc;
        }
        for (int32_t k = 0; k <= n_bins; ++k)
            G[k] *= F[k];
    }
    free(F);
    return ORACLE_OK;
}

/* Step 5.  P(L_B <= tau) with the batch CDF G at the grid points and a
 * linear CDF inside each bin. */
static double finish_probability(const double *G, int32_t n_bins, double w, double tau)
{
    if (!(tau > 0.0))
        return 0.0;
    double u = tau / w;
    if (u >= (double)n_bins)
        return G[n_bins];
    int32_t k = (int32_t)floor(u);
    double theta = u - (double)k;
    return (1.0 - theta) * G[k] + theta * G[k + 1];
}

/* Step 7.  Eq. (2) of §4.1 bin by bin, cost c = 1, for a request with
 * tau = D - t left and batch-latency bin masses mass[i] on bins
 * [l1, l2) = [i w, (i+1) w).  The exponentials e^{b l} e^{-b D} e^{b t} of
 * Eq. (2) are combined into e^{-b (tau - l)} (relative timestamps, §4.4).
 * Returns E[L] * p(t), i.e. Eq. (2) without its 1/E[L] factor. */
static double priority_times_latency(const double *mass, int32_t n_bins, double w,
                                     double tau, double b)
{
    double acc = 0.0;
    for (int32_t i = 0; i < n_bins; ++i) {
        double l1 = (double)i * w;
        double l2 = (double)(i + 1) * w;
        double h = mass[i] / w;                 /* bin density */
        if (tau > l2)                           /* t < D - l2 */
            acc += h / b * (exp(-b * (tau - l2)) - exp(-b * (tau - l1)));
        else if (tau > l1)                      /* D - l2 <= t < D - l1 */
            acc += h / b * (1.0 - exp(-b * (tau - l1)));
        /* else D - l1 <= t: the bin contributes nothing */
    }
    return acc;
}

/* Step 8 bookkeeping: the best candidate so far among prefixes no longer
 * than their batch size, and the final no-batch rule. */
typedef struct {
    int have;
    double score;
    int64_t n;
    int32_t bs;
} best_so_far;

static void best_consider(best_so_far *bt, int64_t n, int32_t bs, double s)
{
    if (n <= bs) {
        if (!bt->have || s > bt->score || (s == bt->score && n > bt->n)) {
            bt->have = 1;
            bt->score = s;
            bt->n = n;
            bt->bs = bs;
        }
    }
}

static void best_write(const best_so_far *bt, int32_t *sel_n, int32_t *sel_bs, double *sel_score)
{
    if (bt->have && bt->score > 0.0) {
        *sel_n = (int32_t)bt->n;
        *sel_bs = bt->bs;
        *sel_score = bt->score;
    } else {
        *sel_n = 0;
        *sel_bs = 0;
        *sel_score = 0.0;
    }
}

/*
 * All candidates of one model.  counts is [n_bs][n_classes][n_bins]; the
 * queue (cls, deadline_ms) is sorted by deadline.  Outputs, in candidate
 * order (batch size major, prefix length n = 1.. minor):
 *   expected_finish[cand], expected_latency_ms[cand], score[cand];
 * and per member m = 1..n of each candidate:
 *   finish_prob[slot], priority[slot] (priority may be NULL).
 * sel_n = 0 means no batch.
 */
int orloj_oracle_score_model(int32_t n_classes, int32_t n_bins, int32_t n_bs,
                             const int32_t *batch_sizes, double bin_width_ms,
                             const uint32_t *counts, int64_t n_queue, const int32_t *cls,
                             const double *deadline_ms, const double *cost, double now_ms,
                             double b_expo, int32_t prefix_mode, double *finish_prob,
                             double *priority,
                             double *expected_finish, double *expected_latency_ms,
                             double *score, int32_t *sel_n, int32_t *sel_bs,
                             double *sel_score)
{
    const int32_t C = n_classes, K = n_bins;
    const double w = bin_width_ms, b = b_expo;
    if (C < 1 || K < 1 || n_bs < 1 || !batch_sizes || !counts || n_queue < 0 ||
        !(w > 0.0) || !(b > 0.0) || (prefix_mode != 0 && prefix_mode != 1) ||
        !sel_n || !sel_bs || !sel_score)
        return ORACLE_E_INVALID;
    if (n_queue > 0 && (!cls || !deadline_ms))
        return ORACLE_E_INVALID;
    for (int32_t i = 0; i < n_bs; ++i)
        if (batch_sizes[i] < 1 || (i > 0 && batch_sizes[i] <= batch_sizes[i - 1]))
            return ORACLE_E_INVALID;
    for (int64_t i = 0; i < n_queue; ++i) {
        if (cls[i] < 0 || cls[i] >= C || isnan(deadline_ms[i]))
            return ORACLE_E_DATA;
        if (i > 0 && deadline_ms[i] < deadline_ms[i - 1])
            return ORACLE_E_DATA;
        if (cost && !(cost[i] >= 0.0 && cost[i] < INFINITY))
            return ORACLE_E_DATA;
    }

    /* Step 1: every (batch size, class) CDF. */
    size_t row = (size_t)K + 1;
    double *F = (double *)malloc(sizeof(double) * row * (size_t)n_bs * (size_t)C);
    double *G = (double *)malloc(sizeof(double) * row);
    double *mass = (double *)malloc(sizeof(double) * (size_t)K);
    if (!F || !G || !mass) {
        free(F); free(G); free(mass);
        return ORACLE_E_NOMEM;
    }
    for (int32_t bi = 0; bi < n_bs; ++bi)
        for (int32_t c = 0; c < C; ++c) {
            size_t t = (size_t)bi * (size_t)C + (size_t)c;
            if (orloj_oracle_cdf(K, counts + t * (size_t)K, F + t * row)) {
                free(F); free(G); free(mass);
                return ORACLE_E_DATA;
            }
        }

    int64_t cand = 0, slot = 0;
    best_so_far best = {0, 0.0, 0, 0};
    for (int32_t bi = 0; bi < n_bs; ++bi) {
        int64_t cap = prefix_mode ? n_queue
                                  : (n_queue < batch_sizes[bi] ? n_queue : batch_sizes[bi]);
        for (int32_t k = 0; k <= K; ++k)
            G[k] = 1.0;                           /* empty product */
        for (int64_t n = 1; n <= cap; ++n) {
            /* Step 3: add member n to the batch. */
            const double *Fn = F + ((size_t)bi * (size_t)C + (size_t)cls[n - 1]) * row;
            for (int32_t k = 0; k <= K; ++k)
                G[k] *= Fn[k];

            /* Step 4: E[L_B] of the batch histogram (trapezoid of 1 - G). */
            double el = 0.0;
            for (int32_t k = 0; k < K; ++k)
                el += 1.0 - 0.5 * (G[k] + G[k + 1]);
            el *= w;
            for (int32_t k = 0; k < K; ++k)
                mass[k] = G[k + 1] - G[k];

            double e_count = 0.0, s = 0.0;
            for (int64_t m = 1; m <= n; ++m) {
                double tau = deadline_ms[m - 1] - now_ms;            /* step 2 */
                double P = finish_probability(G, K, w, tau);         /* step 5 */
                double p = priority_times_latency(mass, K, w, tau, b) / el;  /* step 7 */
                finish_prob[slot] = P;
                if (priority)
                    priority[slot] = p;
                ++slot;
                e_count += P;                                        /* step 6 */
                s += (cost ? cost[m - 1] : 1.0) * p;                 /* miss cost c */
            }
            expected_finish[cand] = e_count;
            expected_latency_ms[cand] = el;
            score[cand] = s;
            ++cand;

            best_consider(&best, n, batch_sizes[bi], s);             /* step 8 */
        }
    }
    best_write(&best, sel_n, sel_bs, sel_score);
    free(F); free(G); free(mass);
    return ORACLE_OK;
}

/*
 * One scheduler iteration (§3.2 Algorithm 1) for one model, with the paper's
 * own per-request priority (§4.1 Eq. (1)-(2), §4.2, §4.3).
 *
 * Readings taken:
 *   - EstimateBatchLatency of the drop phase is read as "could the request
 *     finish by its deadline run alone at batch size s": r stays in Q_s iff
 *     F_{c_r,s}(tau_r) > 0.  A request in no Q_s is timed out.
 *   - The candidate batch size takes the batch sizes ordered by
 *     (D_{Q_s}, s) descending, D_{Q_s} the earliest deadline in Q_s, and
 *     picks the first one whose Q_s holds at least s requests (an empty Q_s
 *     never qualifies).
 *   - The batch a request joins is unknown when its priority is computed
 *     (§4.3), so its batch latency at batch size s is the max of its own
 *     latency and s - 1 others drawn independently from the model's class
 *     mix F_mix,s = sum_c pi_c F_{c,s} (pi uniform unless weights are given):
 *     CDF F_{c_r,s} F_mix,s^(s-1) (§4.2.1: the max of k identical variables
 *     has CDF F^k).  E[L] in the priority is the model-wide expected batch
 *     latency, of F_mix,s^s (§4.3: all of the model's distributions).
 *   - PopBatch returns the s requests of Q_s with the largest priority at
 *     batch size s; equal priorities go to the earlier queue position.
 *   - Costs (§4.1: the cost c of a miss; App. B: piecewise-step costs).  A
 *     request's cost function is c_r (default 1) times either one step at
 *     its deadline, or, with step_off given, the steps
 *     (step_deadline_ms[j], step_cost[j]) for j in [step_off[r],
 *     step_off[r+1]): deadlines increasing, cumulative costs non-decreasing.
 *     App. B: such a function is the sum of single steps at d_j with costs
 *     c_j - c_{j-1}, so its priority is the matching sum of single-step
 *     priorities.  The drop phase uses the request's last step deadline (a
 *     request still has cost to save until then); the queue order and
 *     D_{Q_s} use deadline_ms.
 *
 * counts is [n_bs][n_classes][n_bins]; weights (n_classes, may be NULL) are
 * the class mix; the queue is sorted by deadline.  Outputs:
 *   timed_out[N]   1 when the request is in no Q_s
 *   score[N]       priority at the candidate batch size for requests in
 *                  Q_cand, else 0
 *   *cand_bs       the candidate batch size (0: no batch)
 *   batch[cand_bs] queue indices of the popped batch, highest priority first
 *   *batch_n       cand_bs, or 0
 */
int orloj_oracle_iterate_model(int32_t n_classes, int32_t n_bins, int32_t n_bs,
                               const int32_t *batch_sizes, double bin_width_ms,
                               const uint32_t *counts, const double *weights,
                               int64_t n_queue, const int32_t *cls, const double *deadline_ms,
                               const double *cost, const int64_t *step_off,
                               const double *step_deadline_ms, const double *step_cost,
                               double now_ms, double b_expo, int32_t *timed_out,
                               double *score, int32_t *cand_bs, int32_t *batch,
                               int32_t *batch_n)
{
    const int32_t C = n_classes, K = n_bins;
    const double w = bin_width_ms, b = b_expo;
    if (C < 1 || K < 1 || n_bs < 1 || !batch_sizes || !counts || n_queue < 0 ||
        !(w > 0.0) || !(b > 0.0) || !cand_bs || !batch_n)
        return ORACLE_E_INVALID;
    if (n_queue > 0 && (!cls || !deadline_ms || !timed_out || !score))
        return ORACLE_E_INVALID;
    for (int32_t i = 0; i < n_bs; ++i)
        if (batch_sizes[i] < 1 || (i > 0 && batch_sizes[i] <= batch_sizes[i - 1]))
            return ORACLE_E_INVALID;
    for (int64_t i = 0; i < n_queue; ++i) {
        if (cls[i] < 0 || cls[i] >= C || isnan(deadline_ms[i]))
            return ORACLE_E_DATA;
        if (i > 0 && deadline_ms[i] < deadline_ms[i - 1])
            return ORACLE_E_DATA;
        if (cost && !(cost[i] >= 0.0 && cost[i] < INFINITY))
            return ORACLE_E_DATA;
        if (step_off) {
            if (step_off[i + 1] <= step_off[i] || (i == 0 && step_off[0] != 0))
                return ORACLE_E_DATA;
            for (int64_t j = step_off[i]; j < step_off[i + 1]; ++j) {
                if (isnan(step_deadline_ms[j]) || !(step_cost[j] >= 0.0 && step_cost[j] < INFINITY))
                    return ORACLE_E_DATA;
                if (j > step_off[i] && (step_deadline_ms[j] <= step_deadline_ms[j - 1] ||
                                        step_cost[j] < step_cost[j - 1]))
                    return ORACLE_E_DATA;
            }
        }
    }
    if (step_off && (!step_deadline_ms || !step_cost))
        return ORACLE_E_INVALID;
    double wsum = 0.0;
    if (weights) {
        for (int32_t c = 0; c < C; ++c) {
            if (!(weights[c] >= 0.0))
                return ORACLE_E_INVALID;
            wsum += weights[c];
        }
        if (!(wsum > 0.0))
            return ORACLE_E_INVALID;
    }

    size_t row = (size_t)K + 1;
    double *F = (double *)malloc(sizeof(double) * row * (size_t)n_bs * (size_t)C);
    double *mix = (double *)malloc(sizeof(double) * row);
    double *G = (double *)malloc(sizeof(double) * row);
    double *dG = (double *)malloc(sizeof(double) * (size_t)K);
    int64_t *in_q = (int64_t *)malloc(sizeof(int64_t) * (size_t)n_bs);
    int64_t *first = (int64_t *)malloc(sizeof(int64_t) * (size_t)n_bs);
    int64_t *order = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n_queue > 0 ? n_queue : 1));
    if (!F || !mix || !G || !dG || !in_q || !first || !order) {
        free(F); free(mix); free(G); free(dG); free(in_q); free(first); free(order);
        return ORACLE_E_NOMEM;
    }
    int rc = ORACLE_OK;
    for (int32_t bi = 0; bi < n_bs && rc == ORACLE_OK; ++bi)
        for (int32_t c = 0; c < C; ++c) {
            size_t t = (size_t)bi * (size_t)C + (size_t)c;
            if (orloj_oracle_cdf(K, counts + t * (size_t)K, F + t * row)) {
                rc = ORACLE_E_DATA;
                break;
            }
        }

    /* Drop phase: Q_s membership, |Q_s| and the earliest deadline in Q_s. */
    for (int32_t bi = 0; bi < n_bs && rc == ORACLE_OK; ++bi) {
        in_q[bi] = 0;
        first[bi] = -1;
    }
    for (int64_t r = 0; r < n_queue && rc == ORACLE_OK; ++r) {
        double last = step_off ? step_deadline_ms[step_off[r + 1] - 1] : deadline_ms[r];
        double tau = last - now_ms;
        int any = 0;
        for (int32_t bi = 0; bi < n_bs; ++bi) {
            const double *Fr = F + ((size_t)bi * (size_t)C + (size_t)cls[r]) * row;
            if (finish_probability(Fr, K, w, tau) > 0.0) {
                any = 1;
                if (in_q[bi]++ == 0)
                    first[bi] = r;
            }
        }
        timed_out[r] = any ? 0 : 1;
        score[r] = 0.0;
    }

    /* Candidate batch size: (D_{Q_s}, s) descending, first with |Q_s| >= s. */
    int32_t cand = -1;
    for (int32_t bi = 0; bi < n_bs && rc == ORACLE_OK; ++bi) {
        if (in_q[bi] < batch_sizes[bi])
            continue;
        if (cand < 0) {
            cand = bi;
            continue;
        }
        double d_new = deadline_ms[first[bi]], d_old = deadline_ms[first[cand]];
        if (d_new > d_old || (d_new == d_old && batch_sizes[bi] > batch_sizes[cand]))
            cand = bi;
    }
    *cand_bs = 0;
    *batch_n = 0;
    if (rc == ORACLE_OK && cand >= 0) {
        const int32_t s = batch_sizes[cand];
        /* The class mix at batch size s and the model-wide E[L] of mix^s. */
        for (int32_t k = 0; k <= K; ++k) {
            double acc = 0.0;
            for (int32_t c = 0; c < C; ++c) {
                double pc = weights ? weights[c] / wsum : 1.0 / (double)C;
                acc += pc * F[((size_t)cand * (size_t)C + (size_t)c) * row + (size_t)k];
            }
            mix[k] = acc;
        }
        double el_model = 0.0;
        for (int32_t k = 0; k < K; ++k)
            el_model += 1.0 - 0.5 * (pow(mix[k], s) + pow(mix[k + 1], s));
        el_model *= w;
        /* Priority of every request in Q_s, from its own batch law. */
        int64_t nq = 0;
        for (int64_t r = 0; r < n_queue; ++r) {
            double last = step_off ? step_deadline_ms[step_off[r + 1] - 1] : deadline_ms[r];
            const double *Fr = F + ((size_t)cand * (size_t)C + (size_t)cls[r]) * row;
            if (!(finish_probability(Fr, K, w, last - now_ms) > 0.0))
                continue;
            for (int32_t k = 0; k <= K; ++k)
                G[k] = Fr[k] * pow(mix[k], s - 1);
            for (int32_t k = 0; k < K; ++k)
                dG[k] = G[k + 1] - G[k];
            double cr = cost ? cost[r] : 1.0, pr = 0.0;
            if (step_off) {
                double below = 0.0;             /* App. B: one single step per cost increment */
                for (int64_t j = step_off[r]; j < step_off[r + 1]; ++j) {
                    double tau_j = step_deadline_ms[j] - now_ms;
                    pr += (step_cost[j] - below) * priority_times_latency(dG, K, w, tau_j, b);
                    below = step_cost[j];
                }
            } else {
                pr = priority_times_latency(dG, K, w, deadline_ms[r] - now_ms, b);
            }
            score[r] = cr * pr / el_model;
            order[nq++] = r;
        }
        /* PopBatch: the s best by priority, ties to the earlier position
         * (a stable selection pass, plainly O(s * |Q_s|)). */
        for (int32_t j = 0; j < s; ++j) {
            int64_t best = j;
            for (int64_t i = j + 1; i < nq; ++i) {
                double si = score[order[i]], sb = score[order[best]];
                if (si > sb || (si == sb && order[i] < order[best]))
                    best = i;
            }
            int64_t tmp = order[j];
            order[j] = order[best];
            order[best] = tmp;
            batch[j] = (int32_t)order[j];
        }
        *cand_bs = s;
        *batch_n = s;
    }
    free(F); free(mix); free(G); free(dG); free(in_q); free(first); free(order);
    return rc;
}

/*
 * Profiler feedback (§3.2 "Long-Term Feedback Loop"): execution times of
 * sampled finished requests, measured alone, are accumulated into the
 * histograms the scheduler reads.  counts is [M][n_bs][C][K] (updated in
 * place); sample i adds one count to model model[i], batch-size index
 * bs_index[i], class cls[i], bin floor(latency_ms[i] / w_q), a latency at
 * or beyond the grid counting in the last bin (the grid's convention).
 * Samples with an index out of range or a latency that is negative or not
 * finite are skipped and counted in *n_rejected.  Resetting the profiling
 * memory at the end of a window is the caller zeroing counts.
 */
int orloj_oracle_accumulate(int32_t n_models, int32_t n_bs, int32_t n_classes, int32_t n_bins,
                            const double *bin_width_ms, int64_t n_samples, const int32_t *model,
                            const int32_t *bs_index, const int32_t *cls,
                            const double *latency_ms, uint32_t *counts, int64_t *n_rejected)
{
    if (n_models < 0 || n_bs < 1 || n_classes < 1 || n_bins < 1 || n_samples < 0 || !n_rejected)
        return ORACLE_E_INVALID;
    if (n_samples > 0 && (!bin_width_ms || !model || !bs_index || !cls || !latency_ms || !counts))
        return ORACLE_E_INVALID;
    int64_t rejected = 0;
    for (int64_t i = 0; i < n_samples; ++i) {
        int32_t q = model[i], b = bs_index[i], c = cls[i];
        double lat = latency_ms[i];
        if (q < 0 || q >= n_models || b < 0 || b >= n_bs || c < 0 || c >= n_classes ||
            !(lat >= 0.0 && lat < INFINITY) || !(bin_width_ms[q] > 0.0)) {
            ++rejected;
            continue;
        }
        double u = floor(lat / bin_width_ms[q]);
        int32_t k = u >= (double)(n_bins - 1) ? n_bins - 1 : (int32_t)u;
        size_t at = (((size_t)q * (size_t)n_bs + (size_t)b) * (size_t)n_classes + (size_t)c) *
                    (size_t)n_bins + (size_t)k;
        counts[at] += 1u;
    }
    *n_rejected = rejected;
    return ORACLE_OK;
}

/*
 * Affine batch-latency mode (§4.2.1 Eq. (3), (5); §4.2.2 Eq. (9)): a batch
 * of batch size s whose slowest member takes l runs for c0 + c1 s l, with
 * model constants c0 (ms) and c1, and one histogram per class of the
 * latency of a request run alone (counts is [n_classes][n_bins], no
 * batch-size dimension).  For candidate (n, s):
 *   X = max of the members' solo latencies, CDF G on the base grid as in
 *       step 3 (the product of the members' CDFs);
 *   L_B = c0 + c1 s X, so its histogram has the bins of X mapped to
 *       [c0 + c1 s i w, c0 + c1 s (i+1) w) with the same masses;
 *   E[L_B] = c0 + c1 s E[X]                                     (Eq. (5));
 *   P_m = P(L_B <= tau_m), and the priority is Eq. (2) on L_B's histogram:
 *       both are the base-grid routines with the bin width c1 s w and the
 *       time left tau_m - c0.
 * Outputs, candidate order and selection are those of
 * orloj_oracle_score_model.
 */
int orloj_oracle_score_model_affine(int32_t n_classes, int32_t n_bins, int32_t n_bs,
                                    const int32_t *batch_sizes, double bin_width_ms,
                                    const uint32_t *counts, double c0_ms, double c1,
                                    int64_t n_queue, const int32_t *cls,
                                    const double *deadline_ms, const double *cost,
                                    double now_ms, double b_expo, int32_t prefix_mode,
                                    double *finish_prob, double *priority,
                                    double *expected_finish, double *expected_latency_ms,
                                    double *score, int32_t *sel_n, int32_t *sel_bs,
                                    double *sel_score)
{
    const int32_t C = n_classes, K = n_bins;
    const double w = bin_width_ms, b = b_expo;
    if (C < 1 || K < 1 || n_bs < 1 || !batch_sizes || !counts || n_queue < 0 ||
        !(w > 0.0) || !(b > 0.0) || !(c0_ms >= 0.0 && c0_ms < INFINITY) ||
        !(c1 > 0.0 && c1 < INFINITY) || (prefix_mode != 0 && prefix_mode != 1) ||
        !sel_n || !sel_bs || !sel_score)
        return ORACLE_E_INVALID;
    if (n_queue > 0 && (!cls || !deadline_ms))
        return ORACLE_E_INVALID;
    for (int32_t i = 0; i < n_bs; ++i)
        if (batch_sizes[i] < 1 || (i > 0 && batch_sizes[i] <= batch_sizes[i - 1]))
            return ORACLE_E_INVALID;
    for (int64_t i = 0; i < n_queue; ++i) {
        if (cls[i] < 0 || cls[i] >= C || isnan(deadline_ms[i]))
            return ORACLE_E_DATA;
        if (i > 0 && deadline_ms[i] < deadline_ms[i - 1])
            return ORACLE_E_DATA;
        if (cost && !(cost[i] >= 0.0 && cost[i] < INFINITY))
            return ORACLE_E_DATA;
    }
    size_t row = (size_t)K + 1;
    double *F = (double *)malloc(sizeof(double) * row * (size_t)C);
    double *G = (double *)malloc(sizeof(double) * row);
    double *hist = (double *)malloc(sizeof(double) * (size_t)K);
    if (!F || !G || !hist) {
        free(F); free(G); free(hist);
        return ORACLE_E_NOMEM;
    }
    for (int32_t c = 0; c < C; ++c)
        if (orloj_oracle_cdf(K, counts + (size_t)c * (size_t)K, F + (size_t)c * row)) {
            free(F); free(G); free(hist);
            return ORACLE_E_DATA;
        }
    int64_t cand = 0, slot = 0;
    best_so_far best = {0, 0.0, 0, 0};
    for (int32_t bi = 0; bi < n_bs; ++bi) {
        const double ws = c1 * (double)batch_sizes[bi] * w;     /* bin width of L_B */
        int64_t cap = prefix_mode ? n_queue
                                  : (n_queue < batch_sizes[bi] ? n_queue : batch_sizes[bi]);
        for (int32_t k = 0; k <= K; ++k)
            G[k] = 1.0;
        for (int64_t n = 1; n <= cap; ++n) {
            const double *Fn = F + (size_t)cls[n - 1] * row;
            for (int32_t k = 0; k <= K; ++k)
                G[k] = G[k] * Fn[k];
            double ex = 0.0;                                    /* E[X], Eq. (5) */
            for (int32_t k = 0; k < K; ++k)
                ex += 1.0 - 0.5 * (G[k] + G[k + 1]);
            ex *= w;
            const double el = c0_ms + c1 * (double)batch_sizes[bi] * ex;
            for (int32_t k = 0; k < K; ++k)
                hist[k] = G[k + 1] - G[k];
            double e_count = 0.0, sc = 0.0;
            for (int64_t m = 1; m <= n; ++m) {
                double tau = deadline_ms[m - 1] - now_ms;
                double P = tau > 0.0 ? finish_probability(G, K, ws, tau - c0_ms) : 0.0;
                double p = tau > 0.0 ? priority_times_latency(hist, K, ws, tau - c0_ms, b) / el : 0.0;
                finish_prob[slot] = P;
                if (priority)
                    priority[slot] = p;
                ++slot;
                e_count += P;
                sc += (cost ? cost[m - 1] : 1.0) * p;
            }
            expected_finish[cand] = e_count;
            expected_latency_ms[cand] = el;
            score[cand] = sc;
            ++cand;
            best_consider(&best, n, batch_sizes[bi], sc);
        }
    }
    best_write(&best, sel_n, sel_bs, sel_score);
    free(F); free(G); free(hist);
    return ORACLE_OK;
}
