/*
 * orloj.h - C ABI of the MI355X candidate-batch scorer.
 *
 * Scores candidate batches against latency SLOs with empirical
 * distributions of request execution time, the hot path of Orloj
 * ("Predictably Serving Unpredictable DNNs", arXiv 2209.00159):
 *
 *   orloj_build_cdfs        histogram -> complementary CDF table
 *   orloj_output_sizes      host-side sizing of the per-candidate outputs
 *   orloj_score_candidates  every prefix candidate at every batch size:
 *                           batch CDF, E[L_B], finish probabilities,
 *                           expected finish count, priority score
 *   orloj_score_candidates_affine  the same with the affine batch-latency
 *                           law c0 + c1 s l of §4.2.1 (one table per class)
 *   orloj_score_candidates_affine_noalloc  the same, allocating nothing
 *   orloj_select_batch      highest-scoring candidate per model
 *   orloj_build_model_laws  model-wide batch laws for the scheduler iteration
 *   orloj_iterate           one Algorithm 1 iteration per model (drop phase,
 *                           candidate batch size, PopBatch by priority)
 *   orloj_accumulate        profiler feedback into the histograms
 *   orloj_sched_*           host runtime: per-model deadline queues, drop
 *                           phase, one score + select round per call
 *   orloj_simulate_trace    trace-driven worker simulation on that runtime
 *
 * Conventions.  Pointers named d_* are device (HBM) pointers owned by the
 * caller; h_* pointers and the structs are host memory read during the call
 * only.  Every call is asynchronous on the context's HIP stream: it returns
 * after validating its arguments and enqueueing kernels.  Argument problems
 * return ORLOJ_E_INVALID (or ORLOJ_E_UNSUPPORTED for shapes beyond the
 * compiled limits) before anything is launched; problems found in device
 * data (a histogram with no samples, a class id out of range, a NaN or
 * unsorted deadline) are recorded on the device and returned by
 * orloj_sync() as ORLOJ_E_DATA.  HIP runtime failures return ORLOJ_E_HIP.
 * orloj_last_error() describes the most recent failure of a context.
 * Times are milliseconds throughout.  A context is not thread-safe; calls
 * that share a context must be serialised by the caller.
 */
#ifndef ORLOJ_H
#define ORLOJ_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum orloj_status {
    ORLOJ_OK = 0,
    ORLOJ_E_INVALID = 1,      /* bad argument, detected on the host */
    ORLOJ_E_DATA = 2,         /* bad device data, reported by orloj_sync */
    ORLOJ_E_HIP = 3,          /* HIP runtime error */
    ORLOJ_E_NOMEM = 4,        /* host or device allocation failed */
    ORLOJ_E_UNSUPPORTED = 5   /* valid but beyond the compiled limits */
};

/* Candidate sets (the prefixes of each model's deadline-ordered queue).
 * TRIANGLE: at batch size s, prefixes n = 1 .. min(s, N).  A prefix shorter
 * than s is padded to s and uses s's latency table (a padded batch runs as
 * long as its slowest member, §4.2.1).
 * RECT: prefixes n = 1 .. N at every batch size ("what-if" scores for
 * n > s, never selected). */
enum orloj_prefix_mode { ORLOJ_PREFIX_TRIANGLE = 0, ORLOJ_PREFIX_RECT = 1 };

/* Compiled limits. */
#define ORLOJ_MAX_BINS 8192       /* histogram bins per table */
#define ORLOJ_MAX_BATCH_SIZES 256 /* entries of the batch-size set */
#define ORLOJ_MAX_PREFIX 256      /* longest prefix scored per batch size */
/* Floats of the fixed scratch of orloj_score_candidates_affine_noalloc
 * (4 MiB per device). */
#define ORLOJ_NOALLOC_SCRATCH_FLOATS (1 << 20)

typedef struct orloj_ctx orloj_ctx;

/* Create a context on HIP device `hip_device` that enqueues on `hip_stream`
 * (a hipStream_t; NULL = the null stream).  Allocates a small device status
 * word.  Returns ORLOJ_OK and *out, or an error with *out = NULL. */
int orloj_create(orloj_ctx **out, int32_t hip_device, void *hip_stream);

/* Free a context (waits for its stream first).  NULL is a no-op. */
void orloj_destroy(orloj_ctx *ctx);

/* Switch the stream later calls enqueue on.  If the context holds a
 * scratch block (orloj_score_candidates_affine, or orloj_iterate on long
 * queues), work already enqueued on the previous stream is waited for
 * first. */
int orloj_set_stream(orloj_ctx *ctx, void *hip_stream);

/* Prefix steps one score workgroup takes (orloj_score_candidates and
 * orloj_score_candidates_affine).  A (model, batch size) pair's prefix
 * lengths are scored in sequence; when a launch has too few pairs to fill
 * the GPU, splitting them into chunks of `steps` (each chunk first rebuilds
 * the batch CDF of the prefixes before it) shortens the launch.  -1 (the
 * default): chosen per launch from the queue lengths and the device's
 * compute units; 0: never split; k > 0: chunks of k.  The results are the
 * same bits whatever the setting.  ORLOJ_E_INVALID for steps < -1. */
int orloj_set_score_chunk(orloj_ctx *ctx, int32_t steps);

/* Text of the last error of `ctx` (never NULL; "" when none). */
const char *orloj_last_error(const orloj_ctx *ctx);

/* Wait for all work enqueued on the context's stream, then report and clear
 * any device-detected data error (ORLOJ_E_DATA). */
int orloj_sync(orloj_ctx *ctx);

/*
 * The shared grid of a launch.  Every model has n_classes request classes
 * (applications, §3.2 "Per-Application Tracking") and one latency
 * histogram per (batch size, class) on its own grid of n_bins bins of width
 * bin_width_ms[q]: bin k covers [k w, (k+1) w).  Mass beyond the grid is
 * expected in the last bin.
 */
typedef struct orloj_grid {
    int32_t n_models;               /* M >= 0 */
    int32_t n_classes;              /* C >= 1 */
    int32_t n_bins;                 /* K in [1, ORLOJ_MAX_BINS] */
    int32_t n_bs;                   /* |S| in [1, ORLOJ_MAX_BATCH_SIZES] */
    const int32_t *batch_sizes;     /* host [n_bs], strictly increasing, >= 1 */
    const double *d_bin_width_ms;   /* device [M], each > 0 */
} orloj_grid;

/*
 * Pending requests (§3.1: release time, deadline = release + SLO), one
 * queue per model, stored back to back (CSR).  Each queue is sorted by
 * deadline, non-decreasing; equal deadlines keep the caller's order.
 */
typedef struct orloj_queues {
    const int64_t *h_queue_off;     /* host [M+1], h_queue_off[0] = 0, non-decreasing */
    const int64_t *d_queue_off;     /* device copy of h_queue_off */
    const int32_t *d_class;         /* device [N], class id in [0, C) */
    const double *d_deadline_ms;    /* device [N] absolute deadlines */
    const double *d_now_ms;         /* device [M] current time per model */
    const double *d_cost;           /* device [N] miss cost c of each request (§4.1), finite,
                                       >= 0; NULL = 1 for every request.  It weights the
                                       request's priority; finish probabilities are not
                                       weighted.  A negative or non-finite cost is a data
                                       error (the request then counts with cost 0). */
} orloj_queues;

/*
 * Histogram -> CDF table (§4.2.1: the CDF of a request's latency is read off
 * its histogram), stored as its complement.  For each of n_rows rows of
 * n_bins uint32 counts:
 *   d_ccdf[r][k] = 1 - F(x_{k+1}) = (total - counts[0..k] summed) / total,
 * the probability that the latency exceeds the right edge of bin k.  Entry
 * n_bins-1 is exactly 0.  The running sums are exact 64-bit integers and the
 * complement keeps full relative precision where F is near 1, which the
 * batch CDF (a product of many member CDFs) needs.  Rows are laid out
 * [model][batch size][class][bin] for orloj_score_candidates.  A row with
 * total 0 is a data error (its entries are written as NaN).
 *
 * d_support (optional, NULL = not written): int32 [n_rows][2], the first and
 * the last bin holding mass.  Entries before the first are exactly 1 and
 * entries from the last on are exactly 0, so orloj_score_candidates can skip
 * reading them.  A row with total 0 gets {0, 0}.
 * d_counts, d_ccdf and d_support must not overlap.
 */
int orloj_build_cdfs(orloj_ctx *ctx, int64_t n_rows, int32_t n_bins,
                     const uint32_t *d_counts, float *d_ccdf, int32_t *d_support);

/*
 * Output sizing (host only, no launch).  For model q with queue length N_q
 * and batch size s_b, ncap(q,b) = min(s_b, N_q) (TRIANGLE) or N_q (RECT).
 *   h_cand_off[q+1] - h_cand_off[q] = sum_b ncap(q,b)
 *   h_prob_off[q+1] - h_prob_off[q] = sum_b ncap(q,b) (ncap(q,b) + 1) / 2
 * Candidate (q, b, n) sits at h_cand_off[q] + sum_{b'<b} ncap(q,b') + n - 1.
 * Member m (1..n) of that candidate sits at
 *   h_prob_off[q] + sum_{b'<b} T(ncap(q,b')) + T(n-1) + m - 1,  T(j) = j(j+1)/2.
 * h_cand_off / h_prob_off are host [M+1] outputs; either may be NULL.
 */
int orloj_output_sizes(const orloj_grid *grid, const orloj_queues *queues,
                       int32_t prefix_mode, int64_t *n_cands, int64_t *n_probs,
                       int64_t *h_cand_off, int64_t *h_prob_off);

/*
 * Score every candidate of every model in one launch (§4.1-§4.2).
 * For candidate (q, b, n) with members i = 1..n of q's queue:
 *   G(x_k)      = prod_i F_{c_i, b}(x_k)      batch-latency CDF: the max of
 *                 independent member latencies (§4.2.1-§4.2.2), linear
 *                 inside a bin;
 *   E[L_B]      = sum_k (G(x_{k+1}) - G(x_k)) (x_k + w/2)        (Eq. (5));
 *   P_m         = G(D_m - now)  (0 if the deadline has passed, 1 beyond
 *                 the grid);
 *   p_m         = Eq. (1)-(2) priority of member m with L = L_B, miss cost
 *                 1, anticipated delay ~ Exp(b_expo_per_ms), bin frequency
 *                 read as density;
 *   outputs     d_finish_prob[member slot] = P_m           (float)
 *               d_expected_finish[cand]   = sum_m P_m      (double)
 *               d_expected_latency_ms[cand] = E[L_B]       (float)
 *               d_score[cand]             = sum_m p_m      (float)
 * d_ccdf is the [M][n_bs][C][K] table of orloj_build_cdfs, and d_support
 * (optional) the support it wrote for that same table: with it, table
 * entries known to be exactly 0 or 1 are not read (the results are the same
 * bits either way); NULL reads every entry.  A d_support that does not
 * belong to d_ccdf gives wrong results.  d_cand_off /
 * d_prob_off are device copies of orloj_output_sizes' offsets.  Output
 * buffers hold at least n_cands / n_probs elements.  b_expo_per_ms must be
 * finite and > 0 (the paper uses 1e-4 per ms, §4.4).
 * ORLOJ_E_UNSUPPORTED when a prefix would exceed ORLOJ_MAX_PREFIX.
 */
int orloj_score_candidates(orloj_ctx *ctx, const orloj_grid *grid, const float *d_ccdf,
                           const int32_t *d_support, const orloj_queues *queues, double b_expo_per_ms,
                           int32_t prefix_mode, const int64_t *d_cand_off,
                           const int64_t *d_prob_off, float *d_finish_prob,
                           double *d_expected_finish, float *d_expected_latency_ms,
                           float *d_score);

/*
 * Affine batch-latency mode (§4.2.1 Eq. (3) and (5), §4.2.2 Eq. (9)): a
 * batch of size s whose slowest member takes l runs for c0 + c1 s l, with
 * per-model constants c0 = d_c0_ms[q] (ms, finite, >= 0) and
 * c1 = d_c1[q] (finite, > 0), so one latency histogram per class, of a
 * request run alone, serves every batch size.  d_ccdf is orloj_build_cdfs'
 * table of those histograms, [M][C][K] (no batch-size dimension), and
 * d_support (optional) its support, [M][C][2].  For candidate (q, b, n):
 *   G(x_k)  = prod_i F_{c_i}(x_k) on the base grid (the members' max X);
 *   L_B     = c0 + c1 s_b X: its histogram holds G's bin masses on bins
 *             [c0 + c1 s_b k w, c0 + c1 s_b (k+1) w), linear inside a bin
 *             (Eq. (9) with the Jacobian 1 / (c1 s_b));
 *   E[L_B]  = c0 + c1 s_b E[X]                                  (Eq. (5));
 *   P_m, p_m as in orloj_score_candidates on that histogram: the time left
 *             tau_m - c0 on bins c1 s_b w wide.
 * Outputs, their layout and every other argument are those of
 * orloj_score_candidates; orloj_select_batch applies unchanged.  A
 * negative or non-finite c0, or a c1 that is not finite and > 0, is a data
 * error (orloj_sync); that model's requests then score as dead.
 * The sums of 1 - G behind E[X] do not depend on the batch size, so they
 * are formed once per (model, prefix length) into a scratch block the
 * context owns (M x ceil(K / 256) x the longest prefix floats).  The
 * first call that needs a larger block waits for the context's
 * stream, frees the old block and allocates the new one (ORLOJ_E_NOMEM if
 * that fails); the block is reused by later calls and freed by
 * orloj_destroy.  Calls on one context are ordered by its stream.
 */
int orloj_score_candidates_affine(orloj_ctx *ctx, const orloj_grid *grid, const float *d_ccdf,
                                  const int32_t *d_support, const double *d_c0_ms,
                                  const double *d_c1, const orloj_queues *queues,
                                  double b_expo_per_ms, int32_t prefix_mode,
                                  const int64_t *d_cand_off, const int64_t *d_prob_off,
                                  float *d_finish_prob, double *d_expected_finish,
                                  float *d_expected_latency_ms, float *d_score);

/*
 * orloj_score_candidates_affine without any allocation, for callers that
 * cannot allocate device memory: code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc.  Arguments, outputs and
 * errors are those of orloj_score_candidates_affine, with the same kernels
 * and the same bits; the per-(model, panel, prefix length) sums behind E[X]
 * go to a fixed device array of ORLOJ_NOALLOC_SCRATCH_FLOATS floats instead
 * of the context's grown block.  The library looks up that array's address
 * on a device once (the first orloj_create on it) and each device keeps
 * its array until the process ends.  A call needing more than
 * M x ceil(K / 256) x (the longest prefix) floats of it returns
 * ORLOJ_E_UNSUPPORTED before any launch (128 models of 4096 bins with
 * prefixes up to 64 need 128 x 16 x 64 = 131 072).  ORLOJ_E_HIP if the array is unavailable on the context's
 * device.  Every entry a call reads is written earlier in the same call, so
 * nothing needs clearing; but all calls on one device share the one array,
 * so calls that may overlap on a device (other contexts, other streams,
 * other threads) race and must be ordered by the caller.  The call itself
 * makes no hipMalloc, hipFree or host-synchronising call.
 */
int orloj_score_candidates_affine_noalloc(orloj_ctx *ctx, const orloj_grid *grid,
                                          const float *d_ccdf, const int32_t *d_support,
                                          const double *d_c0_ms, const double *d_c1,
                                          const orloj_queues *queues, double b_expo_per_ms,
                                          int32_t prefix_mode, const int64_t *d_cand_off,
                                          const int64_t *d_prob_off, float *d_finish_prob,
                                          double *d_expected_finish,
                                          float *d_expected_latency_ms, float *d_score);

/*
 * Pick one batch per model (the scheduler pops the top batch, §3.2
 * Algorithm 1): the candidate with the largest score among n <= batch size;
 * exact ties go to the larger n, then the smaller batch size.  When the
 * best score is <= 0 (or the queue is empty) there is no batch:
 * d_sel_n[q] = 0, d_sel_bs[q] = 0, d_sel_score[q] = 0.
 * Outputs are device [M].
 */
int orloj_select_batch(orloj_ctx *ctx, const orloj_grid *grid, const orloj_queues *queues,
                       int32_t prefix_mode, const int64_t *d_cand_off, const float *d_score,
                       int32_t *d_sel_n, int32_t *d_sel_bs, float *d_sel_score);

/*
 * The scheduler iteration of §3.2 Algorithm 1 with the paper's own
 * per-request priority (§4.1 Eq. (1)-(2), §4.2, §4.3), data-parallel over
 * every model's queue.  Two calls:
 *
 * orloj_build_model_laws (off the scheduling path; rebuild when the
 * histograms, the class mix or b_expo change).  When a request's priority
 * is computed, the batch it will run in is not yet known (§4.3), so its
 * batch latency at batch size s is taken as the max of its own latency and
 * s - 1 others drawn independently from the model's class mix
 *   F_mix,s = sum_c pi_c F_{c,s}   (pi = d_class_weights[q][c] normalised;
 *                                    NULL = uniform over the classes),
 * and the expected batch latency in the priority is the model-wide one of
 * F_mix,s^s (§4.2.1: the max of k identical variables has CDF F^k).  For
 * every model q, batch-size index b and class c, at the right edge of bin k:
 *   d_law[q][b][c][k]  = F_{c,b}(x_{k+1}) * F_mix,b(x_{k+1})^(s_b - 1)
 *   d_disc[q][b][c][k] = sum_{i<=k} d_law[q][b][c][i] * d^(k-i),
 *                        d = exp(-b_expo_per_ms * w_q)
 *   d_model_el[q][b]   = E[L] of F_mix,b^(s_b), Eq. (5)       (ms)
 * d_ccdf is orloj_build_cdfs' [M][n_bs][C][K] table; d_law and d_disc have
 * its shape (float32), d_model_el is [M][n_bs] float32.  Negative, infinite
 * or all-zero weights of a model are a data error (orloj_sync).
 *
 * orloj_iterate: one iteration for every model in one launch.  For model q
 * at time now_q, with tau_r = D_r - now_q:
 *   drop phase   r is kept at batch size s iff it could finish by its
 *                deadline run alone at s: F_{c_r,s}(tau_r) > 0, i.e. tau_r is
 *                past the left edge of the first bin with mass (read from
 *                d_support, orloj_build_cdfs' support of the same table).
 *                A request kept at no batch size is timed out.
 *   candidate    batch sizes in (D_{Q_s}, s) descending order, D_{Q_s} the
 *                earliest deadline kept at s; the first whose kept set holds
 *                at least s requests (none: no batch).
 *   PopBatch     the s kept requests with the largest priority at the
 *                candidate size; equal priorities go to the earlier queue
 *                position.
 * Outputs: d_timed_out[N] int32 (1 = timed out), d_score[N] float32 (the
 * priority at the candidate size for requests kept there, else 0),
 * d_cand_bs[M] int32 (0 = no batch), d_batch[M][s_max] int32 (positions in
 * the model's queue, highest priority first, then -1), s_max the largest
 * batch size.  b_expo_per_ms must be the value the laws were built with.
 * ORLOJ_E_UNSUPPORTED for a queue longer than 4096 requests or a batch size
 * above 1024.  Queue data errors are reported by orloj_sync as for
 * orloj_score_candidates.  A queue longer than 1024 requests, when there are
 * few enough models (4 M <= the GPU's compute units), has its drop phase run
 * in parts of 256 requests: the per-part counts (M x parts x |S| x 8 bytes)
 * go to the context's scratch block, grown on demand as for the affine
 * scorer (ORLOJ_E_NOMEM if that fails).  d_support entries are taken to lie
 * in [0, K), as orloj_build_cdfs writes them.
 */
/*
 * Piecewise-step cost functions (App. B) for orloj_iterate: request r's cost
 * rises to d_step_cost[j] when it finishes after d_step_deadline_ms[j], for
 * j in [d_step_off[r], d_step_off[r+1]) (r indexes the whole queue array,
 * all models back to back; deadlines increasing, costs non-decreasing and
 * >= 0, at least one step per request).  Such a function is the sum of
 * single steps at each d_j with cost d_step_cost[j] - d_step_cost[j-1], so
 * the request's priority is the matching sum of single-step priorities,
 * times its d_cost.  The drop phase uses the last step's deadline (the
 * request still has cost to save until then); queue order and D_{Q_s} use
 * d_deadline_ms.  Malformed steps are a data error (the request then scores
 * 0).  h_step_off is the host copy of the offsets (validated on the host).
 */
typedef struct orloj_steps {
    const int64_t *h_step_off;      /* host [N+1] */
    const int64_t *d_step_off;      /* device copy */
    const double *d_step_deadline_ms;
    const double *d_step_cost;
} orloj_steps;

int orloj_build_model_laws(orloj_ctx *ctx, const orloj_grid *grid, const float *d_ccdf,
                           const double *d_class_weights, double b_expo_per_ms,
                           float *d_law, float *d_disc, float *d_model_el);

int orloj_iterate(orloj_ctx *ctx, const orloj_grid *grid, const int32_t *d_support,
                  const float *d_law, const float *d_disc, const float *d_model_el,
                  const orloj_queues *queues, const orloj_steps *steps,
                  double b_expo_per_ms, int32_t *d_timed_out, float *d_score,
                  int32_t *d_cand_bs, int32_t *d_batch);

/*
 * Profiler feedback (§3.2 "Long-Term Feedback Loop"): add n_samples solo
 * execution times of sampled finished requests to the histograms.  Sample i
 * adds one count to d_counts[d_model[i]][d_bs_index[i]][d_class[i]][k],
 * k = floor(d_latency_ms[i] / w_q), a latency at or beyond the grid counting
 * in the last bin.  Samples with an index out of range or a negative or
 * non-finite latency are skipped and counted in *d_n_rejected (device,
 * optional, added to).  Atomic updates: concurrent calls on the same counts
 * add up.  A profiling window is reset by zeroing d_counts; the CDF tables
 * are rebuilt from the counts with orloj_build_cdfs.
 */
int orloj_accumulate(orloj_ctx *ctx, const orloj_grid *grid, int64_t n_samples,
                     const int32_t *d_model, const int32_t *d_bs_index, const int32_t *d_class,
                     const double *d_latency_ms, uint32_t *d_counts,
                     unsigned long long *d_n_rejected);

/*
 * Host scheduling runtime around the scorer (§3.1: one worker per model
 * runs one batch at a time; §3.2 Algorithm 1: drop the requests that can no
 * longer finish, then pick the next batch).  It keeps one queue of pending
 * requests per model in deadline order and makes a decision round per call
 * to orloj_sched_decide: for every idle model it drops the requests that can
 * no longer finish, stages the model's first s_max requests (s_max = the
 * largest batch size: no longer prefix is a candidate), uploads every idle
 * model's queue in one copy from pinned memory, scores and selects (the
 * outputs of orloj_score_candidates and orloj_select_batch, TRIANGLE
 * prefixes, bit for bit; in a round small enough to take its E sums from a
 * pre-pass, that pre-pass shares the score launch and the selection kernel
 * finishes E[L_B] and the scores), reads the selections back and removes
 * the selected members from their queues.
 *
 * orloj_sched_create copies the grid (its d_bin_width_ms must stay valid)
 * and keeps d_ccdf / d_support (orloj_build_cdfs' table of the model's
 * per-batch-size histograms and its support, NULL = none; both stay owned by
 * the caller and must outlive the runtime).  h_drop_ms [M][C] (copied): a
 * request of class c at model q is dropped once its time left
 * (deadline - now) is <= h_drop_ms[q][c], e.g. the smallest latency its
 * class can take run alone.  The runtime allocates pinned host and device
 * buffers for M * s_max requests and the outputs of a full round; it uses
 * the context's stream and device.  Not thread-safe.
 *
 * orloj_sched_admit inserts n requests (model, class, finite deadline) into
 * their queues; equal deadlines keep admission order.  A bad model, class or
 * deadline rejects the whole call (ORLOJ_E_INVALID) before any insertion.
 *
 * orloj_sched_decide runs one round at time now_ms.  h_idle [M] (NULL = all)
 * marks the models whose worker is free; the others are neither dropped nor
 * scored.  Outputs (host): h_sel_n[M], h_sel_bs[M] (0, 0 = no batch);
 * *h_n_dropped (optional) is incremented by the requests dropped; the
 * removed members in queue order, model by model, in h_batch_off[M+1],
 * h_batch_class[], h_batch_deadline[] (optional, room for M * s_max).  The
 * call returns after the selections are on the host: the selection kernel
 * flags each of its workgroups into pinned host memory once its writes are
 * visible there, and the call spins on those flags (after 5 ms without them
 * it synchronises the context's stream, which reports launch errors); work
 * of the round may still be retiring on the stream when it returns.  Data
 * errors of the scoring kernels are reported by the next orloj_sync.
 *
 * orloj_sched_queue_length: pending requests of a model (-1 if out of range).
 */
typedef struct orloj_sched orloj_sched;

int orloj_sched_create(orloj_sched **out, orloj_ctx *ctx, const orloj_grid *grid,
                       const float *d_ccdf, const int32_t *d_support, const double *h_drop_ms,
                       double b_expo_per_ms);
void orloj_sched_destroy(orloj_sched *s);
int orloj_sched_admit(orloj_sched *s, int64_t n, const int32_t *h_model, const int32_t *h_class,
                      const double *h_deadline_ms);
int orloj_sched_decide(orloj_sched *s, double now_ms, const uint8_t *h_idle, int32_t *h_sel_n,
                       int32_t *h_sel_bs, int64_t *h_n_dropped, int64_t *h_batch_off,
                       int32_t *h_batch_class, double *h_batch_deadline);
int64_t orloj_sched_queue_length(const orloj_sched *s, int32_t model);

/*
 * Trace-driven run of the runtime: one worker per model, one batch at a time
 * (§3.1), a decision round every tick_ms of simulated time.  Each tick admits
 * the trace's arrivals released by then (h_release_ms sorted), and, if some
 * idle model has pending requests, runs orloj_sched_decide over the idle
 * models.  A selected batch of batch-size index b keeps its worker busy for
 * h_bs_scale[b] x the max of its members' latencies, each drawn from its
 * class's solo-latency histogram h_solo_counts [M][C][K] (a bin with
 * probability proportional to its count, then uniform inside it, bins
 * h_bin_width_ms[q] wide) with a splitmix64 stream seeded by `seed`.  A
 * member finishing at or before its deadline is on time.  The run ends when
 * the trace is exhausted and every queue is empty, or after max_ticks ticks
 * (> 0).  Statistics go to *out; rec (optional) records every every-th
 * decision's state (the scored queue, the time and the selection), up to
 * `limit` of them, into caller buffers: h_off [limit+1] and h_class /
 * h_deadline_ms with room for limit * s_max entries.
 */
typedef struct orloj_trace {
    int64_t n;
    const double *h_release_ms;
    const int32_t *h_model;
    const int32_t *h_class;
    const double *h_deadline_ms;
} orloj_trace;

typedef struct orloj_sim_stats {
    int64_t ticks, launches, decisions, dispatched, dropped, on_time, late, arrivals;
    double sim_ms;      /* simulated time */
    double wall_s;      /* host wall time of the whole run */
    double device_s;    /* upload + score + select + download of the rounds */
} orloj_sim_stats;

typedef struct orloj_sim_record {
    int32_t every, limit;
    int32_t n;                                  /* out: states recorded */
    int32_t *h_model;
    double *h_now_ms;
    int32_t *h_sel_n, *h_sel_bs;
    int64_t *h_off;
    int32_t *h_class;
    double *h_deadline_ms;
} orloj_sim_record;

int orloj_simulate_trace(orloj_sched *s, const orloj_trace *trace, double tick_ms,
                         const uint32_t *h_solo_counts, const double *h_bin_width_ms,
                         const double *h_bs_scale, uint64_t seed, int64_t max_ticks,
                         orloj_sim_record *rec, orloj_sim_stats *out);

#ifdef __cplusplus
}
#endif

#endif /* ORLOJ_H */
