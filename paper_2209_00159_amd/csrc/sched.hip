// Host scheduling runtime around the scorer (C ABI in include/orloj.h):
//
//   orloj_sched_*          per-model queues of pending requests kept in
//                          deadline order (§3.1: deadline = release + SLO),
//                          the drop of requests that can no longer finish
//                          (§3.2 Algorithm 1), and one decision round per
//                          call: every idle model's queue is staged in
//                          pinned memory, uploaded in one copy, scored and
//                          a batch selected per model (the outputs of
//                          orloj_score_candidates + orloj_select_batch, the
//                          E pre-pass sharing the score launch), the
//                          selections read back,
//                          and the chosen members popped;
//   orloj_simulate_trace   a trace-driven run of one worker per model on top
//                          of it (one batch at a time, §3.1): the arrivals
//                          of a trace, a decision round every tick, batch
//                          latencies sampled from the members' histograms.
//
// Host code only; every scoring step runs in the library's kernels.

#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <chrono>
#include <deque>
#include <new>
#include <vector>

#include "../../include/orloj.h"
#include "orloj_ctx.h"

namespace {

struct Req {
    double deadline;
    int32_t cls;
};

constexpr size_t align8(size_t x) { return (x + 7) & ~(size_t)7; }

int hip_err(orloj_ctx* ctx, hipError_t e, const char* what) {
    return orloj_ctx_fail(ctx, e == hipErrorOutOfMemory ? ORLOJ_E_NOMEM : ORLOJ_E_HIP, "%s: %s",
                          what, hipGetErrorString(e));
}

}  // namespace

struct orloj_sched {
    orloj_ctx* ctx;
    orloj_grid grid;               // batch_sizes points into bs
    std::vector<int32_t> bs;
    const float* d_ccdf;
    const int32_t* d_support;
    std::vector<double> drop;      // [M][C] drop threshold (ms)
    double b;
    int M, C, smax;
    std::vector<std::deque<Req>> queue;

    // Staging block, laid out alike on host (pinned) and device:
    //   off[M+1] i64 | cand_off[M+1] i64 | prob_off[M+1] i64 | now[M] f64 |
    //   deadline[n] f64 | class[n] i32          (n = requests staged)
    size_t fixed;                  // bytes before the deadlines
    size_t stage_bytes;
    unsigned char* h_stage = nullptr;
    unsigned char* d_stage = nullptr;
    int64_t staged = 0;            // n of the last round
    std::vector<int32_t> cls_stage;  // classes of a round, before they are packed after the deadlines

    float* d_P = nullptr;
    double* d_E = nullptr;
    float* d_EL = nullptr;
    float* d_S = nullptr;
    int32_t* h_sel = nullptr;      // pinned, mapped [3M]: n, batch size, score bits
    int32_t* d_sel = nullptr;      // the device's address of h_sel
    int32_t* h_done = nullptr;     // pinned, mapped: select workgroup g writes the round number
    int32_t* d_done = nullptr;
    int32_t round = 0;
    double device_s = 0.0;         // time spent in upload + launches + download

    int64_t* off() { return reinterpret_cast<int64_t*>(h_stage); }
    int64_t* cand_off() { return off() + (M + 1); }
    int64_t* prob_off() { return cand_off() + (M + 1); }
    double* now_ms() { return reinterpret_cast<double*>(prob_off() + (M + 1)); }
    double* deadline() { return reinterpret_cast<double*>(h_stage + fixed); }
    int32_t* cls(int64_t n) { return reinterpret_cast<int32_t*>(h_stage + fixed + 8 * (size_t)n); }
};

namespace {

void sched_free(orloj_sched* s) {
    if (!s) return;
    if (s->ctx) (void)hipSetDevice(s->ctx->device);
    if (s->h_stage) (void)hipHostFree(s->h_stage);
    if (s->h_sel) (void)hipHostFree(s->h_sel);
    if (s->h_done) (void)hipHostFree(s->h_done);
    for (void* p : {(void*)s->d_stage, (void*)s->d_P, (void*)s->d_E, (void*)s->d_EL,
                    (void*)s->d_S})
        if (p) (void)hipFree(p);
    delete s;
}

// One decision round (see orloj_sched_decide).
int decide(orloj_sched* s, double now, const uint8_t* idle, int32_t* sel_n, int32_t* sel_bs,
           int64_t* n_dropped, int64_t* batch_off, int32_t* batch_class, double* batch_deadline) {
    orloj_ctx* ctx = s->ctx;
    const int M = s->M;
    int64_t* off = s->off();
    double* dl = s->deadline();
    int64_t n = 0, dropped = 0;
    off[0] = 0;
    // drop, then stage each idle model's first smax requests: no longer
    // prefix is a candidate at any batch size
    std::vector<int32_t>& cls_tmp = s->cls_stage;
    cls_tmp.clear();
    for (int q = 0; q < M; ++q) {
        if (!idle || idle[q]) {
            std::deque<Req>& Q = s->queue[q];
            const double* thr = s->drop.data() + (size_t)q * s->C;
            const size_t before = Q.size();
            Q.erase(std::remove_if(Q.begin(), Q.end(),
                                   [&](const Req& r) { return !(r.deadline - now > thr[r.cls]); }),
                    Q.end());
            dropped += (int64_t)(before - Q.size());
            const int64_t m = std::min<int64_t>((int64_t)Q.size(), s->smax);
            for (int64_t i = 0; i < m; ++i) {
                dl[n + i] = Q[(size_t)i].deadline;
                cls_tmp.push_back(Q[(size_t)i].cls);
            }
            n += m;
        }
        off[q + 1] = n;
    }
    if (n_dropped) *n_dropped += dropped;
    s->staged = n;
    if (n > 0) memcpy(s->cls(n), cls_tmp.data(), sizeof(int32_t) * (size_t)n);
    for (int q = 0; q < M; ++q) s->now_ms()[q] = now;

    for (int q = 0; q < M; ++q) sel_n[q] = sel_bs[q] = 0;
    if (n > 0) {
        const auto t0 = std::chrono::steady_clock::now();
        orloj_queues hq;
        memset(&hq, 0, sizeof hq);
        hq.h_queue_off = off;
        int64_t nc = 0, np = 0;
        int rc = orloj_output_sizes(&s->grid, &hq, ORLOJ_PREFIX_TRIANGLE, &nc, &np, s->cand_off(),
                                    s->prob_off());
        if (rc) return orloj_ctx_fail(ctx, rc, "orloj_sched_decide: sizing the outputs failed");
        hipError_t e = hipSetDevice(ctx->device);
        if (e != hipSuccess) return hip_err(ctx, e, "orloj_sched_decide: hipSetDevice");
        // Once the upload is enqueued, every return waits for the stream
        // first: the copy reads the pinned staging block, which the next
        // round rewrites.
        auto drained = [&](int code) {
            (void)hipStreamSynchronize(ctx->stream);
            return code;
        };
        e = hipMemcpyAsync(s->d_stage, s->h_stage, s->fixed + 12 * (size_t)n,
                           hipMemcpyHostToDevice, ctx->stream);
        if (e != hipSuccess)
            return drained(hip_err(ctx, e, "orloj_sched_decide: uploading the queues"));
        const size_t o1 = 8 * (size_t)(M + 1);
        orloj_queues dq;
        dq.h_queue_off = off;
        dq.d_queue_off = reinterpret_cast<const int64_t*>(s->d_stage);
        dq.d_now_ms = reinterpret_cast<const double*>(s->d_stage + 3 * o1);
        dq.d_deadline_ms = reinterpret_cast<const double*>(s->d_stage + s->fixed);
        dq.d_class = reinterpret_cast<const int32_t*>(s->d_stage + s->fixed + 8 * (size_t)n);
        dq.d_cost = nullptr;
        const int64_t* d_coff = reinterpret_cast<const int64_t*>(s->d_stage + o1);
        const int64_t* d_poff = reinterpret_cast<const int64_t*>(s->d_stage + 2 * o1);
        // scoring and selection: the outputs of orloj_score_candidates and
        // orloj_select_batch, with the E pre-pass and the score waves of a
        // small round in one launch
        const int32_t round = ++s->round;
        int groups = 0;
        rc = orloj_internal_score_select(ctx, &s->grid, s->d_ccdf, s->d_support, &dq, s->b, d_coff,
                                         d_poff, s->d_P, s->d_E, s->d_EL, s->d_S, s->d_sel,
                                         s->d_sel + M, reinterpret_cast<float*>(s->d_sel + 2 * M),
                                         s->d_done, round, &groups);
        if (rc) return drained(rc);
        // the select kernel writes the selections straight into mapped host
        // memory and then, per workgroup, the round's number: the host spins
        // on those (the stream's completion signal comes later); after 5 ms
        // without them (a failed launch) it waits for the stream, which
        // reports the error
        bool seen = false;
        {
            const auto t1 = std::chrono::steady_clock::now();
            for (;;) {
                bool all = true;
                for (int g = 0; g < groups && all; ++g)
                    all = __atomic_load_n(&s->h_done[g], __ATOMIC_ACQUIRE) == round;
                if (all) { seen = true; break; }
                if (std::chrono::steady_clock::now() - t1 > std::chrono::milliseconds(5)) break;
            }
        }
        if (!seen) {
            e = hipStreamSynchronize(ctx->stream);
            if (e != hipSuccess) return hip_err(ctx, e, "orloj_sched_decide: reading the selections");
        }
        s->device_s += std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
        for (int q = 0; q < M; ++q) {
            sel_n[q] = s->h_sel[q];
            sel_bs[q] = s->h_sel[M + q];
        }
    }
    // pop the selected members (the front of the queue: the scored prefix)
    int64_t nb = 0;
    if (batch_off) batch_off[0] = 0;
    for (int q = 0; q < M; ++q) {
        const int k = sel_n[q];
        std::deque<Req>& Q = s->queue[q];
        if (k < 0 || (size_t)k > Q.size())
            return orloj_ctx_fail(ctx, ORLOJ_E_DATA, "orloj_sched_decide: selection out of range");
        for (int i = 0; i < k; ++i) {
            if (batch_class) batch_class[nb + i] = Q[(size_t)i].cls;
            if (batch_deadline) batch_deadline[nb + i] = Q[(size_t)i].deadline;
        }
        Q.erase(Q.begin(), Q.begin() + k);
        nb += k;
        if (batch_off) batch_off[q + 1] = nb;
    }
    return ORLOJ_OK;
}

// splitmix64: a small counter-based generator for the simulated latencies
struct Rng {
    uint64_t x;
    uint64_t next() {
        uint64_t z = (x += 0x9e3779b97f4a7c15ull);
        z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
        z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
        return z ^ (z >> 31);
    }
    uint64_t below(uint64_t n) { return (uint64_t)(((unsigned __int128)next() * n) >> 64); }
    double unit() { return (double)(next() >> 11) * 0x1.0p-53; }
};

}  // namespace

extern "C" {

int orloj_sched_create(orloj_sched** out, orloj_ctx* ctx, const orloj_grid* grid,
                       const float* d_ccdf, const int32_t* d_support, const double* h_drop_ms,
                       double b_expo_per_ms) {
    if (!out) return ORLOJ_E_INVALID;
    *out = nullptr;
    if (!ctx) return ORLOJ_E_INVALID;
    if (!grid || grid->n_models < 1 || grid->n_classes < 1 || grid->n_bins < 1 || grid->n_bs < 1 ||
        !grid->batch_sizes || !grid->d_bin_width_ms)
        return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "orloj_sched_create: bad grid");
    if (!d_ccdf || !h_drop_ms)
        return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "orloj_sched_create: NULL table or drop thresholds");
    if (!(b_expo_per_ms > 0.0) || !isfinite(b_expo_per_ms))
        return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "orloj_sched_create: b_expo_per_ms");
    for (int i = 0; i < grid->n_bs; ++i)
        if (grid->batch_sizes[i] < 1 || (i > 0 && grid->batch_sizes[i] <= grid->batch_sizes[i - 1]))
            return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "orloj_sched_create: batch sizes");
    const int smax = grid->batch_sizes[grid->n_bs - 1];
    if (smax > ORLOJ_MAX_PREFIX)
        return orloj_ctx_fail(ctx, ORLOJ_E_UNSUPPORTED, "orloj_sched_create: batch size %d > %d",
                              smax, ORLOJ_MAX_PREFIX);
    orloj_sched* s = new (std::nothrow) orloj_sched;
    if (!s) return ORLOJ_E_NOMEM;
    s->ctx = ctx;
    s->M = grid->n_models;
    s->C = grid->n_classes;
    s->smax = smax;
    s->bs.assign(grid->batch_sizes, grid->batch_sizes + grid->n_bs);
    s->grid = *grid;
    s->grid.batch_sizes = s->bs.data();
    s->d_ccdf = d_ccdf;
    s->d_support = d_support;
    s->drop.assign(h_drop_ms, h_drop_ms + (size_t)s->M * s->C);
    s->b = b_expo_per_ms;
    s->queue.resize((size_t)s->M);
    s->cls_stage.reserve((size_t)s->M * smax);
    const int M = s->M;
    const size_t cap = (size_t)M * smax;
    s->fixed = align8(3 * 8 * (size_t)(M + 1) + 8 * (size_t)M);
    s->stage_bytes = s->fixed + 12 * cap;
    size_t n_c = 0, n_p = 0;            // outputs of the fullest round
    for (int i = 0; i < grid->n_bs; ++i) {
        const size_t c = (size_t)std::min(grid->batch_sizes[i], smax);
        n_c += c;
        n_p += c * (c + 1) / 2;
    }
    n_c *= M;
    n_p *= M;
    hipError_t e = hipSetDevice(ctx->device);
    if (e == hipSuccess) e = hipHostMalloc((void**)&s->h_stage, s->stage_bytes, hipHostMallocDefault);
    if (e == hipSuccess) e = hipHostMalloc((void**)&s->h_sel, sizeof(int32_t) * 3 * M, hipHostMallocMapped);
    if (e == hipSuccess) e = hipHostGetDevicePointer((void**)&s->d_sel, s->h_sel, 0);
    if (e == hipSuccess) e = hipHostMalloc((void**)&s->h_done, sizeof(int32_t) * (M + 1), hipHostMallocMapped);
    if (e == hipSuccess) e = hipHostGetDevicePointer((void**)&s->d_done, s->h_done, 0);
    if (e == hipSuccess) memset(s->h_done, 0, sizeof(int32_t) * (M + 1));
    if (e == hipSuccess) e = hipMalloc((void**)&s->d_stage, s->stage_bytes);
    if (e == hipSuccess) e = hipMalloc((void**)&s->d_P, sizeof(float) * n_p);
    if (e == hipSuccess) e = hipMalloc((void**)&s->d_E, sizeof(double) * n_c);
    if (e == hipSuccess) e = hipMalloc((void**)&s->d_EL, sizeof(float) * n_c);
    if (e == hipSuccess) e = hipMalloc((void**)&s->d_S, sizeof(float) * n_c);
    if (e != hipSuccess) {
        const int rc = hip_err(ctx, e, "orloj_sched_create");
        sched_free(s);
        return rc;
    }
    *out = s;
    return ORLOJ_OK;
}

void orloj_sched_destroy(orloj_sched* s) {
    if (s && s->ctx) {
        (void)hipSetDevice(s->ctx->device);
        (void)hipStreamSynchronize(s->ctx->stream);
    }
    sched_free(s);
}

int orloj_sched_admit(orloj_sched* s, int64_t n, const int32_t* h_model, const int32_t* h_class,
                      const double* h_deadline_ms) {
    if (!s) return ORLOJ_E_INVALID;
    if (n < 0 || (n > 0 && (!h_model || !h_class || !h_deadline_ms)))
        return orloj_ctx_fail(s->ctx, ORLOJ_E_INVALID, "orloj_sched_admit: bad arguments");
    for (int64_t i = 0; i < n; ++i)
        if (h_model[i] < 0 || h_model[i] >= s->M || h_class[i] < 0 || h_class[i] >= s->C ||
            !isfinite(h_deadline_ms[i]))
            return orloj_ctx_fail(s->ctx, ORLOJ_E_INVALID,
                                  "orloj_sched_admit: request %lld has a bad model, class or deadline",
                                  (long long)i);
    for (int64_t i = 0; i < n; ++i) {
        std::deque<Req>& Q = s->queue[(size_t)h_model[i]];
        const Req r{h_deadline_ms[i], h_class[i]};
        // after every request with an equal deadline: admission order is kept
        auto at = std::upper_bound(Q.begin(), Q.end(), r.deadline,
                                   [](double d, const Req& x) { return d < x.deadline; });
        Q.insert(at, r);
    }
    return ORLOJ_OK;
}

int64_t orloj_sched_queue_length(const orloj_sched* s, int32_t model) {
    if (!s || model < 0 || model >= s->M) return -1;
    return (int64_t)s->queue[(size_t)model].size();
}

int orloj_sched_decide(orloj_sched* s, double now_ms, const uint8_t* h_idle, int32_t* h_sel_n,
                       int32_t* h_sel_bs, int64_t* h_n_dropped, int64_t* h_batch_off,
                       int32_t* h_batch_class, double* h_batch_deadline) {
    if (!s) return ORLOJ_E_INVALID;
    if (!h_sel_n || !h_sel_bs || !isfinite(now_ms))
        return orloj_ctx_fail(s->ctx, ORLOJ_E_INVALID, "orloj_sched_decide: bad arguments");
    return decide(s, now_ms, h_idle, h_sel_n, h_sel_bs, h_n_dropped, h_batch_off, h_batch_class,
                  h_batch_deadline);
}

int orloj_simulate_trace(orloj_sched* s, const orloj_trace* trace, double tick_ms,
                         const uint32_t* h_solo_counts, const double* h_bin_width_ms,
                         const double* h_bs_scale, uint64_t seed, int64_t max_ticks,
                         orloj_sim_record* rec, orloj_sim_stats* out) {
    if (!s) return ORLOJ_E_INVALID;
    orloj_ctx* ctx = s->ctx;
    if (!trace || !out || !h_solo_counts || !h_bin_width_ms || !h_bs_scale || !(tick_ms > 0.0) ||
        !isfinite(tick_ms) || trace->n < 0 ||
        (trace->n > 0 && (!trace->h_release_ms || !trace->h_model || !trace->h_class ||
                          !trace->h_deadline_ms)))
        return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "orloj_simulate_trace: bad arguments");
    if (rec && rec->every > 0 && rec->limit > 0 &&
        (!rec->h_model || !rec->h_now_ms || !rec->h_sel_n || !rec->h_sel_bs || !rec->h_off ||
         !rec->h_class || !rec->h_deadline_ms))
        return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "orloj_simulate_trace: record buffers");
    const int M = s->M, C = s->C, K = s->grid.n_bins;
    for (int64_t i = 1; i < trace->n; ++i)
        if (!(trace->h_release_ms[i] >= trace->h_release_ms[i - 1]))
            return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "orloj_simulate_trace: releases not sorted");
    // cumulative solo histograms for sampling member latencies, and for
    // each row a guide of kGuide buckets of the draw u: guide[g] is the bin
    // that the draw ceil(g T / kGuide) falls in (T the row's total), so the
    // bin of a draw in bucket g lies in [guide[g], guide[g + 1]].  The search
    // then touches one or two cache lines of the row instead of a dozen
    // (the rows of all models and classes are far larger than the caches).
    constexpr int kGuide = 256;
    std::vector<uint64_t> cum;
    std::vector<uint32_t> guide;
    try {
        cum.resize((size_t)M * C * K);
        guide.resize((size_t)M * C * (kGuide + 1));
    } catch (...) {
        return orloj_ctx_fail(ctx, ORLOJ_E_NOMEM, "orloj_simulate_trace: sampling tables");
    }
    for (size_t r = 0; r < (size_t)M * C; ++r) {
        uint64_t acc = 0;
        uint64_t* row = cum.data() + r * K;
        for (int k = 0; k < K; ++k) row[k] = (acc += h_solo_counts[r * K + k]);
        if (acc == 0)
            return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "orloj_simulate_trace: empty solo histogram");
        uint32_t* gd = guide.data() + r * (kGuide + 1);
        for (int g = 0; g <= kGuide; ++g) {
            const uint64_t ulo = (uint64_t)(((unsigned __int128)g * acc + kGuide - 1) / kGuide);
            gd[g] = (uint32_t)(std::upper_bound(row, row + K, ulo) - row);
        }
    }
    Rng rng{seed};
    auto sample = [&](int q, int c) {
        const size_t r = (size_t)q * C + c;
        const uint64_t* row = cum.data() + r * K;
        const uint64_t tot = row[K - 1];
        const uint64_t u = rng.below(tot);
        // the first bin whose cumulative count exceeds u (std::upper_bound
        // over the whole row gives the same bin)
        const int g = (int)(((unsigned __int128)u * kGuide) / tot);
        const uint32_t* gd = guide.data() + r * (kGuide + 1);
        const int lo = (int)gd[g], hi = std::min((int)gd[g + 1] + 1, K);
        const int k = (int)(std::upper_bound(row + lo, row + hi, u) - row);
        return ((double)k + rng.unit()) * h_bin_width_ms[q];
    };

    orloj_sim_stats st;
    memset(&st, 0, sizeof st);
    if (rec) rec->n = 0;
    std::vector<double> busy_until((size_t)M, -INFINITY);
    std::vector<uint8_t> idle((size_t)M);
    std::vector<int32_t> sel_n((size_t)M), sel_bs((size_t)M);
    std::vector<int64_t> boff((size_t)M + 1);
    std::vector<int32_t> bcls((size_t)M * s->smax);
    std::vector<double> bdl((size_t)M * s->smax);
    const double dev0 = s->device_s;
    const auto w0 = std::chrono::steady_clock::now();
    int64_t i_next = 0;
    int64_t pending = 0;
    for (int q = 0; q < M; ++q) pending += (int64_t)s->queue[(size_t)q].size();
    double t = trace->n > 0 ? trace->h_release_ms[0] : 0.0;
    while (true) {
        if (max_ticks > 0 && st.ticks >= max_ticks) break;
        if (i_next >= trace->n && pending == 0) break;
        // admit the arrivals released by now
        int64_t j = i_next;
        while (j < trace->n && trace->h_release_ms[j] <= t) ++j;
        if (j > i_next) {
            int rc = orloj_sched_admit(s, j - i_next, trace->h_model + i_next, trace->h_class + i_next,
                                       trace->h_deadline_ms + i_next);
            if (rc) return rc;
            pending += j - i_next;
            i_next = j;
        }
        bool any_idle = false;
        for (int q = 0; q < M; ++q) {
            idle[(size_t)q] = busy_until[(size_t)q] <= t;
            any_idle = any_idle || (idle[(size_t)q] && !s->queue[(size_t)q].empty());
        }
        if (any_idle) {
            int64_t dropped = 0;
            int rc = decide(s, t, idle.data(), sel_n.data(), sel_bs.data(), &dropped, boff.data(),
                            bcls.data(), bdl.data());
            if (rc) return rc;
            st.dropped += dropped;
            pending -= dropped;
            if (s->staged > 0) ++st.launches;
            const int64_t* off = s->off();
            for (int q = 0; q < M; ++q) {
                const int k = sel_n[(size_t)q];
                if (k == 0) continue;
                if (rec && rec->every > 0 && st.decisions % rec->every == 0 && rec->n < rec->limit) {
                    const int r = rec->n++;
                    rec->h_model[r] = q;
                    rec->h_now_ms[r] = t;
                    rec->h_sel_n[r] = k;
                    rec->h_sel_bs[r] = sel_bs[(size_t)q];
                    if (r == 0) rec->h_off[0] = 0;
                    const int64_t a = off[q], b = off[q + 1];
                    for (int64_t i = a; i < b; ++i) {
                        rec->h_class[rec->h_off[r] + (i - a)] = s->cls(s->staged)[i];
                        rec->h_deadline_ms[rec->h_off[r] + (i - a)] = s->deadline()[i];
                    }
                    rec->h_off[r + 1] = rec->h_off[r] + (b - a);
                }
                const int bi = (int)(std::lower_bound(s->bs.begin(), s->bs.end(), sel_bs[(size_t)q]) -
                                     s->bs.begin());
                double lat = 0.0;
                for (int64_t i = boff[(size_t)q]; i < boff[(size_t)q + 1]; ++i)
                    lat = std::max(lat, sample(q, bcls[(size_t)i]));
                const double done = t + lat * h_bs_scale[bi];
                for (int64_t i = boff[(size_t)q]; i < boff[(size_t)q + 1]; ++i) {
                    if (bdl[(size_t)i] >= done) ++st.on_time;
                    else ++st.late;
                }
                busy_until[(size_t)q] = done;
                ++st.decisions;
                st.dispatched += k;
                pending -= k;
            }
        }
        ++st.ticks;
        st.sim_ms += tick_ms;
        t += tick_ms;
    }
    st.wall_s = std::chrono::duration<double>(std::chrono::steady_clock::now() - w0).count();
    st.device_s = s->device_s - dev0;
    st.arrivals = i_next;
    *out = st;
    return ORLOJ_OK;
}

}  // extern "C"
