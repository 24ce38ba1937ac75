// Internal to the library: the context every entry point takes, shared by
// its translation units (orloj.hip: kernels and scoring entry points;
// sched.hip: the host scheduling runtime).  Not part of the C ABI.
#ifndef ORLOJ_CTX_INTERNAL_H
#define ORLOJ_CTX_INTERNAL_H

#include <hip/hip_runtime_api.h>
#include <stdarg.h>
#include <stdio.h>

#include "../../include/orloj.h"

struct orloj_ctx {
    int device;
    int n_cu;        // compute units of the device
    int chunk_pref;  // prefix steps per score workgroup: -1 automatic, 0 all
    hipStream_t stream;
    int* d_err;      // device status word (data error bits)
    float* d_fill;   // stand-in table entries: 16 zeros, 16 ones
    void* d_work;    // scratch of the affine scorer (grown on demand), or NULL
    size_t work_bytes;
    float* noalloc_scratch;   // this device's fixed scratch array (NULL: unavailable)
    hipError_t noalloc_err;   // why it is unavailable
    char msg[512];
};

// Record a failure message on the context and return `code`.
static inline int orloj_ctx_fail(orloj_ctx* ctx, int code, const char* fmt, ...)
    __attribute__((format(printf, 3, 4)));
static inline int orloj_ctx_fail(orloj_ctx* ctx, int code, const char* fmt, ...) {
    if (ctx) {
        va_list ap;
        va_start(ap, fmt);
        vsnprintf(ctx->msg, sizeof ctx->msg, fmt, ap);
        va_end(ap);
    }
    return code;
}

// One scheduling round's scoring and selection (sched.hip): the outputs of
// orloj_score_candidates (triangle prefixes) followed by orloj_select_batch,
// bit for bit.  In launches that take their E sums from emax_kernel, that
// kernel's waves and the score waves share one launch, and the selection
// forms E[L_B] and the scores from the panel sums before its argmax.
// d_done (mapped host memory, or NULL): each select workgroup g writes
// `round` to d_done[g] once its writes are visible to the host;
// *n_groups receives the number of select workgroups.
__attribute__((visibility("hidden"))) int orloj_internal_score_select(
    orloj_ctx* ctx, const orloj_grid* grid, const float* d_ccdf, const int32_t* d_support,
    const orloj_queues* queues, double b_expo_per_ms, const int64_t* d_cand_off,
    const int64_t* d_prob_off, float* d_finish_prob, double* d_expected_finish,
    float* d_expected_latency_ms, float* d_score, int32_t* d_sel_n, int32_t* d_sel_bs,
    float* d_sel_score, int32_t* d_done, int32_t round, int* n_groups);

#endif
