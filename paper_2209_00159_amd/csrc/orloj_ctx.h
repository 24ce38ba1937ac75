// Internal to the library: the context every entry point takes, shared by
// its translation units (orloj.hip: kernels and scoring entry points;
// sched.hip: the host scheduling runtime).  Not part of the C ABI.
#ifndef ORLOJ_CTX_INTERNAL_H
#define ORLOJ_CTX_INTERNAL_H

#include <hip/hip_runtime_api.h>
#include <stdarg.h>
#include <stdio.h>

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

#endif
