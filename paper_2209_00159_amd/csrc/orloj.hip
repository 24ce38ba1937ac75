// Candidate-batch scoring against latency SLOs on MI355X (gfx950).
//
// Implements the C ABI of include/orloj.h: the hot path of Orloj
// ("Predictably Serving Unpredictable DNNs", arXiv 2209.00159) as three
// hand-written HIP kernels for CDNA4:
//
//   cdf_kernel     histogram rows -> 1 - CDF (exact 64-bit running sums)
//   score_kernel   one workgroup per (model, batch size): scan over queue
//                  position of the members' CDF rows into the batch CDF,
//                  E[L_B], finish probabilities and Eq. (2) priorities of
//                  every prefix candidate, all in one pass
//   select_kernel  one workgroup per model: argmax over its candidates
//
// The work is a scan plus reductions over HBM-resident tables, not a dense
// contraction, so it runs on the vector ALUs (no MFMA): row loads
// prefetched into registers, fp64 running products, wave64 DPP scans and
// reductions, and LDS for the per-step snapshot the member lookups read.

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdarg.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <new>

#include "/root/repo/include/orloj.h"

namespace {

constexpr int kThreads = 256;               // 4 wave64 per workgroup
constexpr int kWaves = kThreads / 64;

// Device-side data error bits (reported by orloj_sync as ORLOJ_E_DATA).
constexpr int kErrEmptyHistogram = 1;
constexpr int kErrClassRange = 2;
constexpr int kErrDeadlineNaN = 4;
constexpr int kErrUnsorted = 8;
constexpr int kErrNowNaN = 16;

// ---------------------------------------------------------------------------
// wave64 helpers
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint64_t wave_incl_scan_u64(uint64_t x, int lane) {
#pragma unroll
    for (int s = 1; s < 64; s <<= 1) {
        uint64_t t = __shfl_up(x, s, 64);
        if (lane >= s) x += t;
    }
    return x;
}

// ---------------------------------------------------------------------------
// cdf_kernel: one workgroup per histogram row.  Thread t owns the VPT
// consecutive bins [t*VPT, t*VPT + VPT): it loads them once, the workgroup
// scans the per-thread sums (64-bit, exact), and each thread writes the
// complementary CDF 1 - F(x_{k+1}) = (total - running sum) / total.  The
// complement keeps full relative precision where F is close to 1, which is
// where the batch CDF (a product over up to hundreds of members) is most
// sensitive.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float survival(uint64_t cum, uint64_t tot, double rtot) {
    if (cum >= tot) return 0.0f;
    return (float)((double)(tot - cum) * rtot);
}

template <int VPT>
__global__ __launch_bounds__(kThreads) void cdf_kernel(const uint32_t* __restrict__ counts,
                                                       float* __restrict__ out, int64_t n_rows,
                                                       int K, int* __restrict__ err) {
    __shared__ uint64_t s_wave[kWaves];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int base = tid * VPT;
    const bool vec = (VPT % 4 == 0) && ((K & 3) == 0);
    for (int64_t r = blockIdx.x; r < n_rows; r += gridDim.x) {
        const uint32_t* row = counts + (size_t)r * (size_t)K;
        uint32_t v[VPT];
        if (vec && base + VPT <= K) {
#pragma unroll
            for (int j = 0; j < VPT; j += 4) {
                const uint4 t = *reinterpret_cast<const uint4*>(row + base + j);
                v[j] = t.x; v[j + 1] = t.y; v[j + 2] = t.z; v[j + 3] = t.w;
            }
        } else {
#pragma unroll
            for (int j = 0; j < VPT; ++j) v[j] = (base + j < K) ? row[base + j] : 0u;
        }
        uint64_t local = 0;
#pragma unroll
        for (int j = 0; j < VPT; ++j) local += v[j];
        const uint64_t incl = wave_incl_scan_u64(local, lane);
        if (lane == 63) s_wave[wv] = incl;
        __syncthreads();
        uint64_t off = incl - local, tot = 0;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            const uint64_t t = s_wave[w];
            if (w < wv) off += t;
            tot += t;
        }
        __syncthreads();   // s_wave is reused by the next row
        float* orow = out + (size_t)r * (size_t)K;
        if (tot == 0) {
            if (tid == 0) atomicOr(err, kErrEmptyHistogram);
#pragma unroll
            for (int j = 0; j < VPT; ++j)
                if (base + j < K) orow[base + j] = NAN;
            continue;
        }
        const double rtot = 1.0 / (double)tot;
        float o[VPT];
        uint64_t cum = off;
#pragma unroll
        for (int j = 0; j < VPT; ++j) {
            cum += v[j];
            o[j] = survival(cum, tot, rtot);
        }
        if (vec && base + VPT <= K) {
#pragma unroll
            for (int j = 0; j < VPT; j += 4)
                *reinterpret_cast<float4*>(orow + base + j) =
                    make_float4(o[j], o[j + 1], o[j + 2], o[j + 3]);
        } else {
#pragma unroll
            for (int j = 0; j < VPT; ++j)
                if (base + j < K) orow[base + j] = o[j];
        }
    }
}

// ---------------------------------------------------------------------------
// DPP building blocks (gfx9 encodings: row_shr:s = 0x110+s, row_bcast:15 =
// 0x142, row_bcast:31 = 0x143).  Lanes without a source read 0.
// ---------------------------------------------------------------------------
template <int CTRL, int ROWMASK = 0xf>
__device__ __forceinline__ float dpp(float x) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(
                                         0, __builtin_bit_cast(int, x), CTRL, ROWMASK, 0xf, true));
}

// Inclusive wave64 scan with geometric weights: lane L ends with
// sum_{L' <= L} x_{L'} r^(L - L').  rp[i] = r^(2^i); w15 = r^((L & 15) + 1);
// w31 = r^(L - 31) for lanes >= 32.
__device__ __forceinline__ float wave_wscan(float x, const float (&rp)[4], float w15, float w31) {
    x = fmaf(dpp<0x111>(x), rp[0], x);
    x = fmaf(dpp<0x112>(x), rp[1], x);
    x = fmaf(dpp<0x114>(x), rp[2], x);
    x = fmaf(dpp<0x118>(x), rp[3], x);
    x = fmaf(dpp<0x142, 0xa>(x), w15, x);
    x = fmaf(dpp<0x143, 0xc>(x), w31, x);
    return x;
}

// Inclusive wave64 sum scan: lane 63 ends with the total.
__device__ __forceinline__ float wave_scan_sum(float x) {
    x += dpp<0x111>(x);
    x += dpp<0x112>(x);
    x += dpp<0x114>(x);
    x += dpp<0x118>(x);
    x += dpp<0x142, 0xa>(x);
    x += dpp<0x143, 0xc>(x);
    return x;
}

template <int CTRL, int ROWMASK = 0xf>
__device__ __forceinline__ double dpp64(double x) {
    const uint64_t u = __builtin_bit_cast(uint64_t, x);
    const int lo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)u, CTRL, ROWMASK, 0xf, true);
    const int hi = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)(u >> 32), CTRL, ROWMASK, 0xf, true);
    return __builtin_bit_cast(double, ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

__device__ __forceinline__ double wave_scan_sum64(double x) {
    x += dpp64<0x111>(x);
    x += dpp64<0x112>(x);
    x += dpp64<0x114>(x);
    x += dpp64<0x118>(x);
    x += dpp64<0x142, 0xa>(x);
    x += dpp64<0x143, 0xc>(x);
    return x;
}

// Barrier that orders LDS only: global loads issued before it stay in
// flight (the prefetched rows of later steps).
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// 2^x by the hardware instruction; results below 2^-126 flush to 0.
__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

// ---------------------------------------------------------------------------
// score_kernel
// ---------------------------------------------------------------------------
struct ScoreArgs {
    const float* tab;          // [M][nbs][C][K] 1 - F(x_{k+1})
    const int64_t* queue_off;  // [M+1]
    const int32_t* cls;        // [N]
    const double* deadline;    // [N]
    const double* now;         // [M]
    const double* width;       // [M]
    const int64_t* cand_off;   // [M+1]
    const int64_t* prob_off;   // [M+1]
    float* P;
    double* E;
    float* EL;
    float* S;
    int* err;
    double b;
    int M, C, K, nbs, rect, maxcap;
    int bs[ORLOJ_MAX_BATCH_SIZES];
};

// Per-member lookup plan, built once per workgroup in LDS (it depends on
// the deadline only, not on the step).  For member m with deadline bin k
// and offset theta, every step the member wave reads from the snapshot
//   gk  = G(x_k) (bin k-1),   gk1 = G(x_{k+1}) (bin k),
// and assembles the discounted prefix Z(k-2) = sum_{i <= k-2} G(x_{i+1}) d^(k-2-i)
// from the wave prefixes, the lane prefix A, the quarter-end value of the
// thread's chunk and the G values of one 4-bin quarter:
//   zq  = fb * (fa * pre[wsel] + A[la]) + fq * zqe[izq] + sum_r wq[r] g4[r]
// then combines with fixed coefficients:
//   P   = gk + theta (gk1 - gk)
//   num = cg * (gk - omd * zq) + psi (gk1 - gk)
// An index of -1 reads as 0; beyond-the-grid members add one = 1 to both G
// values.  Dead requests and the k < 2 edge cases need no branch.
struct Member {
    int cls;      // class id (clamped into range)
    int ig0;      // snapshot index of G(x_k)     (-1: k = 0, dead or beyond)
    int ig1;      // snapshot index of G(x_{k+1}) (-1: dead or beyond)
    int ig4;      // float4 slot of the quarter holding bin k-2 (-1: k < 2 or dead)
    int izq;      // quarter-end snapshot index before that quarter (-1: none)
    int la;       // lane whose wave-internal scan precedes bin k-2 (-1: none)
    int wsel;     // which wave prefix (0: none, 1..3)
    float fa;     // d^(CPL (la - 64 wsel + 1)): weight of the wave prefix
    float fb;     // d^(j+1): weight of the lane prefix at bin k-2 (j = its chunk offset)
    float fq;     // d^(r+1): weight of the previous quarter end (r = offset in quarter)
    float wq[4];  // d^(r - r') for r' <= r, else 0
    float theta;  // position inside bin k
    float cg;     // gamma * exp(-b theta w), or gamma * exp(-b (tau - K w))
    float psi;    // (1 - exp(-b theta w)) / (b w)
    float one;    // 1 for beyond-the-grid members (P = 1), else 0
};

// LDS layout of one workgroup (floats unless noted):
//   g[2][256 CPL]   batch CDF G(x_{k+1}) of the current prefix, by step parity
//   zqe[2][256 NQ]  in-chunk discounted prefix of g at each quarter end
//   A[2][256]       wave-internal discounted scan of the chunk totals
//   e[2][4]         per-wave sums of (1 - g)
//   mem[maxcap]     Member
// g is stored float4-interleaved: the j-th float4 of thread t's chunk sits
// at float4 slot j * 256 + t, so a wave's snapshot stores are contiguous
// (no bank conflicts) and bin k is found by snap_index().
template <int CPL>
struct Quarters {
    static constexpr int QW = CPL < 4 ? CPL : 4;   // bins per quarter
    static constexpr int NQ = CPL / QW;            // quarters per thread
};

template <int CPL>
__host__ __device__ constexpr size_t score_smem_floats() {
    // + 8 padding keeps Member 16-byte aligned
    return 2 * (size_t)kThreads * CPL + 2 * (size_t)kThreads * Quarters<CPL>::NQ +
           2 * kThreads + 2 * kWaves + 8;
}

template <int CPL>
__device__ __forceinline__ int snap_index(int k) {
    if constexpr (CPL >= 4) {
        const int t = k / CPL, j = k - t * CPL;
        return ((j >> 2) * kThreads + t) * 4 + (j & 3);
    } else {
        return k;
    }
}

// Branch-free load of one thread's CPL bins of a row.  EXACT: the row
// fills the sweep waves (K = 256 CPL), so the loads are whole float4s.
// Otherwise indices past the end of the row are clamped to a valid address
// and their values are masked at use.  Every load is issued
// unconditionally so the prefetch ring keeps fixed registers.
template <int CPL, bool EXACT>
__device__ __forceinline__ void load_chunk(float (&v)[CPL], const float* __restrict__ row,
                                           int base, int K) {
    if constexpr (EXACT && CPL % 4 == 0) {
        const float4* r4 = reinterpret_cast<const float4*>(row + base);
#pragma unroll
        for (int j = 0; j < CPL / 4; ++j) {
            const float4 t = r4[j];
            v[4 * j] = t.x; v[4 * j + 1] = t.y; v[4 * j + 2] = t.z; v[4 * j + 3] = t.w;
        }
    } else {
#pragma unroll
        for (int j = 0; j < CPL; ++j) v[j] = row[min(base + j, K - 1)];
    }
}

// One workgroup scores every prefix of one model's queue at one batch size.
// Waves 0-3 (the sweep waves) own the bins: thread t keeps the batch CDF
// G_n(x_{k+1}) = prod_{i <= n} F_{c_i}(x_{k+1}) of its CPL consecutive bins
// as an fp64 running product (the table holds 1 - F, so a step is one fma).
// Step n: fold in member n's row (prefetched PF steps earlier), the
// per-thread sums of (1 - G) and of discounted G (split into 4-bin quarters
// so the dependency chains stay short), and a snapshot of G and of the
// quarter-end discounted prefixes in LDS, then one LDS barrier.  Wave 4 (the
// member wave) reads that snapshot after the barrier, scores the n+1
// members and writes the candidate's outputs while the sweep waves run
// step n+1 into the other snapshot buffer.  Only the member wave stores to
// global memory, so the sweep waves' outstanding-load counts stay exact and
// the prefetch ring is never drained early.
constexpr int kScoreThreads = kThreads + 64;

template <int CPL, int PF, bool EXACT>
__global__ __launch_bounds__(kScoreThreads) void score_kernel(const ScoreArgs a) {
    using Q = Quarters<CPL>;
    extern __shared__ __align__(16) float smem[];
    constexpr int KP = kThreads * CPL;
    constexpr int QP = kThreads * Q::NQ;
    float* s_g = smem;
    float* s_zq = s_g + 2 * KP;
    float* s_A = s_zq + 2 * QP;
    float* s_e = s_A + 2 * kThreads;
    Member* s_mem = reinterpret_cast<Member*>(s_e + 2 * kWaves + 8);

    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;

    // Largest batch sizes first: their workgroups run longest.
    const int bi = a.nbs - 1 - (int)(blockIdx.x / (unsigned)a.M);
    const int q = (int)(blockIdx.x % (unsigned)a.M);
    const int64_t q0 = a.queue_off[q];
    const int64_t N = a.queue_off[q + 1] - q0;
    const int bsz = a.bs[bi];
    const int64_t cap64 = a.rect ? N : (N < bsz ? N : (int64_t)bsz);
    if (cap64 <= 0 || cap64 > a.maxcap) return;   // the host sizes maxcap
    const int ncap = (int)cap64;

    const double w = a.width[q];
    const double nowq = a.now[q];
    const double b = a.b;
    const double bw = b * w;
    const int K = a.K;

    // Per-bin discount d = exp(-b w) and the powers the scans need.
    const float d = (float)exp(-bw);
    const float log2d = (float)(-bw * 1.4426950408889634);
    const int nsteps = (ncap + PF - 1) / PF * PF;
    const float gamma = (float)(-expm1(-bw) / bw);   // (1 - d) / (b w)

    // Members: bin and offset of each deadline (fp64 time, relative to
    // now) and their lookup plans.
    for (int m = tid; m < ncap; m += kScoreThreads) {
        int c = a.cls[q0 + m];
        const double D = a.deadline[q0 + m];
        int flag = 0;
        if (c < 0 || c >= a.C) { flag |= kErrClassRange; c = 0; }
        if (isnan(D)) flag |= kErrDeadlineNaN;
        if (m > 0 && D < a.deadline[q0 + m - 1]) flag |= kErrUnsorted;
        if (m == 0 && isnan(nowq)) flag |= kErrNowNaN;
        if (flag) atomicOr(a.err, flag);
        Member mb;
        mb.cls = c;
        mb.ig0 = mb.ig1 = mb.ig4 = mb.izq = mb.la = -1;
        mb.wsel = 0;
        mb.fa = mb.fb = mb.fq = 0.0f;
        mb.wq[0] = mb.wq[1] = mb.wq[2] = mb.wq[3] = 0.0f;
        mb.theta = mb.cg = mb.psi = mb.one = 0.0f;
        const double tau = D - nowq;
        int kz = -1;   // bin whose discounted prefix Z the priority needs
        if (tau > 0.0) {
            const double u = tau / w;
            if (u >= (double)K) {                  // beyond the grid: P = 1
                mb.one = 1.0f;
                mb.cg = gamma * (float)exp(-b * (tau - (double)K * w));
                kz = K - 2;
            } else {
                const double kf = floor(u);
                const double th = u - kf;
                const int k = (int)kf;
                mb.theta = (float)th;
                mb.cg = gamma * (float)exp(-b * th * w);
                mb.psi = (float)(-expm1(-b * th * w) / bw);
                mb.ig1 = snap_index<CPL>(k);
                if (k >= 1) mb.ig0 = snap_index<CPL>(k - 1);
                kz = k - 2;
            }
        }
        if (kz >= 0) {
            const int L = kz / CPL, j = kz - L * CPL;
            const int qq = j / Q::QW, r = j - qq * Q::QW;
            mb.ig4 = (qq * kThreads + L) * Q::QW;          // start of the quarter's G values
            if (qq > 0) mb.izq = L * Q::NQ + qq - 1;
            mb.fq = exp2f(log2d * (float)(r + 1));
            for (int rr = 0; rr <= r; ++rr) mb.wq[rr] = exp2f(log2d * (float)(r - rr));
            mb.fb = exp2f(log2d * (float)(j + 1));
            if (L > 0) {
                const int Lp = L - 1, wl = Lp >> 6;
                mb.la = Lp;
                mb.wsel = wl;
                mb.fa = exp2f(log2d * (float)(CPL * (Lp - 64 * wl + 1)));
            }
        }
        s_mem[m] = mb;
    }

    lds_barrier();

    if (wv < kWaves) {
        // ======================= sweep waves =======================
        float rp[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) rp[i] = exp2_hw(log2d * (float)(CPL << i));
        const float w15 = exp2_hw(log2d * (float)(CPL * ((lane & 15) + 1)));
        const float w31 = exp2_hw(log2d * (float)(CPL * (lane >= 32 ? lane - 31 : 0)));
        const float dQ = exp2_hw(log2d * (float)Q::QW);
        const int base = tid * CPL;
        const float* tab_qb =
            a.tab + ((size_t)q * (size_t)a.nbs + (size_t)bi) * (size_t)a.C * (size_t)K;
        double Gacc[CPL];   // G(x_{k+1}) of the current prefix, fp64 running product
#pragma unroll
        for (int j = 0; j < CPL; ++j) Gacc[j] = 1.0;

        // Prefetch ring: buf[i] holds the row of step n0 + i.  The tail is
        // padded to a multiple of PF with ghost steps (their rows repeat the
        // last member's and nobody reads their snapshot).
        float buf[PF][CPL];
#pragma unroll
        for (int i = 0; i < PF; ++i) {
            load_chunk<CPL, EXACT>(buf[i], tab_qb + (size_t)s_mem[min(i, ncap - 1)].cls * (size_t)K,
                                   base, K);
            // keep the priming loads in ring order, as the loop issues them
            __builtin_amdgcn_sched_barrier(0);
        }

        for (int n0 = 0; n0 < nsteps; n0 += PF) {
#pragma unroll
            for (int i = 0; i < PF; ++i) {
                const int n = n0 + i;
                const int par = n & 1;
                float* g_out = s_g + par * KP;
                // G <- G * F = G - G (1 - F), in fp64; per-quarter sums
                double gs[Q::QW];
                float zqv[Q::NQ];
                float gv[CPL];
#pragma unroll
                for (int r = 0; r < Q::QW; ++r) gs[r] = 0.0;
#pragma unroll
                for (int qq = 0; qq < Q::NQ; ++qq) {
                    float zz = 0.0f;
#pragma unroll
                    for (int r = 0; r < Q::QW; ++r) {
                        const int j = qq * Q::QW + r;
                        const float t = (EXACT || base + j < K) ? buf[i][j] : 0.0f;
                        Gacc[j] = fma(-Gacc[j], (double)t, Gacc[j]);
                        gs[r] += Gacc[j];
                        const float g = (float)Gacc[j];
                        zz = fmaf(zz, d, g);
                        gv[j] = g;
                    }
                    zqv[qq] = zz;
                }
                load_chunk<CPL, EXACT>(
                    buf[i], tab_qb + (size_t)s_mem[min(n + PF, ncap - 1)].cls * (size_t)K, base, K);
                // quarter ends of the in-chunk discounted prefix, and its total
                float zc = 0.0f;
#pragma unroll
                for (int qq = 0; qq < Q::NQ; ++qq) {
                    zc = fmaf(zc, dQ, zqv[qq]);
                    zqv[qq] = zc;
                }
                double gsum = 0.0;
#pragma unroll
                for (int r = 0; r < Q::QW; ++r) gsum += gs[r];
                // sum over this thread's bins of 1 - G (padding bins hold G = 1)
                const float e = (float)((double)CPL - gsum);
                if constexpr (CPL >= 4) {
#pragma unroll
                    for (int j = 0; j < CPL; j += 4) {
                        const int slot = ((j >> 2) * kThreads + tid) * 4;
                        *reinterpret_cast<float4*>(g_out + slot) =
                            make_float4(gv[j], gv[j + 1], gv[j + 2], gv[j + 3]);
                    }
                } else {
#pragma unroll
                    for (int j = 0; j < CPL; ++j) g_out[base + j] = gv[j];
                }
                float* zq_out = s_zq + par * QP + tid * Q::NQ;
                if constexpr (Q::NQ == 4) {
                    *reinterpret_cast<float4*>(zq_out) = make_float4(zqv[0], zqv[1], zqv[2], zqv[3]);
                } else {
#pragma unroll
                    for (int qq = 0; qq < Q::NQ; ++qq) zq_out[qq] = zqv[qq];
                }
                const float esum = wave_scan_sum(e);
                const float A = wave_wscan(zc, rp, w15, w31);

                s_A[par * kThreads + tid] = A;
                if (lane == 63) s_e[par * kWaves + wv] = esum;
                lds_barrier();
            }
        }
    } else {
        // ======================= member wave =======================
        const float omd = (float)(-expm1(-bw));          // 1 - d
        const float d64c = exp2_hw(log2d * (float)(64 * CPL));
        int64_t cand = a.cand_off[q], prob = a.prob_off[q];
        for (int j = 0; j < bi; ++j) {
            const int64_t c = a.rect ? N : (N < a.bs[j] ? N : (int64_t)a.bs[j]);
            cand += c;
            prob += c * (c + 1) / 2;
        }
        for (int n = 0; n < nsteps; ++n) {
            lds_barrier();
            if (n >= ncap) continue;
            const int par = n & 1;
            const float* g = s_g + par * KP;
            const float* zq = s_zq + par * QP;
            const float* As = s_A + par * kThreads;
            // discounted totals at the end of waves 0..2
            const float T0 = As[63], T1 = As[127], T2 = As[191];
            const float W2 = fmaf(T0, d64c, T1);
            const float W3 = fmaf(W2, d64c, T2);
            const double es = (double)s_e[par * kWaves + 0] + (double)s_e[par * kWaves + 1] +
                              (double)s_e[par * kWaves + 2] + (double)s_e[par * kWaves + 3];
            const double el = w * (0.5 + es);
            const int nn = n + 1;
            double pP = 0.0;
            float pN = 0.0f;
            for (int m = lane; m < nn; m += 64) {
                const Member mb = s_mem[m];
                const float g0 = g[max(mb.ig0, 0)];
                const float g1 = g[max(mb.ig1, 0)];
                const float al0 = As[max(mb.la, 0)];
                const float zq0 = zq[max(mb.izq, 0)];
                float g4[4];
                if constexpr (Q::QW == 4) {
                    const float4 t4 = *reinterpret_cast<const float4*>(g + max(mb.ig4, 0));
                    g4[0] = t4.x; g4[1] = t4.y; g4[2] = t4.z; g4[3] = t4.w;
                } else {
#pragma unroll
                    for (int r = 0; r < 4; ++r) g4[r] = r < Q::QW ? g[max(mb.ig4, 0) + r] : 0.0f;
                }
                const float gk = (mb.ig0 >= 0 ? g0 : 0.0f) + mb.one;
                const float gk1 = (mb.ig1 >= 0 ? g1 : 0.0f) + mb.one;
                const float al = mb.la >= 0 ? al0 : 0.0f;
                const float zqp = mb.izq >= 0 ? zq0 : 0.0f;
                const float pre = mb.wsel == 1 ? T0 : (mb.wsel == 2 ? W2 : (mb.wsel == 3 ? W3 : 0.0f));
                float zin = mb.fq * zqp;
#pragma unroll
                for (int r = 0; r < 4; ++r) zin = fmaf(mb.wq[r], g4[r], zin);
                const float zqv = fmaf(mb.fb, fmaf(mb.fa, pre, al), mb.ig4 >= 0 ? zin : 0.0f);
                const float h = gk1 - gk;
                const float P = fmaf(mb.theta, h, gk);
                const float num = fmaf(mb.cg, fmaf(-omd, zqv, gk), h * mb.psi);
                a.P[prob + (int64_t)n * nn / 2 + m] = P;
                pP += (double)P;
                pN += num;
            }
            pP = wave_scan_sum64(pP);
            pN = wave_scan_sum(pN);
            if (lane == 63) {
                a.E[cand + n] = pP;
                a.EL[cand + n] = (float)el;
                a.S[cand + n] = (float)((double)pN / el);
            }
        }
    }
}

// ---------------------------------------------------------------------------
// select_kernel: one workgroup per model; thread i reads candidates i,
// i + 256, ... (coalesced) and finds its (batch size, n) from the block
// starts of the model's batch sizes.
// ---------------------------------------------------------------------------
struct SelectArgs {
    const int64_t* queue_off;
    const int64_t* cand_off;
    const float* S;
    int32_t* sel_n;
    int32_t* sel_bs;
    float* sel_score;
    int nbs, rect;
    int bs[ORLOJ_MAX_BATCH_SIZES];
};

struct Best {
    float s;
    int n;
    int bs;
};

__device__ __forceinline__ bool better(const Best& x, const Best& y) {
    // larger score; exact ties: larger n, then smaller batch size
    if (x.n == 0) return false;
    if (y.n == 0) return true;
    if (x.s != y.s) return x.s > y.s;
    if (x.n != y.n) return x.n > y.n;
    return x.bs < y.bs;
}

__global__ __launch_bounds__(kThreads) void select_kernel(const SelectArgs a) {
    __shared__ int64_t s_start[ORLOJ_MAX_BATCH_SIZES + 1];
    __shared__ Best s_best[kWaves];
    const int q = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int64_t N = a.queue_off[q + 1] - a.queue_off[q];
    if (tid == 0) {
        int64_t acc = 0;
        for (int bi = 0; bi < a.nbs; ++bi) {
            s_start[bi] = acc;
            const int bsz = a.bs[bi];
            acc += a.rect ? N : (N < bsz ? N : (int64_t)bsz);
        }
        s_start[a.nbs] = acc;
    }
    __syncthreads();
    const int64_t total = s_start[a.nbs];
    const float* S = a.S + a.cand_off[q];
    Best best{0.0f, 0, 0};
    for (int64_t i = tid; i < total; i += kThreads) {
        int lo = 0, hi = a.nbs - 1;          // last bi with s_start[bi] <= i
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (s_start[mid] <= i) lo = mid; else hi = mid - 1;
        }
        const int n = (int)(i - s_start[lo]) + 1;
        const int bsz = a.bs[lo];
        const float s = S[i];
        if (n <= bsz && s == s) {   // NaN never wins
            const Best c{s, n, bsz};
            if (better(c, best)) best = c;
        }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        Best o;
        o.s = __shfl_xor(best.s, off, 64);
        o.n = __shfl_xor(best.n, off, 64);
        o.bs = __shfl_xor(best.bs, off, 64);
        if (better(o, best)) best = o;
    }
    if (lane == 0) s_best[wv] = best;
    __syncthreads();
    if (tid == 0) {
        for (int w = 1; w < kWaves; ++w)
            if (better(s_best[w], best)) best = s_best[w];
        if (best.n > 0 && best.s > 0.0f) {
            a.sel_n[q] = best.n;
            a.sel_bs[q] = best.bs;
            a.sel_score[q] = best.s;
        } else {
            a.sel_n[q] = 0;
            a.sel_bs[q] = 0;
            a.sel_score[q] = 0.0f;
        }
    }
}

}  // namespace

// ===========================================================================
// C ABI
// ===========================================================================
struct orloj_ctx {
    int device;
    hipStream_t stream;
    int* d_err;
    char msg[512];
};

namespace {

int fail(orloj_ctx* ctx, int code, const char* fmt, ...) __attribute__((format(printf, 3, 4)));
int fail(orloj_ctx* ctx, int code, const char* fmt, ...) {
    if (ctx) {
        va_list ap;
        va_start(ap, fmt);
        vsnprintf(ctx->msg, sizeof ctx->msg, fmt, ap);
        va_end(ap);
    }
    return code;
}

int hip_fail(orloj_ctx* ctx, hipError_t e, const char* what) {
    return fail(ctx, ORLOJ_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

int check_grid(orloj_ctx* ctx, const orloj_grid* g) {
    if (!g) return fail(ctx, ORLOJ_E_INVALID, "grid is NULL");
    if (g->n_models < 0) return fail(ctx, ORLOJ_E_INVALID, "n_models < 0");
    if (g->n_classes < 1) return fail(ctx, ORLOJ_E_INVALID, "n_classes < 1");
    if (g->n_bins < 1) return fail(ctx, ORLOJ_E_INVALID, "n_bins < 1");
    if (g->n_bins > ORLOJ_MAX_BINS)
        return fail(ctx, ORLOJ_E_UNSUPPORTED, "n_bins %d > %d", g->n_bins, ORLOJ_MAX_BINS);
    if (g->n_bs < 1) return fail(ctx, ORLOJ_E_INVALID, "n_bs < 1");
    if (g->n_bs > ORLOJ_MAX_BATCH_SIZES)
        return fail(ctx, ORLOJ_E_UNSUPPORTED, "n_bs %d > %d", g->n_bs, ORLOJ_MAX_BATCH_SIZES);
    if (!g->batch_sizes) return fail(ctx, ORLOJ_E_INVALID, "batch_sizes is NULL");
    for (int i = 0; i < g->n_bs; ++i) {
        if (g->batch_sizes[i] < 1) return fail(ctx, ORLOJ_E_INVALID, "batch size < 1");
        if (i > 0 && g->batch_sizes[i] <= g->batch_sizes[i - 1])
            return fail(ctx, ORLOJ_E_INVALID, "batch sizes not strictly increasing");
    }
    if (g->n_models > 0 && !g->d_bin_width_ms)
        return fail(ctx, ORLOJ_E_INVALID, "d_bin_width_ms is NULL");
    return ORLOJ_OK;
}

int check_queues(orloj_ctx* ctx, const orloj_grid* g, const orloj_queues* qs) {
    if (!qs) return fail(ctx, ORLOJ_E_INVALID, "queues is NULL");
    if (!qs->h_queue_off) return fail(ctx, ORLOJ_E_INVALID, "h_queue_off is NULL");
    if (qs->h_queue_off[0] != 0) return fail(ctx, ORLOJ_E_INVALID, "h_queue_off[0] != 0");
    for (int q = 0; q < g->n_models; ++q)
        if (qs->h_queue_off[q + 1] < qs->h_queue_off[q])
            return fail(ctx, ORLOJ_E_INVALID, "h_queue_off decreases at model %d", q);
    if (g->n_models > 0) {
        if (!qs->d_queue_off || !qs->d_now_ms)
            return fail(ctx, ORLOJ_E_INVALID, "d_queue_off / d_now_ms is NULL");
        if (qs->h_queue_off[g->n_models] > 0 && (!qs->d_class || !qs->d_deadline_ms))
            return fail(ctx, ORLOJ_E_INVALID, "d_class / d_deadline_ms is NULL");
    }
    return ORLOJ_OK;
}

int64_t ncap_of(int64_t N, int bsz, int rect) { return rect ? N : (N < bsz ? N : (int64_t)bsz); }

int chunk_per_lane(int K) {
    int c = 1;
    while (c * kThreads < K) c <<= 1;
    return c;
}

#ifndef ORLOJ_SCORE_PREFETCH
#define ORLOJ_SCORE_PREFETCH 2   // rows in flight per sweep thread at 16+ bins per thread
#endif

template <int CPL, bool EXACT>
hipError_t launch_score_v(const ScoreArgs& a, unsigned grid, hipStream_t st) {
    constexpr int PF = CPL >= 16 ? ORLOJ_SCORE_PREFETCH : 3;
    const size_t sm = score_smem_floats<CPL>() * sizeof(float) + (size_t)a.maxcap * sizeof(Member);
    static size_t attr_bytes = 0;   // per template instance; device-independent
    if (sm > attr_bytes) {
        hipError_t e = hipFuncSetAttribute((const void*)score_kernel<CPL, PF, EXACT>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)sm);
        if (e != hipSuccess) return e;
        attr_bytes = sm;
    }
    hipLaunchKernelGGL((score_kernel<CPL, PF, EXACT>), dim3(grid), dim3(kScoreThreads), sm, st, a);
    return hipGetLastError();
}

template <int CPL>
hipError_t launch_score(const ScoreArgs& a, unsigned grid, hipStream_t st) {
    return a.K == kThreads * CPL ? launch_score_v<CPL, true>(a, grid, st)
                                 : launch_score_v<CPL, false>(a, grid, st);
}

template <int VPT>
hipError_t launch_cdf(const uint32_t* c, float* o, int64_t rows, int K, int* err, hipStream_t st) {
    const int64_t cap = 1 << 20;
    const unsigned grid = (unsigned)(rows < cap ? rows : cap);
    hipLaunchKernelGGL(cdf_kernel<VPT>, dim3(grid), dim3(kThreads), 0, st, c, o, rows, K, err);
    return hipGetLastError();
}

}  // namespace

extern "C" {

int orloj_create(orloj_ctx** out, int32_t hip_device, void* hip_stream) {
    if (!out) return ORLOJ_E_INVALID;
    *out = nullptr;
    orloj_ctx* ctx = new (std::nothrow) orloj_ctx;
    if (!ctx) return ORLOJ_E_NOMEM;
    ctx->device = hip_device;
    ctx->stream = (hipStream_t)hip_stream;
    ctx->d_err = nullptr;
    ctx->msg[0] = 0;
    int n = 0;
    if (hipGetDeviceCount(&n) != hipSuccess || hip_device < 0 || hip_device >= n) {
        delete ctx;
        return ORLOJ_E_INVALID;
    }
    hipError_t e = hipSetDevice(hip_device);
    if (e == hipSuccess) e = hipMalloc((void**)&ctx->d_err, sizeof(int));
    if (e == hipSuccess) e = hipMemset(ctx->d_err, 0, sizeof(int));
    if (e != hipSuccess) {
        if (ctx->d_err) (void)hipFree(ctx->d_err);
        delete ctx;
        return e == hipErrorOutOfMemory ? ORLOJ_E_NOMEM : ORLOJ_E_HIP;
    }
    *out = ctx;
    return ORLOJ_OK;
}

void orloj_destroy(orloj_ctx* ctx) {
    if (!ctx) return;
    (void)hipSetDevice(ctx->device);
    (void)hipStreamSynchronize(ctx->stream);
    if (ctx->d_err) (void)hipFree(ctx->d_err);
    delete ctx;
}

int orloj_set_stream(orloj_ctx* ctx, void* hip_stream) {
    if (!ctx) return ORLOJ_E_INVALID;
    ctx->stream = (hipStream_t)hip_stream;
    return ORLOJ_OK;
}

const char* orloj_last_error(const orloj_ctx* ctx) { return ctx ? ctx->msg : "context is NULL"; }

int orloj_sync(orloj_ctx* ctx) {
    if (!ctx) return ORLOJ_E_INVALID;
    hipError_t e = hipSetDevice(ctx->device);
    if (e == hipSuccess) e = hipStreamSynchronize(ctx->stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "hipStreamSynchronize");
    int flags = 0;
    e = hipMemcpy(&flags, ctx->d_err, sizeof(int), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(ctx, e, "reading the device status word");
    if (flags) {
        e = hipMemset(ctx->d_err, 0, sizeof(int));
        if (e != hipSuccess) return hip_fail(ctx, e, "clearing the device status word");
        return fail(ctx, ORLOJ_E_DATA, "device data error:%s%s%s%s%s",
                    (flags & kErrEmptyHistogram) ? " histogram-with-no-samples" : "",
                    (flags & kErrClassRange) ? " class-id-out-of-range" : "",
                    (flags & kErrDeadlineNaN) ? " NaN-deadline" : "",
                    (flags & kErrUnsorted) ? " deadlines-not-sorted" : "",
                    (flags & kErrNowNaN) ? " NaN-now" : "");
    }
    return ORLOJ_OK;
}

int orloj_build_cdfs(orloj_ctx* ctx, int64_t n_rows, int32_t n_bins, const uint32_t* d_counts,
                     float* d_ccdf) {
    if (!ctx) return ORLOJ_E_INVALID;
    if (n_rows < 0) return fail(ctx, ORLOJ_E_INVALID, "n_rows < 0");
    if (n_bins < 1) return fail(ctx, ORLOJ_E_INVALID, "n_bins < 1");
    if (n_bins > ORLOJ_MAX_BINS)
        return fail(ctx, ORLOJ_E_UNSUPPORTED, "n_bins %d > %d", n_bins, ORLOJ_MAX_BINS);
    if (n_rows == 0) return ORLOJ_OK;
    if (!d_counts || !d_ccdf) return fail(ctx, ORLOJ_E_INVALID, "NULL buffer");
    const char* cb = (const char*)d_counts;
    const char* ob = (const char*)d_ccdf;
    const size_t bytes = (size_t)n_rows * (size_t)n_bins * 4;
    if (cb < ob + bytes && ob < cb + bytes)
        return fail(ctx, ORLOJ_E_INVALID, "d_counts and d_ccdf overlap");
    hipError_t e = hipSetDevice(ctx->device);
    if (e != hipSuccess) return hip_fail(ctx, e, "hipSetDevice");
    const int vpt = chunk_per_lane(n_bins);
    switch (vpt) {
        case 1: e = launch_cdf<1>(d_counts, d_ccdf, n_rows, n_bins, ctx->d_err, ctx->stream); break;
        case 2: e = launch_cdf<2>(d_counts, d_ccdf, n_rows, n_bins, ctx->d_err, ctx->stream); break;
        case 4: e = launch_cdf<4>(d_counts, d_ccdf, n_rows, n_bins, ctx->d_err, ctx->stream); break;
        case 8: e = launch_cdf<8>(d_counts, d_ccdf, n_rows, n_bins, ctx->d_err, ctx->stream); break;
        case 16: e = launch_cdf<16>(d_counts, d_ccdf, n_rows, n_bins, ctx->d_err, ctx->stream); break;
        default: e = launch_cdf<32>(d_counts, d_ccdf, n_rows, n_bins, ctx->d_err, ctx->stream); break;
    }
    if (e != hipSuccess) return hip_fail(ctx, e, "cdf_kernel launch");
    return ORLOJ_OK;
}

int orloj_output_sizes(const orloj_grid* grid, const orloj_queues* queues, int32_t prefix_mode,
                       int64_t* n_cands, int64_t* n_probs, int64_t* h_cand_off,
                       int64_t* h_prob_off) {
    if (prefix_mode != ORLOJ_PREFIX_TRIANGLE && prefix_mode != ORLOJ_PREFIX_RECT)
        return ORLOJ_E_INVALID;
    int rc = check_grid(nullptr, grid);
    if (rc) return rc;
    if (!queues || !queues->h_queue_off || queues->h_queue_off[0] != 0) return ORLOJ_E_INVALID;
    int64_t nc = 0, np = 0;
    if (h_cand_off) h_cand_off[0] = 0;
    if (h_prob_off) h_prob_off[0] = 0;
    for (int q = 0; q < grid->n_models; ++q) {
        const int64_t N = queues->h_queue_off[q + 1] - queues->h_queue_off[q];
        if (N < 0) return ORLOJ_E_INVALID;
        for (int bi = 0; bi < grid->n_bs; ++bi) {
            const int64_t c = ncap_of(N, grid->batch_sizes[bi], prefix_mode);
            nc += c;
            np += c * (c + 1) / 2;
        }
        if (h_cand_off) h_cand_off[q + 1] = nc;
        if (h_prob_off) h_prob_off[q + 1] = np;
    }
    if (n_cands) *n_cands = nc;
    if (n_probs) *n_probs = np;
    return ORLOJ_OK;
}

int orloj_score_candidates(orloj_ctx* ctx, const orloj_grid* grid, const float* d_ccdf,
                           const orloj_queues* queues, double b_expo_per_ms, int32_t prefix_mode,
                           const int64_t* d_cand_off, const int64_t* d_prob_off,
                           float* d_finish_prob, double* d_expected_finish,
                           float* d_expected_latency_ms, float* d_score) {
    if (!ctx) return ORLOJ_E_INVALID;
    int rc = check_grid(ctx, grid);
    if (rc) return rc;
    rc = check_queues(ctx, grid, queues);
    if (rc) return rc;
    if (prefix_mode != ORLOJ_PREFIX_TRIANGLE && prefix_mode != ORLOJ_PREFIX_RECT)
        return fail(ctx, ORLOJ_E_INVALID, "prefix_mode %d", prefix_mode);
    if (!(b_expo_per_ms > 0.0) || !isfinite(b_expo_per_ms))
        return fail(ctx, ORLOJ_E_INVALID, "b_expo_per_ms must be finite and > 0");
    const int M = grid->n_models;
    if (M == 0) return ORLOJ_OK;
    int64_t maxcap = 0, total = 0;
    for (int q = 0; q < M; ++q) {
        const int64_t N = queues->h_queue_off[q + 1] - queues->h_queue_off[q];
        for (int bi = 0; bi < grid->n_bs; ++bi) {
            const int64_t c = ncap_of(N, grid->batch_sizes[bi], prefix_mode);
            if (c > maxcap) maxcap = c;
            total += c;
        }
    }
    if (maxcap > ORLOJ_MAX_PREFIX)
        return fail(ctx, ORLOJ_E_UNSUPPORTED, "prefix of %lld members > %d",
                    (long long)maxcap, ORLOJ_MAX_PREFIX);
    if (total == 0) return ORLOJ_OK;
    if (!d_ccdf || !d_cand_off || !d_prob_off || !d_finish_prob || !d_expected_finish ||
        !d_expected_latency_ms || !d_score)
        return fail(ctx, ORLOJ_E_INVALID, "NULL device buffer");
    const int64_t nblk = (int64_t)M * grid->n_bs;
    if (nblk > 0x7fffffff) return fail(ctx, ORLOJ_E_UNSUPPORTED, "too many (model, batch size) pairs");

    ScoreArgs a;
    a.tab = d_ccdf;
    a.queue_off = queues->d_queue_off;
    a.cls = queues->d_class;
    a.deadline = queues->d_deadline_ms;
    a.now = queues->d_now_ms;
    a.width = grid->d_bin_width_ms;
    a.cand_off = d_cand_off;
    a.prob_off = d_prob_off;
    a.P = d_finish_prob;
    a.E = d_expected_finish;
    a.EL = d_expected_latency_ms;
    a.S = d_score;
    a.err = ctx->d_err;
    a.b = b_expo_per_ms;
    a.M = M;
    a.C = grid->n_classes;
    a.K = grid->n_bins;
    a.nbs = grid->n_bs;
    a.rect = prefix_mode;
    a.maxcap = (int)maxcap;
    memset(a.bs, 0, sizeof a.bs);
    for (int i = 0; i < grid->n_bs; ++i) a.bs[i] = grid->batch_sizes[i];

    hipError_t e = hipSetDevice(ctx->device);
    if (e != hipSuccess) return hip_fail(ctx, e, "hipSetDevice");
    const unsigned g = (unsigned)nblk;
    switch (chunk_per_lane(grid->n_bins)) {
        case 1: e = launch_score<1>(a, g, ctx->stream); break;
        case 2: e = launch_score<2>(a, g, ctx->stream); break;
        case 4: e = launch_score<4>(a, g, ctx->stream); break;
        case 8: e = launch_score<8>(a, g, ctx->stream); break;
        case 16: e = launch_score<16>(a, g, ctx->stream); break;
        default: e = launch_score<32>(a, g, ctx->stream); break;
    }
    if (e != hipSuccess) return hip_fail(ctx, e, "score_kernel launch");
    return ORLOJ_OK;
}

int orloj_select_batch(orloj_ctx* ctx, const orloj_grid* grid, const orloj_queues* queues,
                       int32_t prefix_mode, const int64_t* d_cand_off, const float* d_score,
                       int32_t* d_sel_n, int32_t* d_sel_bs, float* d_sel_score) {
    if (!ctx) return ORLOJ_E_INVALID;
    int rc = check_grid(ctx, grid);
    if (rc) return rc;
    rc = check_queues(ctx, grid, queues);
    if (rc) return rc;
    if (prefix_mode != ORLOJ_PREFIX_TRIANGLE && prefix_mode != ORLOJ_PREFIX_RECT)
        return fail(ctx, ORLOJ_E_INVALID, "prefix_mode %d", prefix_mode);
    const int M = grid->n_models;
    if (M == 0) return ORLOJ_OK;
    if (!d_cand_off || !d_sel_n || !d_sel_bs || !d_sel_score)
        return fail(ctx, ORLOJ_E_INVALID, "NULL device buffer");
    const int64_t total = queues->h_queue_off[M];
    if (total > 0 && !d_score) return fail(ctx, ORLOJ_E_INVALID, "d_score is NULL");
    SelectArgs a;
    a.queue_off = queues->d_queue_off;
    a.cand_off = d_cand_off;
    a.S = d_score;
    a.sel_n = d_sel_n;
    a.sel_bs = d_sel_bs;
    a.sel_score = d_sel_score;
    a.nbs = grid->n_bs;
    a.rect = prefix_mode;
    memset(a.bs, 0, sizeof a.bs);
    for (int i = 0; i < grid->n_bs; ++i) a.bs[i] = grid->batch_sizes[i];
    hipError_t e = hipSetDevice(ctx->device);
    if (e != hipSuccess) return hip_fail(ctx, e, "hipSetDevice");
    hipLaunchKernelGGL(select_kernel, dim3((unsigned)M), dim3(kThreads), 0, ctx->stream, a);
    e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(ctx, e, "select_kernel launch");
    return ORLOJ_OK;
}

}  // extern "C"

