// Candidate-batch scoring against latency SLOs on MI355X (gfx950).
//
// Implements the C ABI of include/orloj.h: the hot path of Orloj
// ("Predictably Serving Unpredictable DNNs", arXiv 2209.00159) as
// hand-written HIP kernels for CDNA4:
//
//   cdf_kernel     histogram rows -> 1 - CDF (exact 64-bit running sums)
//   score_kernel   one workgroup per (model, batch size): scan over queue
//                  position of the members' CDF rows into the batch CDF,
//                  E[L_B], finish probabilities and Eq. (2) priorities of
//                  every prefix candidate, all in one pass
//   emax_kernel    affine mode: the sums behind E[L_B], once per prefix
//                  length instead of once per batch size
//   select_kernel  one workgroup per model: argmax over its candidates
//
// and, around the path, laws_kernel / iterate_kernel (one Algorithm 1
// iteration with the paper's own priority) and accumulate_kernel (profiler
// samples into the histograms).
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

#include <algorithm>
#include <mutex>
#include <new>
#include <type_traits>

#include "../../include/orloj.h"
#include "orloj_ctx.h"

namespace {

constexpr int kThreads = 256;               // 4 wave64 per workgroup
constexpr int kWaves = kThreads / 64;

// Device-side data error bits (reported by orloj_sync as ORLOJ_E_DATA).
constexpr int kErrEmptyHistogram = 1;
constexpr int kErrClassRange = 2;
constexpr int kErrDeadlineNaN = 4;
constexpr int kErrUnsorted = 8;
constexpr int kErrNowNaN = 16;
constexpr int kErrWidth = 32;
constexpr int kErrWeights = 64;
constexpr int kErrCost = 128;
constexpr int kErrAffine = 256;

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

// Sum over the wave, in every lane.
__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t x, int lane) {
    const uint64_t s = wave_incl_scan_u64(x, lane);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)s, 63);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(s >> 32), 63);
    return ((uint64_t)hi << 32) | lo;
}

// ---------------------------------------------------------------------------
// cdf_kernel: one workgroup per histogram row.  Thread t owns the VPT
// consecutive bins [t*VPT, t*VPT + VPT): it loads them once, the workgroup
// scans the per-thread sums (64-bit, exact), and each thread writes the
// complementary CDF 1 - F(x_{k+1}) = (total - running sum) / total.  The
// complement keeps full relative precision where F is close to 1, which is
// where the batch CDF (a product over up to hundreds of members) is most
// sensitive.  Optionally the row's support is recorded as well: the first
// bin holding mass (every earlier entry is exactly 1) and the last bin
// holding mass (it and every later entry are exactly 0).
// ---------------------------------------------------------------------------
__device__ __forceinline__ float survival(uint64_t cum, uint64_t tot, double rtot) {
    if (cum >= tot) return 0.0f;
    return (float)((double)(tot - cum) * rtot);
}

__device__ __forceinline__ int wave_min_i32(int x) {
#pragma unroll
    for (int s = 1; s < 64; s <<= 1) x = min(x, __shfl_xor(x, s, 64));
    return x;
}

__device__ __forceinline__ int wave_max_i32(int x) {
#pragma unroll
    for (int s = 1; s < 64; s <<= 1) x = max(x, __shfl_xor(x, s, 64));
    return x;
}

template <int VPT>
__global__ __launch_bounds__(kThreads) void cdf_kernel(const uint32_t* __restrict__ counts,
                                                       float* __restrict__ out,
                                                       int32_t* __restrict__ support, int64_t n_rows,
                                                       int K, int* __restrict__ err) {
    __shared__ uint64_t s_wave[kWaves];
    __shared__ int s_sup[2][kWaves];
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
        float* orow = out + (size_t)r * (size_t)K;
        if (support) {
            // first bin with mass; last bin with mass (K when the row is empty)
            int lo = K, hi = -1;
#pragma unroll
            for (int j = 0; j < VPT; ++j) {
                if (v[j] != 0u) {
                    lo = min(lo, base + j);
                    hi = max(hi, base + j);
                }
            }
            lo = wave_min_i32(lo);
            hi = -wave_min_i32(-hi);
            if (lane == 0) { s_sup[0][wv] = lo; s_sup[1][wv] = hi; }
            __syncthreads();
            if (tid == 0) {
                for (int w = 1; w < kWaves; ++w) {
                    lo = min(lo, s_sup[0][w]);
                    hi = max(hi, s_sup[1][w]);
                }
                support[2 * r] = hi < 0 ? 0 : lo;
                support[2 * r + 1] = hi < 0 ? 0 : hi;
            }
        }
        __syncthreads();   // s_wave and s_sup are reused by the next row
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
// Each stage is x <- x' r + x with x' the DPP-moved x (0 where a lane has no
// source, and rows outside the row mask keep x): one v_fmac_f32 with the
// DPP move on its first source.  The compiler emits a separate move and
// fma per stage, so the stages are written out; a VALU write of a VGPR
// needs two wait states before a DPP read of it (s_nop 1), and the last
// stage is followed by two as well, since the compiler cannot see into the
// block when it places the next reader.
__device__ __forceinline__ float wave_wscan(float x, const float (&rp)[4], float w15, float w31) {
    asm volatile(
        "s_nop 1\n\t"
        "v_fmac_f32_dpp %0, %0, %1 row_shr:1 row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"
        "s_nop 1\n\t"
        "v_fmac_f32_dpp %0, %0, %2 row_shr:2 row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"
        "s_nop 1\n\t"
        "v_fmac_f32_dpp %0, %0, %3 row_shr:4 row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"
        "s_nop 1\n\t"
        "v_fmac_f32_dpp %0, %0, %4 row_shr:8 row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"
        "s_nop 1\n\t"
        "v_fmac_f32_dpp %0, %0, %5 row_bcast:15 row_mask:0xa bank_mask:0xf bound_ctrl:1\n\t"
        "s_nop 1\n\t"
        "v_fmac_f32_dpp %0, %0, %6 row_bcast:31 row_mask:0xc bank_mask:0xf bound_ctrl:1\n\t"
        "s_nop 1"
        : "+v"(x)
        : "v"(rp[0]), "v"(rp[1]), "v"(rp[2]), "v"(rp[3]), "v"(w15), "v"(w31));
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

// Two wave sums at once.  v_permlane32_swap exchanges the upper half of x
// with the lower half of y, so after one add lane l < 32 holds x_l + x_(l+32)
// and lane l >= 32 holds y_(l-32) + y_l; a DPP sum within each half (rows of
// 16, then row 0 into row 1 and row 2 into row 3) leaves the total of x in
// lane 31 and that of y in lane 63.  Each total comes out of one fixed tree,
// whatever the other value is.
__device__ __forceinline__ float wave_pair_sum(float x, float y) {
    const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(unsigned, x),
                                                    __builtin_bit_cast(unsigned, y), false, false);
    float z = __builtin_bit_cast(float, (unsigned)r[0]) + __builtin_bit_cast(float, (unsigned)r[1]);
    z += dpp<0x111>(z);
    z += dpp<0x112>(z);
    z += dpp<0x114>(z);
    z += dpp<0x118>(z);
    z += dpp<0x142, 0xa>(z);
    return z;
}

__device__ __forceinline__ double wave_pair_sum64(double x, double y) {
    const uint64_t ux = __builtin_bit_cast(uint64_t, x), uy = __builtin_bit_cast(uint64_t, y);
    const auto lo = __builtin_amdgcn_permlane32_swap((unsigned)ux, (unsigned)uy, false, false);
    const auto hi = __builtin_amdgcn_permlane32_swap((unsigned)(ux >> 32), (unsigned)(uy >> 32), false, false);
    const double a = __builtin_bit_cast(double, ((uint64_t)(unsigned)hi[0] << 32) | (unsigned)lo[0]);
    const double b = __builtin_bit_cast(double, ((uint64_t)(unsigned)hi[1] << 32) | (unsigned)lo[1]);
    double z = a + b;
    z += dpp64<0x111>(z);
    z += dpp64<0x112>(z);
    z += dpp64<0x114>(z);
    z += dpp64<0x118>(z);
    z += dpp64<0x142, 0xa>(z);
    return z;
}

// 2^x by the hardware instruction; results below 2^-126 flush to 0.
__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

// ---------------------------------------------------------------------------
// score_kernel
// ---------------------------------------------------------------------------
// Launches over many models of which only a few have a queue (a scheduling
// round scores the idle models only) list those models in their arguments
// and launch workgroups for them alone: workgroups that only find an empty
// queue and exit would still hold the dispatch slots for a memory round
// trip each.
constexpr int kMaxActive = 256;

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
    const int32_t* sup;        // [M][nbs][C][2] first / last bin with mass, or NULL
    const double* cost;        // [N] miss cost per request, or NULL (1)
    const double* c0;          // affine mode: [M] fixed batch overhead (ms); else NULL
    const double* c1;          // affine mode: [M] per-member slope; NULL = tabulated mode
    const float* fill;         // [2][16] zeros, ones (the context's stand-in rows)
    float* psum;               // affine mode: [M][np_e][maxcap] panel sums of 1 - G
    int np_e;                  // panels of those sums (emax_kernel's panel width)
    int* err;
    int defer;                 // 1: write the priority sum to S, leave E[L_B] and S to the selection
    int chunk;                 // prefix lengths scored per workgroup (0: all of them)
    int nchunk;                // workgroups per (model, batch size)
    double b;
    int M, C, K, nbs, rect, maxcap;
    int Mg;                    // models the grid covers: M, or the listed ones
    int compact;               // 1: grid model i is act[i]
    int bs[ORLOJ_MAX_BATCH_SIZES];
    int act[kMaxActive];       // the models with a non-empty queue (compact)
};

__device__ __forceinline__ int grid_model(const ScoreArgs& a, unsigned i) {
    return a.compact ? a.act[i] : (int)i;
}

// Stand-in rows for lane chunks that lie wholly outside a row's support:
// there every entry of 1 - F is exactly 0 (past the last bin with mass) or
// exactly 1 (before the first), so the update G <- G - G (1 - F) gives the
// same bits whether it reads the table or these constants.  They live in a
// small buffer of the context (kFillFloats floats: 16 zeros, then 16 ones),
// stay in cache, and keep every row load a plain global load.
constexpr int kFillFloats = 32;

// Per-member lookup plan (it depends on the deadline only, not on the step).
//
// The bins are swept in panels of 64 CPL bins (one chunk of CPL
// consecutive bins per lane); a member with deadline bin k is handled in the
// pass over its home panel hp (the panel of bin k; dead requests in pass 0,
// beyond-the-grid requests in the last pass).  Deadline order makes the
// members of each panel a contiguous range.  In that pass, at step n, the
// wave has
//   W     = Z at the last bin of panel hp-1   (discounted prefix carried in)
//   gl    = G at the last bin of panel hp-1
//   A[]   = in-panel discounted scan of the lane chunk totals
//   g[], zq[]  snapshot of G (fp64) and of each chunk's quarter-end prefixes
// and assembles
//   G(x_k)     = g[o0]
//   G(x_{k+1}) = g[o1]
//   Z(k-2) = cW W + cG gl + cA f[oa] + fq f[oz] + z4
//   z4     = the in-quarter discounted prefix of g[o4 + 0 .. rq] (Horner)
//   P   = G(x_k) + theta (G(x_{k+1}) - G(x_k))          (fp64)
//   num = cg (G(x_k) - (1 - d) Z(k-2)) + psi (G(x_{k+1}) - G(x_k))
// where g is the fp64 area of the workgroup's LDS (the snapshot and three
// constant slots: 0, 1 and gl, the last written at every scoring step) and
// f its float area (zq, A and a zero).  The plan resolves every case into an
// offset: G(x_k) is gl when bin k-1 lies in the previous panel, 0 when
// k = 0; both G values are 0 when the deadline has passed and 1 when it lies
// beyond the grid; a term the member does not need has weight 0 and reads a
// finite slot.  So the lookup takes no branch.  P and the expected finish
// count are formed in fp64 from the fp64 snapshot and an fp64 theta (a
// float pair); the priority's terms are fp32.  A plan is 48 bytes, so that
// 64 of them and the fp64 snapshot of a 1024-bin panel leave room for
// twelve waves per compute unit.
constexpr int kMaxPanels = 63;   // panels per row (their first members sit in one lane each)

struct Member {
    uint8_t hp;     // home panel
    uint8_t rq;     // bin k-2's place in its quarter (kNoQuarter: no quarter term)
    uint16_t o0;    // LDS byte offsets of G(x_k),
    uint16_t o1;    //   G(x_{k+1}),
    uint16_t o4;    //   the quarter holding bin k-2,
    uint16_t oz;    //   the quarter-end prefix before that quarter,
    uint16_t oa;    //   and the in-panel scan before bin k-2's lane
    float cW;       // weight of W
    float cG;       // weight of gl
    float cA;       // weight of f[oa]
    float fq;       // weight of f[oz]
    float theta;    // position inside bin k (rounded to fp32) ...
    float thlo;     //   ... and the rest of the fp64 position
    float cg;       // gamma exp(-b theta w), or gamma exp(-b (tau - K w))
    float psi;      // (1 - exp(-b theta w)) / (b w)
    float cost;     // the request's miss cost (weights its priority)
};
static_assert(sizeof(Member) == 48, "member plan size");
constexpr int kNoQuarter = 0xff;

template <int CPL>
struct Quarters {
    static constexpr int QW = CPL < 4 ? CPL : 4;   // bins per quarter
    static constexpr int NQ = CPL / QW;            // quarters per lane chunk
};

// LDS layout of one workgroup (one wave), byte offsets:
//   GD  g[64 CPL]   snapshot of G over the current panel, fp64; pairs of
//                   bins interleaved over the lanes, bins j, j+1 of lane l
//                   at pair slot 64 (j/2) + (l ^ (j/2)): a lane writes 16
//                   consecutive bytes, each write is a permutation of 64
//                   consecutive slots, and the members that read the
//                   different pairs of one lane chunk hit different banks
//   KD  k[4]        constant slots (fp64): 0, 1, gl (G carried in), unused
//   ZQ  zq[64 NQ]   quarter-end discounted prefixes of each lane chunk (f32)
//   AA  A[64]       in-panel discounted scan of the lane chunk totals (f32)
//   FZ  4 zeros     (f32) what a weight-0 float term reads
//   MEM mem[maxcap] Member plans
template <int CPL>
struct ScoreLds {
    static constexpr int GD = 0;
    static constexpr int KD = 8 * 64 * CPL;
    static constexpr int ZQ = KD + 32;
    static constexpr int AA = ZQ + 4 * 64 * Quarters<CPL>::NQ;
    static constexpr int FZ = AA + 4 * 64;
    static constexpr int MEM = FZ + 16;
    static_assert(MEM % 16 == 0 && MEM < 65536, "LDS layout");
};
template <int CPL>
__host__ __device__ constexpr size_t score_fixed_bytes() { return (size_t)ScoreLds<CPL>::MEM; }
__host__ __device__ constexpr size_t score_bytes_per_member() { return sizeof(Member); }

// Byte offset of the snapshot's bin r (bin offset inside the panel).
template <int CPL>
__device__ __forceinline__ int snap_byte(int r) {
    if constexpr (CPL >= 2) {
        const int l = r / CPL, j = r - l * CPL, jp = j >> 1;
        return 8 * ((jp * 64 + (l ^ jp)) * 2 + (j & 1));
    } else {
        return 8 * r;
    }
}

// Branch-free load of one lane's CPL entries starting at p.  EXACT: the
// panels tile the row exactly, so the loads are whole float4s.  Otherwise
// offsets past lim (the row's last entry) are clamped to it and their
// values are masked at use.  Every load is issued unconditionally so the
// prefetch ring keeps fixed registers.
template <int CPL, bool EXACT>
__device__ __forceinline__ void load_chunk(float (&v)[CPL], const float* __restrict__ p, int lim) {
    if constexpr (EXACT && CPL % 4 == 0) {
        const float4* r4 = reinterpret_cast<const float4*>(p);
#pragma unroll
        for (int j = 0; j < CPL / 4; ++j) {
            const float4 t = r4[j];
            v[4 * j] = t.x; v[4 * j + 1] = t.y; v[4 * j + 2] = t.z; v[4 * j + 3] = t.w;
        }
    } else {
#pragma unroll
        for (int j = 0; j < CPL; ++j) v[j] = p[min(j, lim)];
    }
}

// Value of lane 63 in every lane.
__device__ __forceinline__ float lane63(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 63));
}
__device__ __forceinline__ double lane63(double v) {
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, 63);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), 63);
    return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

// Value of lane L (a constant) in every lane.
__device__ __forceinline__ float lane_read(float v, int L) {
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), L));
}
__device__ __forceinline__ double lane_read(double v, int L) {
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, L);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), L);
    return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

// Same-wave LDS ordering point: keeps the compiler from moving LDS accesses
// across it (the hardware already executes one wave's LDS operations in
// order).
__device__ __forceinline__ void wave_lds_fence() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
}

template <bool B>
struct BoolTag { static constexpr bool value = B; };

// Per-step state carried from one panel pass to the next, spread over the
// lanes: step n lives in lane n % 64 of register n / 64.  Reads and writes
// take a wave-uniform step index.
template <int CR>
struct LaneCarry {
    float v[CR];
    __device__ __forceinline__ void zero() {
#pragma unroll
        for (int r = 0; r < CR; ++r) v[r] = 0.0f;
    }
    __device__ __forceinline__ float get(int n) const {
        float out = 0.0f;
#pragma unroll
        for (int r = 0; r < CR; ++r) {
            const float x = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v[r]), n & 63));
            out = (n >> 6) == r ? x : out;
        }
        return out;
    }
    __device__ __forceinline__ void set(int n, float x) {
        const int l = (int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
#pragma unroll
        for (int r = 0; r < CR; ++r) v[r] = (l + 64 * r) == n ? x : v[r];
    }
    // step n's value += x (wave-uniform), added by the lane that holds it
    __device__ __forceinline__ void add(int n, float x) {
        const int l = (int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
#pragma unroll
        for (int r = 0; r < CR; ++r) v[r] = (l + 64 * r) == n ? v[r] + x : v[r];
    }
    // value of step r * 64 + lane
    __device__ __forceinline__ float mine(int r) const { return v[r]; }
};

template <int CR>
struct LaneCarry64 {
    LaneCarry<CR> lo, hi;
    __device__ __forceinline__ void zero() { lo.zero(); hi.zero(); }
    __device__ __forceinline__ double get(int n) const {
        const uint32_t l = __builtin_bit_cast(uint32_t, lo.get(n));
        const uint32_t h = __builtin_bit_cast(uint32_t, hi.get(n));
        return __builtin_bit_cast(double, ((uint64_t)h << 32) | l);
    }
    __device__ __forceinline__ void set(int n, double x) {
        const uint64_t u = __builtin_bit_cast(uint64_t, x);
        lo.set(n, __builtin_bit_cast(float, (uint32_t)u));
        hi.set(n, __builtin_bit_cast(float, (uint32_t)(u >> 32)));
    }
    __device__ __forceinline__ double mine(int r) const {
        const uint32_t l = __builtin_bit_cast(uint32_t, lo.mine(r));
        const uint32_t h = __builtin_bit_cast(uint32_t, hi.mine(r));
        return __builtin_bit_cast(double, ((uint64_t)h << 32) | l);
    }
    // step n's value += x (wave-uniform), added by the lane that holds it:
    // the same fp64 addition as get + set, without reading the lane out
    __device__ __forceinline__ void add(int n, double x) {
        const int l = (int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
#pragma unroll
        for (int r = 0; r < CR; ++r) {
            const double v = mine(r) + x;
            const uint64_t u = __builtin_bit_cast(uint64_t, v);
            const bool own = (l + 64 * r) == n;
            lo.v[r] = own ? __builtin_bit_cast(float, (uint32_t)u) : lo.v[r];
            hi.v[r] = own ? __builtin_bit_cast(float, (uint32_t)(u >> 32)) : hi.v[r];
        }
    }
};

// One workgroup (a single wave) scores every prefix of one model's queue at
// one batch size.  Lane l of pass p owns bins [(p*64 + l) CPL, +CPL) and
// keeps their batch CDF G_n(x_{k+1}) = prod_{i <= n} F_{c_i}(x_{k+1}) as an
// fp64 running product over the steps n (the table holds 1 - F, so a step
// is one fma per bin).  Per step: the sums of 1 - G and the discounted
// prefix over the panel (4-bin quarters keep the dependency chains short,
// a DPP scan joins the lanes), the carries into the next panel, and, if
// some member's deadline falls in this panel, a snapshot in LDS that the
// same wave then reads to score those members.  Rows are prefetched PF
// iterations ahead through a register ring.  Panels past the last member's
// deadline need only the sums of 1 - G: a second, lean loop takes them
// (tabulated mode).  A workgroup may take a chunk of the steps only, after
// warm-up steps that rebuild G over the steps before it.
#ifndef ORLOJ_SCORE_PREFETCH
#define ORLOJ_SCORE_PREFETCH 2   // iterations a row is loaded ahead of its use
#endif
#ifndef ORLOJ_SPLIT_PREFETCH
#define ORLOJ_SPLIT_PREFETCH 4   // the same in launches with an E pre-pass
#endif
#ifndef ORLOJ_EONLY_PREFETCH
#define ORLOJ_EONLY_PREFETCH 3   // iterations ahead in the E-only panels' loop
#endif
#ifndef ORLOJ_EONLY_CACHE
#define ORLOJ_EONLY_CACHE 2      // classes whose slices the E-only loop keeps in registers
#endif
#ifndef ORLOJ_EONLY_LDS_CACHE
#define ORLOJ_EONLY_LDS_CACHE 3  // further classes whose slices it keeps in LDS
#endif
#ifndef ORLOJ_WARMUP_PREFETCH
#define ORLOJ_WARMUP_PREFETCH 4  // steps ahead in a chunk's warm-up loop
#endif
template <int CPL, int PF, bool EXACT, int CR, bool AFF, bool ESPLIT>
__device__ __forceinline__ void score_wave(const ScoreArgs& a, const unsigned bid) {
    static_assert(ESPLIT || !AFF, "the affine mode takes its E sums from emax_kernel");
    using Q = Quarters<CPL>;
    constexpr int PW = 64 * CPL;                   // bins per panel
    extern __shared__ __align__(16) unsigned char smem_raw[];
    using L = ScoreLds<CPL>;
    double* s_kd = reinterpret_cast<double*>(smem_raw + L::KD);   // constant slots
    float* s_zq = reinterpret_cast<float*>(smem_raw + L::ZQ);
    float* s_A = reinterpret_cast<float*>(smem_raw + L::AA);
    float* s_fz = reinterpret_cast<float*>(smem_raw + L::FZ);
    Member* s_mem = reinterpret_cast<Member*>(smem_raw + L::MEM);   // CR > 1 only
    const int maxcap = a.maxcap;

    const int lane = threadIdx.x;

    // Largest batch sizes first, and their last chunks first: those
    // workgroups run longest.
    const unsigned per_bs = (unsigned)a.Mg * (unsigned)a.nchunk;
    const int bi = a.nbs - 1 - (int)(bid / per_bs);
    const unsigned rem = bid % per_bs;
    const int kc = a.nchunk - 1 - (int)(rem / (unsigned)a.Mg);
    const int q = grid_model(a, rem % (unsigned)a.Mg);
    const int64_t q0 = a.queue_off[q];
    const int64_t N = a.queue_off[q + 1] - q0;
    const int bsz = a.bs[bi];
    const int64_t cap64 = a.rect ? N : (N < bsz ? N : (int64_t)bsz);
    if (cap64 <= 0 || cap64 > maxcap || cap64 > 64 * CR) return;   // the host sizes both
    const int ncap = (int)cap64;
    // This workgroup scores prefix lengths n0 + 1 .. n1 (steps n0 .. n1 - 1).
    // A launch too small to fill the chip splits them into chunks: the
    // steps before n0 only rebuild G (warm-up steps), with the same fma
    // sequence, so every chunk gives the bits a single workgroup would.
    const int CH = a.chunk > 0 ? a.chunk : ncap;
    const int n0 = kc * CH;
    if (n0 >= ncap) return;
    const int n1 = min(ncap, n0 + CH);
    // The longest workgroups set a saturated launch's length (their steps
    // run one after another while shorter ones share their SIMD): they
    // take issue priority over the short ones, graded by their step count.
    if (n1 - n0 >= 48) __builtin_amdgcn_s_setprio(3);
    else if (n1 - n0 >= 32) __builtin_amdgcn_s_setprio(2);
    else if (n1 - n0 >= 16) __builtin_amdgcn_s_setprio(1);

    // Affine mode (Eq. (3)): a batch of size s whose slowest member takes l
    // runs c0 + c1 s l, so its latency histogram is the base grid's with
    // bins c1 s w wide, shifted by c0.  Everything below works on that
    // grid: the bin width is c1 s w, the time left is tau - c0, and
    // E[L_B] = c0 + c1 s E[max] (Eq. (5)).  Tabulated mode: c0 = 0, width w.
    // The product over members is the same for every batch size there, so
    // E[max]'s sums come from emax_kernel, and a wave walks only the panels
    // up to its last member's home panel.
    const double wq = a.width[q];
    double c0q = 0.0;
    bool aok = true;
    double w = wq;
    if constexpr (AFF) {
        c0q = a.c0[q];
        const double c1 = a.c1[q];
        aok = c0q >= 0.0 && c0q < HUGE_VAL && c1 > 0.0 && c1 < HUGE_VAL;
        w = c1 * (double)bsz * wq;
    }
    const bool wok = wq > 0.0 && wq < HUGE_VAL && aok && w > 0.0 && w < HUGE_VAL;   // else a data error
    const double nowq = a.now[q];
    const double b = a.b;
    const double bw = b * w;
    const int K = a.K;
    const int NP = (K + PW - 1) / PW;

    const double d64 = exp(-bw);                      // discount per bin
    const float log2d = (float)(-bw * 1.4426950408889634);
    const float gamma = (float)(-expm1(-bw) / bw);   // (1 - d) / (b w)
    const float omd = (float)(-expm1(-bw));          // 1 - d

    // ---- member lookup plans (fp64 time relative to now).  `check` flags
    // the member's data errors (once per member and workgroup).
    auto make_plan = [&](int m, bool check) -> Member {
        int c = a.cls[q0 + m];
        const double D = a.deadline[q0 + m];
        double cm = a.cost ? a.cost[q0 + m] : 1.0;
        if (check) {
            int flag = 0;
            if (c < 0 || c >= a.C) flag |= kErrClassRange;
            if (isnan(D)) flag |= kErrDeadlineNaN;
            if (m > 0 && D < a.deadline[q0 + m - 1]) flag |= kErrUnsorted;
            if (m == 0 && isnan(nowq)) flag |= kErrNowNaN;
            if (m == 0 && !(wq > 0.0 && wq < HUGE_VAL)) flag |= kErrWidth;
            if (m == 0 && !aok) flag |= kErrAffine;
            if (!(cm >= 0.0 && cm < HUGE_VAL)) flag |= kErrCost;
            if (flag) atomicOr(a.err, flag);
        }
        if (c < 0 || c >= a.C) c = 0;
        if (!(cm >= 0.0 && cm < HUGE_VAL)) cm = 0.0;
        Member mb;
        mb.cost = (float)cm;
        mb.rq = (uint8_t)kNoQuarter;
        // byte offsets: KD reads 0, KD + 8 reads 1, KD + 16 reads gl; FZ
        // reads a float 0
        int hp = 0, o0 = L::KD, o1 = L::KD, o4 = 0, oz = L::FZ, oa = L::FZ;
        mb.cW = mb.cG = mb.cA = mb.fq = 0.0f;
        mb.theta = mb.thlo = mb.cg = mb.psi = 0.0f;
        const double tau = D - nowq - c0q;
        int kz = -1;   // bin whose discounted prefix Z the priority needs
        if (tau > 0.0 && wok) {
            const double u = tau / w;
            if (u >= (double)K) {                  // beyond the grid: P = 1
                o0 = o1 = L::KD + 8;
                mb.cg = gamma * (float)exp(-b * (tau - (double)K * w));
                hp = NP - 1;
                kz = K - 2;
            } else {
                const double kf = floor(u);
                const double th = u - kf;
                const int k = (int)kf;
                hp = k / PW;
                mb.theta = (float)th;
                mb.thlo = (float)(th - (double)mb.theta);
                mb.cg = gamma * (float)exp(-b * th * w);
                mb.psi = (float)(-expm1(-b * th * w) / bw);
                o1 = snap_byte<CPL>(k - hp * PW);
                if (k >= 1) o0 = k - 1 >= hp * PW ? snap_byte<CPL>(k - 1 - hp * PW) : L::KD + 16;
                kz = k - 2;
            }
        }
        if (kz >= 0) {
            const int p0 = hp * PW;                // first bin of the home panel
            if (kz >= p0) {
                const int r = kz - p0, l = r / CPL, j = r - l * CPL;
                const int qq = j / Q::QW, rq = j - qq * Q::QW;
                mb.cW = hp > 0 ? exp2f(log2d * (float)(kz - p0 + 1)) : 0.0f;
                if (l > 0) {
                    oa = L::AA + 4 * (l - 1);
                    mb.cA = exp2f(log2d * (float)(j + 1));
                }
                if (qq > 0) {
                    oz = L::ZQ + 4 * (l * Q::NQ + qq - 1);
                    mb.fq = exp2f(log2d * (float)(rq + 1));
                }
                o4 = snap_byte<CPL>(r - rq);       // first bin of the quarter
                mb.rq = (uint8_t)rq;
            } else if (kz == p0 - 1) {             // last bin of the previous panel
                mb.cW = 1.0f;
            } else {                               // kz = p0 - 2: step back one bin
                mb.cW = (float)exp(bw);
                mb.cG = -(float)exp(bw);
            }
        }
        mb.hp = (uint8_t)hp;
        mb.o0 = (uint16_t)o0; mb.o1 = (uint16_t)o1; mb.o4 = (uint16_t)o4;
        mb.oz = (uint16_t)oz; mb.oa = (uint16_t)oa;
        return mb;
    };
    // Everything from here on is compiled twice: for the waves whose members
    // all lie in panel 0 (ONE: no carries between panel passes, every step
    // scores members; at configuration 5 that is every wave) and for the
    // rest.  The branch comes before any per-lane state, so the two versions
    // share no registers' worth of live values.  The last member's plan
    // gives its home panel, as it does below.
    const int lastp = __builtin_amdgcn_readfirstlane((int)make_plan(n1 - 1, false).hp);
    auto rest = [&](auto one_tag) {
        constexpr bool ONE = decltype(one_tag)::value;
        // The prologue is a chain of memory round trips, which the launches too
        // small to fill the chip wait on: the loads that do not depend on each
        // other are issued together.  This batch size's block of candidates and
        // member slots starts after those of the batch sizes before it (one per
        // lane, summed across the wave).
        int64_t cand = a.cand_off[q], prob = a.prob_off[q];
        {
            uint64_t dc = 0, dp = 0;
            for (int j0 = 0; j0 < bi; j0 += 64) {
                const int j = j0 + lane;
                if (j < bi) {
                    const int64_t c = a.rect ? N : (N < a.bs[j] ? N : (int64_t)a.bs[j]);
                    dc += (uint64_t)c;
                    dp += (uint64_t)(c * (c + 1) / 2);
                }
            }
            cand += (int64_t)wave_sum_u64(dc, lane);
            prob += (int64_t)wave_sum_u64(dp, lane);
        }
        // rows of this (model, batch size); affine mode has one set per model
        const size_t qb = AFF ? (size_t)q : (size_t)q * (size_t)a.nbs + (size_t)bi;
        const float* tab_qb = a.tab + qb * (size_t)a.C * (size_t)K;

        // class and support of member n in lane n % 64 of register n / 64, and
        // the members' plans, in one pass
        LaneCarry<CR> cls_r, lo_r, hi_r;
        const int32_t* sup_qb = a.sup ? a.sup + qb * (size_t)a.C * 2 : nullptr;
#pragma unroll
        for (int r = 0; r < CR; ++r) {
            const int m = r * 64 + lane;
            int c = a.cls[q0 + min(m, n1 - 1)];
            if (c < 0 || c >= a.C) c = 0;                     // flagged by its plan
            cls_r.v[r] = __builtin_bit_cast(float, c);
            lo_r.v[r] = __builtin_bit_cast(float, sup_qb ? sup_qb[2 * c] : 0);
            hi_r.v[r] = __builtin_bit_cast(float, sup_qb ? sup_qb[2 * c + 1] : K);
            if (m < n1) s_mem[m] = make_plan(m, true);
        }
        if (lane == 0) {
            s_kd[0] = 0.0;
            s_kd[1] = 1.0;
            s_kd[2] = 0.0;
            s_kd[3] = 0.0;
        }
        if (lane < 4) s_fz[lane] = 0.0f;
        wave_lds_fence();
        // Home panel of the last member (the latest deadline): past it no member
        // needs G or the discounted prefix, only E[L_B] needs the sums of 1 - G.
        // The main loop walks the panels up to LASTP; the tabulated mode then
        // sums the rest (E-only panels) in a loop of its own, the affine mode
        // takes them from emax_kernel.
        const int LASTP = ONE ? 0 : __builtin_amdgcn_readfirstlane((int)s_mem[n1 - 1].hp);
        const int NPW = LASTP + 1;
        // first member of each panel p in lane p (home panels are non-decreasing
        // in m): counted up to LASTP; every member's home panel lies before the
        // later ones, so their lanes hold n1
        int mlo_r = n1;
        for (int p = 0; p <= LASTP; ++p) {
            int cnt = 0;
            for (int m0 = 0; m0 < n1; m0 += 64) {
                const int m = m0 + lane;
                const bool below = m < n1 && s_mem[m].hp < p;
                cnt += __builtin_popcountll(__ballot(below));
            }
            mlo_r = lane == p ? cnt : mlo_r;
        }

        // ---- scan constants
        float rp[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) rp[i] = exp2_hw(log2d * (float)(CPL << i));
        const float w15 = exp2_hw(log2d * (float)(CPL * ((lane & 15) + 1)));
        const float w31 = exp2_hw(log2d * (float)(CPL * (lane >= 32 ? lane - 31 : 0)));
        const float dQ = exp2_hw(log2d * (float)Q::QW);
        const float dq1 = exp2f(log2d);                   // d in fp32
        // A member's in-quarter discounted prefix up to bin k-2, the quarter's
        // r-th bin being bin k-2 (rq = r <= 3): sum over j <= rq of
        // d^(rq - j) G_j, formed as a dot product with these weights (all 0
        // when the member needs no quarter term, rq = kNoQuarter).
        const float dq2 = dq1 * dq1, dq3 = dq2 * dq1;
        auto quarter_weights = [&](int rq, float (&wv)[4]) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int e = rq - r;
                wv[r] = (e < 0 || rq > 3) ? 0.0f : e == 0 ? 1.0f : e == 1 ? dq1 : e == 2 ? dq2 : dq3;
            }
        };
        const float dPW = exp2_hw(log2d * (float)PW);

        // Load the lane chunk starting at bin c0 of member n's row; chunks wholly
        // outside the row's support, and every chunk when `none` (the row's
        // values cannot change G), read a constant row instead.
        // The member's support bounds go to lo / hi: the ring slot keeps them
        // for the step that uses the row.
        auto load_step = [&](float (&v)[CPL], int n, int c0, bool none, int& lo, int& hi) {
            const int c = __builtin_bit_cast(int, cls_r.get(n));
            lo = __builtin_bit_cast(int, lo_r.get(n));
            hi = __builtin_bit_cast(int, hi_r.get(n));
            // The affine mode's solo table (M x C rows) stays in the Infinity
            // Cache, so it reads every chunk rather than spend a per-lane test
            // and select on each load; entries outside the support are exactly
            // 1 and 0 either way.
            const bool ones = !AFF && !none && c0 + CPL <= lo, zeros = none || (!AFF && c0 >= hi);
            const float* src = tab_qb + (size_t)c * (size_t)K + c0;
            int lim = K - 1 - c0;
            if (ones || zeros) {
                src = a.fill + (ones ? 16 : 0);
                lim = CPL - 1;
            }
            load_chunk<CPL, EXACT>(v, src, lim);
        };

        LaneCarry<CR> cW, cN;
        LaneCarry64<CR> cE, cP, cGl;
        cW.zero(); cGl.zero(); cN.zero(); cE.zero(); cP.zero();

        // One flat loop over (panel p, step n in [ns, n1)), n fastest, padded at
        // the end to a multiple of PF with ghost iterations (p == NP) so that
        // ring slot i always holds iteration it0 + i.  The row of iteration
        // it + PF is loaded PF iterations ahead; (p, n) and the prefetch
        // position advance by counting.  A chunk of a split launch rebuilds G
        // over the steps before n0 (warm-up): in a loop of its own at each pass
        // start when its E sums come from emax_kernel (WARM_LOOP: the loop's
        // deeper ring costs registers, which the launches that fill the chip
        // cannot spare), else as iterations of this loop that update G only.
        constexpr bool WARM_LOOP = ESPLIT && !AFF;
        const int ns = WARM_LOOP ? n0 : 0;
        const int total = NPW * (n1 - ns);
        const int iters = (total + PF - 1) / PF * PF;
        const int base = lane * CPL;

        double Gacc[CPL];
        float buf[PF][CPL];
        int slo[PF], shi[PF];                                 // the slots' support bounds
        int pf_p = 0, pf_n = ns;                              // prefetch position
#pragma unroll
        for (int i = 0; i < PF; ++i) {
            load_step(buf[i], pf_n, pf_p * PW + base, false, slo[i], shi[i]);
            // keep the priming loads in ring order, as the loop issues them
            __builtin_amdgcn_sched_barrier(0);
            if (++pf_n == n1) { pf_n = ns; pf_p = min(pf_p + 1, NPW - 1); }
        }
        int p = 0, n = ns;
        int mlo = __builtin_amdgcn_readlane(mlo_r, 0);
        int mend = __builtin_amdgcn_readlane(mlo_r, 1);
        // Trivial steps.  Where a panel lies wholly past the last bin with mass
        // of member n's row (every 1 - F there is exactly 0), or where G is
        // already exactly 0 over the whole panel (an earlier member's row had
        // no mass up to its end), step n leaves G unchanged bit for bit; if no
        // member of the panel needs scoring at that step, its panel sums are
        // those of step n-1 and the update, its loads and its reductions are
        // skipped.
        bool pass_zero = false;                  // G == 0 on every bin of this pass's panel
        Member pass_mb;                          // CR == 1: this lane's member of the pass
        double pass_th = 0.0;                    //   and its position in bin k, fp64,
        float pass_wq[4] = {0.0f, 0.0f, 0.0f, 0.0f};   // and its quarter weights
        bool pass_valid = false;
        float etot_prev = 0.0f, T_prev = 0.0f;
        double gl_prev = 0.0;

        // Warm-up: G over steps 0 .. n0-1 of panel pp (the product only, the
        // same fma per bin and step as a scored step, so the same bits; a step
        // whose row cannot change G multiplies by an exact 0 or finds G = 0),
        // with rows loaded PFW steps ahead: these steps are short and would
        // otherwise wait on their loads.  Leaves pass_zero for the steps after.
        constexpr int PFW = ORLOJ_WARMUP_PREFETCH;
        auto warm_up = [&](int pp) {
            const int p0w = pp * PW, pbw = p0w + base;
            float wb[PFW][CPL];
            int wlo[PFW], whi[PFW];
            bool zero = false;                   // G == 0 over the panel
#pragma unroll
            for (int i = 0; i < PFW; ++i) {
                load_step(wb[i], min(i, n0 - 1), pbw, false, wlo[i], whi[i]);
                __builtin_amdgcn_sched_barrier(0);
            }
            for (int w0 = 0; w0 < n0; w0 += PFW) {
#pragma unroll
                for (int i = 0; i < PFW; ++i) {
                    const int nw = w0 + i;
                    if (nw < n0) {
#pragma unroll
                        for (int j = 0; j < CPL; ++j) {
                            const float t = (EXACT || pbw + j < K) ? wb[i][j] : 0.0f;
                            Gacc[j] = fma(-Gacc[j], (double)t, Gacc[j]);
                        }
                        zero = zero || min(p0w + PW, K) <= wlo[i];
                    }
#pragma unroll
                    for (int j = 0; j < CPL; ++j) asm volatile("" : "+v"(Gacc[j])::"memory");
                    load_step(wb[i], min(nw + PFW, n0 - 1), pbw, zero, wlo[i], whi[i]);
                }
            }
            pass_zero = zero;
        };

        static_assert(PF % 2 == 0, "steps are reduced in pairs");
        for (int it0 = 0; it0 < iters; it0 += PF) {
            // each scoring step's member sums (0 in lanes without a member) and
            // its index (-1: no member scored)
            double redP[PF];
            float redN[PF];
            int red_n[PF];
#pragma unroll
            for (int i = 0; i < PF; ++i) redP[i] = 0.0, redN[i] = 0.0f, red_n[i] = -1;
#pragma unroll
            for (int i = 0; i < PF; ++i) {
                if (n == ns) {
                    // a real branch (the asm keeps it from becoming selects)
                    asm volatile("" ::: "memory");
#pragma unroll
                    for (int j = 0; j < CPL; ++j) Gacc[j] = 1.0;
                    pass_zero = false;
                    if constexpr (WARM_LOOP) {
                        if (n0 > 0 && p < NPW) warm_up(p);
                    }
                    if constexpr (CR == 1) {
                        // at most 64 members: lane l scores member mlo + l of this
                        // pass at every step, so its plan is read from LDS once
                        pass_valid = mlo + lane < mend;
                        pass_mb = s_mem[min(mlo + lane, n1 - 1)];
                        pass_th = (double)pass_mb.theta + (double)pass_mb.thlo;
                        quarter_weights(pass_mb.rq, pass_wq);
                    }
                }
                const int p0 = ONE ? 0 : p * PW;              // first bin of the panel
                const int pbase = p0 + base;                  // first bin of this lane chunk
                const int hi_n = shi[i];
                const int lo_n = slo[i];
                // members of this panel among the first n+1 (ONE: all of them)
                const int mhi = ONE ? n + 1 : min(mend, n + 1);
                const bool real = n >= n0;                    // else a warm-up step
                const bool due = real && (ONE || mlo < mhi);  // some member is scored at this step
                // G unchanged by this step (a panel past the row's support, or G
                // already 0 on it): a warm-up step then does nothing, a scored
                // step after the chunk's first reuses the previous step's sums
                const bool unchanged = pass_zero || p0 >= hi_n;
                const bool skip = p >= NPW || (real ? (n > n0 && unchanged && !due) : unchanged);
                // G <- G * F = G - G (1 - F), in fp64; per-quarter sums
                double gs[Q::QW];
                float zqv[Q::NQ];
                if (!skip) {
#pragma unroll
                    for (int qq = 0; qq < Q::NQ; ++qq) {
                        double zz = 0.0;
#pragma unroll
                        for (int r = 0; r < Q::QW; ++r) {
                            const int j = qq * Q::QW + r;
                            const float t = (EXACT || pbase + j < K) ? buf[i][j] : 0.0f;
                            Gacc[j] = fma(-Gacc[j], (double)t, Gacc[j]);
                            if constexpr (!ESPLIT) gs[r] = qq == 0 ? Gacc[j] : gs[r] + Gacc[j];
                            zz = r == 0 ? Gacc[j] : fma(zz, d64, Gacc[j]);
                        }
                        zqv[qq] = (float)zz;
                    }
                }
                // the slot is refilled only after the update has consumed it, so
                // the ring keeps its registers (no copies, no wait on the loads
                // just issued)
#pragma unroll
                for (int j = 0; j < CPL; ++j) asm volatile("" : "+v"(Gacc[j])::"memory");
                // G == 0 over the pass from here on: later steps of it need no row
                const bool zero_after = pass_zero || min(p0 + PW, K) <= lo_n;
                load_step(buf[i], pf_n, pf_p * PW + base, zero_after && pf_p == p, slo[i], shi[i]);
                if (++pf_n == n1) { pf_n = ns; pf_p = ONE ? 0 : min(pf_p + 1, NPW - 1); }
                if (p < NPW && real) {                        // else a ghost or warm-up iteration
                    float etot = etot_prev, T = T_prev;
                    double glast_here = gl_prev;
                    // carries in from the previous panel pass (zero in the first)
                    float Win = 0.0f;
                    double glin64 = 0.0;
                    if (!ONE && p > 0) {
                        Win = cW.get(n);
                        glin64 = cGl.get(n);
                    }
                    const float glin = (float)glin64;
                    float A = 0.0f;
                    if (!skip) {
                        // quarter ends of the in-chunk discounted prefix, and its total
                        float zc = zqv[0];
#pragma unroll
                        for (int qq = 1; qq < Q::NQ; ++qq) {
                            zc = fmaf(zc, dQ, zqv[qq]);
                            zqv[qq] = zc;
                        }
                        A = wave_wscan(zc, rp, w15, w31);
                        if (!ONE && p < LASTP) {              // carried into the next pass
                            T = lane63(A);                    // discounted prefix at the panel end
                            T_prev = T;
                        }
                    }
                    if (!skip) {
                        if constexpr (!ESPLIT) {
                            double gsum = gs[0];
#pragma unroll
                            for (int r = 1; r < Q::QW; ++r) gsum += gs[r];
                            // 1 - G summed over the lane's bins (padding bins hold G = 1)
                            const float e = (float)((double)CPL - gsum);
                            etot = lane63(wave_scan_sum(e));
                        }
                        if (!ONE && p < LASTP) {              // carried into the next pass
                            glast_here = lane63(Gacc[CPL - 1]);
                            gl_prev = glast_here;
                        }
                        etot_prev = etot;

                        if (due) {
                            // snapshot of G over the panel, fp64, pairs of bins
                            // interleaved over the lanes (16-byte writes)
                            if constexpr (CPL >= 2) {
#pragma unroll
                                for (int j = 0; j < CPL; j += 2) {
                                    const int pair = (j >> 1) * 64 + (lane ^ (j >> 1));
                                    *reinterpret_cast<double2*>(smem_raw + L::GD + 16 * pair) =
                                        make_double2(Gacc[j], Gacc[j + 1]);
                                }
                            } else {
                                *reinterpret_cast<double*>(smem_raw + L::GD + 8 * lane) = Gacc[0];
                            }
#pragma unroll
                            for (int qq = 0; qq < Q::NQ; ++qq) s_zq[lane * Q::NQ + qq] = zqv[qq];
                            s_A[lane] = A;
                            if (!ONE && lane == 0) s_kd[2] = glin64;   // (ONE: stays 0)
                            wave_lds_fence();
                            double pP = 0.0;
                            float pN = 0.0f;
                            const int nn = n + 1;
                            auto score_member = [&](const Member& mb, int m, double th, const float (&wq4)[4]) {
                                const unsigned char* f = smem_raw;
                                auto atf = [&](int off) { return *reinterpret_cast<const float*>(f + off); };
                                auto atd = [&](int off) { return *reinterpret_cast<const double*>(f + off); };
                                const double gk64 = atd(mb.o0);
                                const double gk164 = atd(mb.o1);
                                const float al0 = atf(mb.oa);
                                const float zq0 = atf(mb.oz);
                                // the quarter's G values (fp32 terms of the priority)
                                float g4[4];
                                if constexpr (Q::QW == 4) {
                                    const double2 t0 = *reinterpret_cast<const double2*>(f + mb.o4);
                                    // the quarter's second pair: its slot follows
                                    // the first's by 64, with the lane index's
                                    // low bit flipped (the first pair's index is even)
                                    const double2 t1 = *reinterpret_cast<const double2*>(f + ((mb.o4 + 16 * 64) ^ 16));
                                    g4[0] = (float)t0.x; g4[1] = (float)t0.y;
                                    g4[2] = (float)t1.x; g4[3] = (float)t1.y;
                                } else if constexpr (Q::QW == 2) {
                                    const double2 t0 = *reinterpret_cast<const double2*>(f + mb.o4);
                                    g4[0] = (float)t0.x; g4[1] = (float)t0.y;
                                    g4[2] = g4[3] = 0.0f;
                                } else {
                                    g4[0] = (float)atd(mb.o4);
                                    g4[1] = g4[2] = g4[3] = 0.0f;
                                }
                                // discounted prefix of the quarter up to bin k-2
                                // (weights 0 when the member needs no quarter term)
                                const float z4 = fmaf(wq4[0], g4[0], fmaf(wq4[1], g4[1], fmaf(wq4[2], g4[2], wq4[3] * g4[3])));
                                const float zin = fmaf(mb.fq, zq0, z4);
                                // (ONE: no pass before this one, so no carried
                                // terms: their weights are 0 and the rest is
                                // >= +0, so dropping them keeps the bits)
                                const float Zv = ONE ? fmaf(mb.cA, al0, zin)
                                                     : fmaf(mb.cW, Win, fmaf(mb.cG, glin, fmaf(mb.cA, al0, zin)));
                                const float gk = (float)gk64, gk1 = (float)gk164;
                                const float h = gk1 - gk;
                                // P in fp64: the expected finish count sums it
                                const double P64 = fma(th, gk164 - gk64, gk64);
                                const float num = mb.cost * fmaf(mb.cg, fmaf(-omd, Zv, gk), h * mb.psi);
                                a.P[prob + (int64_t)n * nn / 2 + m] = (float)P64;
                                // (one member per lane and pass when CR == 1:
                                // its values, not a sum with 0)
                                pP = CR == 1 ? P64 : pP + P64;
                                pN = CR == 1 ? num : pN + num;
                            };
                            if constexpr (CR == 1) {
                                // the lane's member of this pass, already in registers
                                if (pass_valid && mlo + lane < mhi) score_member(pass_mb, mlo + lane, pass_th, pass_wq);
                            } else {
                                for (int m = mlo + lane; m < mhi; m += 64) {
                                    const Member mb = s_mem[m];
                                    float wq4[4];
                                    quarter_weights(mb.rq, wq4);
                                    score_member(mb, m, (double)mb.theta + (double)mb.thlo, wq4);
                                }
                            }
                            // reduced across the lanes with the other step of
                            // its pair, after the pair
                            redP[i] = pP;
                            redN[i] = pN;
                            red_n[i] = n;
                            wave_lds_fence();
                        }
                    }
                    // carries out to the next panel pass, per-step sums
                    if (!ONE && p < LASTP) {
                        cW.set(n, fmaf(Win, dPW, T));
                        cGl.set(n, glast_here);
                    }
                    if constexpr (!ESPLIT) cE.add(n, (double)etot);
                }
                pass_zero = zero_after;
                if (++n == n1) {
                    n = ns;
                    ++p;
                    if (!ONE) {
                        mlo = __builtin_amdgcn_readlane(mlo_r, min(p, NP));
                        mend = __builtin_amdgcn_readlane(mlo_r, min(p + 1, NP));
                    }
                }
            }
            // Sum P (fp64) and the priority terms (fp32) over the lanes, two
            // steps at a time: each step's total comes out of the same tree
            // whichever step it is paired with.
#pragma unroll
            for (int i = 0; i < PF; i += 2) {
                if (red_n[i] >= 0 || red_n[i + 1] >= 0) {
                    const double zP = wave_pair_sum64(redP[i], redP[i + 1]);
                    const float zN = wave_pair_sum(redN[i], redN[i + 1]);
                    if (red_n[i] >= 0) {
                        cP.add(red_n[i], lane_read(zP, 31));
                        cN.add(red_n[i], lane_read(zN, 31));
                    }
                    if (red_n[i + 1] >= 0) {
                        cP.add(red_n[i + 1], lane_read(zP, 63));
                        cN.add(red_n[i + 1], lane_read(zN, 63));
                    }
                }
            }
        }

        // ---- E-only panels (tabulated mode): past LASTP no member reads G, so
        // these panels only add their sums of 1 - G to E[L_B], in a loop of its
        // own: the product and the sum, no discounted prefix, snapshot or
        // carries.  Its ring is primed afresh; the panels' sums are added in
        // panel order after those of the member panels, as before.  (ESPLIT:
        // every panel's sums come from emax_kernel.)
        if constexpr (!ESPLIT) {
            if (LASTP + 1 < NP) {
                constexpr int PFB = ORLOJ_EONLY_PREFETCH;   // its ring is deeper: fewer registers live here
                // Classes repeat along a deadline-ordered queue (fast classes
                // come first), and a repeat's row slice has usually left L2 by
                // the time the wave reads it again.  The RC classes with the
                // most members (at most 64 members, one per lane) keep their
                // slice of the current panel in registers for the pass: the
                // class's first member in step order loads it through the ring
                // as any step does and copies it, and its later members read the
                // copy while the ring loads the constant row for them.  Same
                // values, same bits.  (Where a step is skipped because G is 0
                // over the panel, every later step of the pass is skipped too,
                // so a copy taken then is never read.)
                // The next RL classes keep theirs in LDS, in the space of the
                // member panels' snapshot, prefixes and plans (unused from here
                // on), as far as this launch's LDS holds them: the first member
                // writes its slice there, and later members read it back into
                // their ring slot (loaded with the constant row) at their step.
                // The LDS read is issued at the step rather than with the ring's
                // loads: a ring filled from two kinds of loads would make every
                // step wait for all of the ring's memory loads.
                constexpr int RC = CR == 1 ? ORLOJ_EONLY_CACHE : 0;
                constexpr int RL = CR == 1 && CPL % 4 == 0 ? ORLOJ_EONLY_LDS_CACHE : 0;
                constexpr int NC = RC + RL;
                constexpr int RCA = RC > 0 ? RC : 1;
                constexpr int SLOT = 4 * PW;                        // bytes of one slice
                const int rl = min(RL, (int)((score_fixed_bytes<CPL>() + (size_t)maxcap * score_bytes_per_member()) / SLOT));
                // step code of member `lane`: NC (read from memory), k < NC (a
                // later member of cached class k: registers below RC, LDS from
                // RC), NC + 1 + k (the first member of class k)
                int rk_r = NC;
                if constexpr (NC > 0) {
                    const int cl = lane < n1 ? __builtin_bit_cast(int, cls_r.v[0]) : -1 - lane;
                    int cnt = 0, first = 64;        // members with this lane's class, the first of them
                    for (int m = n1 - 1; m >= 0; --m) {
                        const bool same = __builtin_amdgcn_readlane(cl, m) == cl;
                        cnt += same ? 1 : 0;
                        first = same ? m : first;
                    }
                    bool taken = lane >= n1;
#pragma unroll
                    for (int k = 0; k < NC; ++k) {
                        // most members first, ties to the earlier member; a
                        // class with a single member gains nothing
                        const int key = (taken || cnt < 2 || k >= RC + rl) ? -1 : (cnt << 6) | (63 - lane);
                        const int best = wave_max_i32(key);
                        if (best >= 0) {
                            const int ck = __builtin_amdgcn_readlane(cl, 63 - (best & 63));
                            if (cl == ck)
                                rk_r = first == lane ? NC + 1 + k : k;
                            taken = taken || cl == ck;
                        }
                    }
                }
                auto code = [&](int n) -> int {
                    if constexpr (NC > 0) return __builtin_amdgcn_readlane(rk_r, n);
                    return NC;
                };
                // slice k of the LDS classes: float4 j of lane l at 1024 j + 16 l
                // (each access a run of 64 consecutive 16-byte words)
                auto lds_slice = [&](int k, int j) {
                    return reinterpret_cast<float4*>(smem_raw + (size_t)k * SLOT + 1024 * j + 16 * lane);
                };
                // the ring's load for step n: the constant row for a later member
                // of a cached class (and where `none`), else memory
                auto load_e = [&](float (&v)[CPL], int n, int c0, bool none, int& lo, int& hi) {
                    load_step(v, n, c0, none || code(n) < NC, lo, hi);
                };
                float creg[RCA][CPL];
#pragma unroll
                for (int k = 0; k < RCA; ++k)
#pragma unroll
                    for (int j = 0; j < CPL; ++j) creg[k][j] = 0.0f;
                float bufb[PFB][CPL];
                int blo[PFB], bhi[PFB];
                const int totalB = (NP - LASTP - 1) * n1;
                const int itersB = (totalB + PFB - 1) / PFB * PFB;
                int qf_p = LASTP + 1, qf_n = 0;
#pragma unroll
                for (int i = 0; i < PFB; ++i) {
                    load_e(bufb[i], qf_n, qf_p * PW + base, false, blo[i], bhi[i]);
                    __builtin_amdgcn_sched_barrier(0);
                    if (++qf_n == n1) { qf_n = 0; qf_p = min(qf_p + 1, NP - 1); }
                }
                int pb = LASTP + 1, nb = 0;
                bool zero_b = false;
                float eprev = 0.0f;
                for (int it0 = 0; it0 < itersB; it0 += PFB) {
#pragma unroll
                    for (int i = 0; i < PFB; ++i) {
                        const int p0 = pb * PW;
                        const int pbase = p0 + base;
                        if (nb == 0) {
                            asm volatile("" ::: "memory");
#pragma unroll
                            for (int j = 0; j < CPL; ++j) Gacc[j] = 1.0;
                            zero_b = false;
                        }
                        const int hi_n = bhi[i];
                        const int lo_n = blo[i];
                        const bool real = nb >= n0;
                        const bool unchanged = zero_b || p0 >= hi_n;
                        const bool skip = pb >= NP || (real ? (nb > n0 && unchanged) : unchanged);
                        double gs[Q::QW];
                        // G <- G (1 - t) over the lane's bins, t from the row
                        // slice (ring slot or cache register)
                        auto update = [&](const float (&tv)[CPL]) {
#pragma unroll
                            for (int qq = 0; qq < Q::NQ; ++qq) {
#pragma unroll
                                for (int r = 0; r < Q::QW; ++r) {
                                    const int j = qq * Q::QW + r;
                                    const float t = (EXACT || pbase + j < K) ? tv[j] : 0.0f;
                                    Gacc[j] = fma(-Gacc[j], (double)t, Gacc[j]);
                                    gs[r] = qq == 0 ? Gacc[j] : gs[r] + Gacc[j];
                                }
                            }
                        };
                        const int kc = code(nb);
                        // a cached class's first member: keep its slice
#pragma unroll
                        for (int k = 0; k < RC; ++k) {
                            if (kc == NC + 1 + k) {
                                asm volatile("" ::: "memory");
#pragma unroll
                                for (int j = 0; j < CPL; ++j) creg[k][j] = bufb[i][j];
                            }
                        }
                        if constexpr (RL > 0) {
                            if (kc >= NC + 1 + RC) {
                                asm volatile("" ::: "memory");
#pragma unroll
                                for (int j = 0; j < CPL / 4; ++j)
                                    *lds_slice(kc - NC - 1 - RC, j) =
                                        make_float4(bufb[i][4 * j], bufb[i][4 * j + 1], bufb[i][4 * j + 2], bufb[i][4 * j + 3]);
                            }
                        }
                        if (!skip) {
                            bool done = false;
#pragma unroll
                            for (int k = 0; k < RC; ++k) {
                                if (!done && kc == k) {
                                    // a real branch per slot (the asm keeps it
                                    // from becoming per-bin selects)
                                    asm volatile("" ::: "memory");
                                    update(creg[k]);
                                    done = true;
                                }
                            }
                            if constexpr (RL > 0) {
                                if (!done && kc >= RC && kc < NC) {
                                    asm volatile("" ::: "memory");
#pragma unroll
                                    for (int j = 0; j < CPL / 4; ++j) {
                                        const float4 t = *lds_slice(kc - RC, j);
                                        bufb[i][4 * j] = t.x; bufb[i][4 * j + 1] = t.y;
                                        bufb[i][4 * j + 2] = t.z; bufb[i][4 * j + 3] = t.w;
                                    }
                                }
                            }
                            if (!done) update(bufb[i]);
                        }
#pragma unroll
                        for (int j = 0; j < CPL; ++j) asm volatile("" : "+v"(Gacc[j])::"memory");
                        const bool zero_after = zero_b || min(p0 + PW, K) <= lo_n;
                        load_e(bufb[i], qf_n, qf_p * PW + base, zero_after && qf_p == pb, blo[i], bhi[i]);
                        if (++qf_n == n1) { qf_n = 0; qf_p = min(qf_p + 1, NP - 1); }
                        if (pb < NP && real) {
                            float etot = eprev;
                            if (!skip) {
                                double gsum = gs[0];
#pragma unroll
                                for (int r = 1; r < Q::QW; ++r) gsum += gs[r];
                                const float e = (float)((double)CPL - gsum);
                                etot = lane63(wave_scan_sum(e));
                                eprev = etot;
                            }
                            cE.add(nb, (double)etot);
                        }
                        zero_b = zero_after;
                        if (++nb == n1) { nb = 0; ++pb; }
                    }
                }
            }
        }

        // ---- candidate outputs: lane l holds steps l, l + 64, ...
#pragma unroll
        for (int r = 0; r < CR; ++r) {
            const int n = r * 64 + lane;
            if (n >= n0 && n < n1) {
                double esum = cE.mine(r);
                if (ESPLIT && !a.defer) {
                    // the panels' sums in panel order, as this kernel adds them
                    esum = 0.0;
                    const size_t pair = AFF ? (size_t)q : (size_t)q * (size_t)a.nbs + (size_t)bi;
                    const float* ps = a.psum + pair * (size_t)a.np_e * (size_t)maxcap + n;
                    for (int pp = 0; pp < a.np_e; ++pp) esum += (double)ps[(size_t)pp * (size_t)maxcap];
                }
                a.E[cand + n] = cP.mine(r);
                if (ESPLIT && a.defer) {
                    // the selection finishes E[L_B] and the score from the
                    // panel sums (same expression, same bits): it runs after
                    // emax_kernel's waves, which share this launch
                    a.S[cand + n] = cN.mine(r);
                } else {
                    const double el = c0q + w * (0.5 + esum);
                    a.EL[cand + n] = (float)el;
                    a.S[cand + n] = (float)((double)cN.mine(r) / el);
                }
            }
        }
    };
    if (lastp == 0) rest(BoolTag<true>{});
    else rest(BoolTag<false>{});
}

// The affine mode's waves (at most 64 members) are held to 80 VGPRs, six
// waves per SIMD instead of the four their 100 would allow: the spills that
// costs lie outside the step loop (cfg5 affine call 0.0788 -> 0.0738 ms; at
// 72 VGPRs the loop spills and it takes 0.0856 ms).
template <int CPL, int PF, bool EXACT, int CR, bool AFF, bool ESPLIT>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(AFF && CR == 1 ? 6 : 1)))
void score_kernel(const ScoreArgs a) {
    score_wave<CPL, PF, EXACT, CR, AFF, ESPLIT>(a, blockIdx.x);
}

// ---------------------------------------------------------------------------
// emax_kernel: the sums behind E[L_B], one wave per (pair, panel), ahead of
// score_kernel.  E[L_B] = w (1/2 + sum_k (1 - G_n(x_{k+1}))) (Eq. (5)) needs
// the panel sums of 1 - G for every prefix length n.  A wave keeps the
// running product of its panel's bins over the pair's prefixes and writes
// each step's panel sum to psum[(pair * panels + p) * maxcap + n], rounded
// as score_kernel rounds its own per-panel sums, so E[L_B] has the same
// bits either way.
//   Affine mode: a pair is a model.  Under Eq. (3) every batch size's
//     histogram is the same product G_n of the members' solo CDFs on the
//     base grid, mapped onto a wider grid, so E[max] needs one product per
//     prefix length, not one per batch size (c0 + c1 s E[max]).
//   Tabulated mode, in launches split into step chunks: a pair is a (model,
//     batch size).  The panels past every member's deadline then need no
//     chunk to repeat their products: the score waves walk only the
//     panels that hold members.
// Rows are loaded PFE steps ahead; the class and support of step n sit in
// lane n % 64, so a step's row address needs no memory round trip.
// ---------------------------------------------------------------------------
// Steps loaded ahead by an emax_kernel wave: the loads of a step wait on
// nothing but the step's class, so a wave of narrow panels (few waves per
// SIMD) keeps more rows in flight.  A power of two that divides 64.
#ifndef ORLOJ_EMAX_PREFETCH_OF
#define ORLOJ_EMAX_PREFETCH_OF(CPL) ((CPL) >= 16 ? 8 : (CPL) >= 8 ? 16 : 32)
#endif

template <int CPL, bool EXACT, int CR, bool AFF>
__device__ __forceinline__ void emax_wave(const ScoreArgs& a, const unsigned bid) {
    using Q = Quarters<CPL>;
    constexpr int PW = 64 * CPL;
    constexpr int PFE = ORLOJ_EMAX_PREFETCH_OF(CPL);
    static_assert(PFE > 0 && 64 % PFE == 0, "a block of 64 steps ends on a prefetch round");
    const int K = a.K;
    const int NP = (K + PW - 1) / PW;
    const unsigned pair = bid / (unsigned)NP;
    const int p = (int)(bid - pair * (unsigned)NP);
    int q, bi;
    size_t qb;                                  // the pair's rows and sums
    if constexpr (AFF) {
        q = grid_model(a, pair);
        bi = a.nbs - 1;                         // the longest prefix (batch sizes increase)
        qb = (size_t)q;
    } else {
        bi = a.nbs - 1 - (int)(pair / (unsigned)a.Mg);   // largest batch sizes first
        q = grid_model(a, pair % (unsigned)a.Mg);
        qb = (size_t)q * (size_t)a.nbs + (size_t)bi;
    }
    const int64_t q0 = a.queue_off[q];
    const int64_t N = a.queue_off[q + 1] - q0;
    const int64_t cap64 = a.rect ? N : (N < a.bs[bi] ? N : (int64_t)a.bs[bi]);
    if (cap64 <= 0 || cap64 > a.maxcap || cap64 > 64 * CR) return;
    const int ncap = (int)cap64;
    const int lane = threadIdx.x;
    const int pbase = p * PW + lane * CPL;
    const float* tab_q = a.tab + qb * (size_t)a.C * (size_t)K;
    const int32_t* sup_q = a.sup ? a.sup + qb * (size_t)a.C * 2 : nullptr;
    float* out = a.psum + (qb * (size_t)NP + (size_t)p) * (size_t)a.maxcap;

    LaneCarry<CR> cls_r, lo_r, hi_r;
#pragma unroll
    for (int r = 0; r < CR; ++r) {
        const int m = min(r * 64 + lane, ncap - 1);
        int c = a.cls[q0 + m];
        if (c < 0 || c >= a.C) c = 0;                     // score_kernel flags it
        cls_r.v[r] = __builtin_bit_cast(float, c);
        lo_r.v[r] = __builtin_bit_cast(float, sup_q ? sup_q[2 * c] : 0);
        hi_r.v[r] = __builtin_bit_cast(float, sup_q ? sup_q[2 * c + 1] : K);
    }
    // the lane chunk of member n's row; chunks wholly outside the row's
    // support read the constant rows (the same bits, see score_kernel)
    auto load = [&](float (&v)[CPL], int n) {
        const int c = __builtin_bit_cast(int, cls_r.get(n));
        const int lo = __builtin_bit_cast(int, lo_r.get(n));
        const int hi = __builtin_bit_cast(int, hi_r.get(n));
        const bool ones = pbase + CPL <= lo, zeros = pbase >= hi;
        const float* src = tab_q + (size_t)c * (size_t)K + pbase;
        int lim = K - 1 - pbase;
        if (ones || zeros) {
            src = a.fill + (ones ? 16 : 0);
            lim = CPL - 1;
        }
        load_chunk<CPL, EXACT>(v, src, lim);
    };

    double G[CPL];
#pragma unroll
    for (int j = 0; j < CPL; ++j) G[j] = 1.0;
    float buf[PFE][CPL];
#pragma unroll
    for (int i = 0; i < PFE; ++i) {
        load(buf[i], min(i, ncap - 1));
        __builtin_amdgcn_sched_barrier(0);
    }
    // Each step's lane sums are parked in LDS, one row per step, and every
    // 64 steps lane r adds up row r in the pairwise order in which the wave
    // scan of score_kernel reaches its last lane (pairs of neighbouring
    // lanes, then pairs of those, ...), so the panel sums have that
    // kernel's bits without a cross-lane reduction on every step.
    __shared__ float s_e[64][65];
    for (int n0 = 0; n0 < ncap; n0 += PFE) {
#pragma unroll
        for (int i = 0; i < PFE; ++i) {
            const int n = n0 + i;
            if (n < ncap) {
                double gs[Q::QW];
#pragma unroll
                for (int qq = 0; qq < Q::NQ; ++qq) {
#pragma unroll
                    for (int r = 0; r < Q::QW; ++r) {
                        const int j = qq * Q::QW + r;
                        const float t = (EXACT || pbase + j < K) ? buf[i][j] : 0.0f;
                        G[j] = fma(-G[j], (double)t, G[j]);
                        gs[r] = qq == 0 ? G[j] : gs[r] + G[j];
                    }
                }
                double gsum = gs[0];
#pragma unroll
                for (int r = 1; r < Q::QW; ++r) gsum += gs[r];
                s_e[n & 63][lane] = (float)((double)CPL - gsum);   // padding bins hold G = 1
            }
            // refill the slot only after the update has read it
#pragma unroll
            for (int j = 0; j < CPL; ++j) asm volatile("" : "+v"(G[j])::"memory");
            load(buf[i], min(n + PFE, ncap - 1));
        }
        // a full block of 64 steps, or the last steps: lane r sums step
        // (block start + r)
        const int done = n0 + PFE;
        if ((done & 63) == 0 || done >= ncap) {
            wave_lds_fence();
            const int blk = (done - 1) & ~63;
            const int nr = blk + lane;
            if (nr < ncap) {
                float v[32];
#pragma unroll
                for (int k = 0; k < 32; ++k) v[k] = s_e[lane][2 * k] + s_e[lane][2 * k + 1];
#pragma unroll
                for (int w = 16; w >= 1; w >>= 1)
#pragma unroll
                    for (int k = 0; k < w; ++k) v[k] = v[2 * k] + v[2 * k + 1];
                out[nr] = v[0];
            }
            wave_lds_fence();
        }
    }
}

template <int CPL, bool EXACT, int CR, bool AFF>
__global__ __launch_bounds__(64) void emax_kernel(const ScoreArgs a) {
    emax_wave<CPL, EXACT, CR, AFF>(a, blockIdx.x);
}

// One launch for a scheduling round's tabulated scoring when the E sums come
// from emax_kernel's waves: workgroups [0, n_emax) are those waves, the rest
// score_kernel's (their E[L_B] and scores are finished by the selection,
// which runs after the launch).  Nothing in the launch waits on anything
// else in it, so the two kinds of waves run side by side.
template <int CPL, bool EXACT, int CR>
__global__ __launch_bounds__(64) void round_kernel(const ScoreArgs a, const unsigned n_emax) {
    if (blockIdx.x < n_emax) {
        emax_wave<CPL, EXACT, CR, false>(a, blockIdx.x);
    } else {
        score_wave<CPL, ORLOJ_SPLIT_PREFETCH, EXACT, CR, false, true>(a, blockIdx.x - n_emax);
    }
}

// ---------------------------------------------------------------------------
// select_kernel: one workgroup per model; thread i reads candidates i,
// i + kSelThreads, ... (coalesced) and finds its (batch size, n) from the
// block starts of the model's batch sizes.
// ---------------------------------------------------------------------------
struct SelectArgs {
    const int64_t* queue_off;
    const int64_t* cand_off;
    float* S;                  // read; written too when finishing
    // finishing (a scheduling round whose score launch left it here): each
    // candidate's E[L_B] and score from emax_kernel's panel sums and the
    // priority sum the score waves wrote to S
    int finish;
    // scheduling rounds (mapped host memory, or NULL): after its writes,
    // each workgroup g makes them visible to the host and writes `round`
    // to done[g], so the host can see the round finish without waiting for
    // the stream
    int32_t* done;
    int32_t round;
    const float* psum;         // [M][nbs][np_e][maxcap]
    int np_e, maxcap;
    const double* width;       // [M]
    float* EL;
    int32_t* sel_n;
    int32_t* sel_bs;
    float* sel_score;
    int nbs, rect;
    int M;
    int n_act;                 // compact: workgroup g < n_act selects for act[g],
    int compact;               //   workgroup n_act clears the models with an empty queue
    int bs[ORLOJ_MAX_BATCH_SIZES];
    int act[kMaxActive];
};

struct Best {
    float s;
    int n;
    int bs;
};

__device__ __forceinline__ bool better(const Best& x, const Best& y) {
    // larger score; exact ties: larger n, then smaller batch size (n = 0:
    // no candidate).  Written without branches, and applied with selects
    // (take_if_better): the branchy form of the update lost the new n on
    // some paths when compiled for gfx950.
    const bool sgt = x.s > y.s, seq = x.s == y.s;
    const bool tie = seq && (x.n > y.n || (x.n == y.n && x.bs < y.bs));
    return x.n != 0 && (y.n == 0 || sgt || tie);
}

__device__ __forceinline__ void take_if_better(Best& best, const Best& c) {
    const bool t = better(c, best);
    best.s = t ? c.s : best.s;
    best.n = t ? c.n : best.n;
    best.bs = t ? c.bs : best.bs;
}

// 16 waves per model: the kernel is a chain of latencies (block starts,
// candidate loads, reductions), so more threads per model shorten it.
constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / 64;

__global__ __launch_bounds__(kSelThreads) void select_kernel(const SelectArgs a) {
    __shared__ int64_t s_start[ORLOJ_MAX_BATCH_SIZES + 1];
    __shared__ Best s_best[kSelWaves];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    if (a.compact && (int)blockIdx.x >= a.n_act) {
        // the workgroup after the selecting ones: no batch for the models
        // with an empty queue (not listed).  Its clears, and their fence,
        // run beside the selections.
        for (int m = tid; m < a.M; m += kSelThreads) {
            if (a.queue_off[m + 1] == a.queue_off[m]) {
                a.sel_n[m] = 0;
                a.sel_bs[m] = 0;
                a.sel_score[m] = 0.0f;
            }
        }
        if (a.done) {
            // the clears reach the host before the flag (every thread that
            // cleared fences its own writes)
            if (tid < a.M) __threadfence_system();
            __syncthreads();
            if (tid == 0) __hip_atomic_store(&a.done[blockIdx.x], a.round, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        }
        return;
    }
    const int q = a.compact ? a.act[blockIdx.x] : (int)blockIdx.x;
    __shared__ int64_t s_wsum[kSelWaves];
    const int64_t N = a.queue_off[q + 1] - a.queue_off[q];
    // block starts: an exclusive scan of the prefix caps over the batch
    // sizes, kSelThreads at a time (a workgroup scan of per-wave scans)
    int64_t carry = 0;
    for (int b0 = 0; b0 < a.nbs; b0 += kSelThreads) {
        const int bi = b0 + tid;
        const int bsz = bi < a.nbs ? a.bs[bi] : 0;
        const int64_t cap = bi < a.nbs ? (a.rect ? N : (N < bsz ? N : (int64_t)bsz)) : 0;
        const int64_t incl = wave_incl_scan_u64((uint64_t)cap, lane);
        if (lane == 63) s_wsum[wv] = incl;
        __syncthreads();
        int64_t before = carry;
        for (int w = 0; w < wv; ++w) before += s_wsum[w];
        if (bi < a.nbs) s_start[bi] = before + incl - cap;
        for (int w = 0; w < kSelWaves; ++w) carry += s_wsum[w];
        __syncthreads();
    }
    if (tid == 0) s_start[a.nbs] = carry;
    __syncthreads();
    const float* S = a.S + a.cand_off[q];
    Best best{0.0f, 0, 0};
    // candidates i = tid, tid + kSelThreads, ... (coalesced); a candidate's
    // (batch size, n) from the block starts.  The comparison is a total
    // order, so the pick does not depend on the order of the visits.
    const int64_t total = s_start[a.nbs];
    const double wq = a.finish ? a.width[q] : 0.0;
    for (int64_t i = tid; i < total; i += kSelThreads) {
        float sc = S[i];
        int lo = 0, hi = a.nbs - 1;          // last bi with s_start[bi] <= i
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (s_start[mid] <= i) lo = mid; else hi = mid - 1;
        }
        const int n = (int)(i - s_start[lo]) + 1;
        const int bsz = a.bs[lo];
        if (a.finish) {
            // E[L_B] = w (1/2 + the panels' sums in panel order) and the
            // score, as the score waves form them when they finish
            const float* ps = a.psum + ((size_t)q * (size_t)a.nbs + (size_t)lo) * (size_t)a.np_e *
                                           (size_t)a.maxcap + (size_t)(n - 1);
            double esum = 0.0;
            for (int pp = 0; pp < a.np_e; ++pp) esum += (double)ps[(size_t)pp * (size_t)a.maxcap];
            const double el = 0.0 + wq * (0.5 + esum);
            sc = (float)((double)sc / el);
            a.EL[a.cand_off[q] + i] = (float)el;
            a.S[a.cand_off[q] + i] = sc;
        }
        if (n <= bsz && sc == sc)            // NaN never wins
            take_if_better(best, Best{sc, n, bsz});
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        Best o;
        o.s = __shfl_xor(best.s, off, 64);
        o.n = __shfl_xor(best.n, off, 64);
        o.bs = __shfl_xor(best.bs, off, 64);
        take_if_better(best, o);
    }
    if (lane == 0) s_best[wv] = best;
    __syncthreads();
    if (wv == 0) {
        // the waves' picks, reduced across the first kSelWaves lanes
        best = lane < kSelWaves ? s_best[lane] : Best{0.0f, 0, 0};
#pragma unroll
        for (int off = kSelWaves / 2; off > 0; off >>= 1) {
            Best o;
            o.s = __shfl_xor(best.s, off, 64);
            o.n = __shfl_xor(best.n, off, 64);
            o.bs = __shfl_xor(best.bs, off, 64);
            take_if_better(best, o);
        }
        if (lane == 0) {
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
    if (a.done) {
        // the selection (written by thread 0, above) reaches the host before
        // the flag
        if (tid == 0) {
            __threadfence_system();
            __hip_atomic_store(&a.done[blockIdx.x], a.round, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        }
    }
}

}  // namespace

// ===========================================================================
// C ABI
// ===========================================================================
namespace {

// ---------------------------------------------------------------------------
// Scheduler iteration (§3.2 Algorithm 1) with the paper's own priority.
//
// laws_kernel: one workgroup per (model, batch size).  Thread t owns the VPT
// consecutive bins [t*VPT, t*VPT + VPT).  It forms the model's class mix
// F_mix = sum_c pi_c F_c in fp64, then for each class the CDF of a
// request's batch latency, F_c F_mix^(s-1) (the request plus s-1 members
// drawn from the mix; §4.2.1: the max of k identical variables has CDF
// F^k), and its discounted prefix Z(k) = sum_{i<=k} G(x_{i+1}) d^(k-i),
// d = e^{-b w}: an in-thread fp64 prefix, a weighted DPP scan across the
// wave and a weighted combination across the four waves.  Block 0 of each
// model also writes the model-wide E[L] of F_mix^s (§4.3).
// ---------------------------------------------------------------------------
struct LawArgs {
    const float* tab;          // [M][nbs][C][K] 1 - F(x_{k+1})
    const double* weights;     // [M][C] class mix, or NULL (uniform)
    const double* width;       // [M]
    float* law;                // [M][nbs][C][K]
    float* disc;               // [M][nbs][C][K]
    float* model_el;           // [M][nbs]
    int* err;
    double b;
    int M, C, K, nbs;
    int bs[ORLOJ_MAX_BATCH_SIZES];
};

// One thread's VPT consecutive entries of a table row: F = 1 - t, and 1
// beyond the row's end.  Whole float4s when the row length is a multiple
// of 4 (rows and thread chunks are then 16-byte aligned).
template <int VPT>
__device__ __forceinline__ void load_cdf_chunk(double (&F)[VPT], const float* __restrict__ t, int base,
                                               int K) {
    if constexpr (VPT % 4 == 0) {
        if ((K & 3) == 0) {
#pragma unroll
            for (int j = 0; j < VPT; j += 4) {
                if (base + j < K) {
                    const float4 v = *reinterpret_cast<const float4*>(t + base + j);
                    F[j] = 1.0 - (double)v.x; F[j + 1] = 1.0 - (double)v.y;
                    F[j + 2] = 1.0 - (double)v.z; F[j + 3] = 1.0 - (double)v.w;
                } else {
                    F[j] = F[j + 1] = F[j + 2] = F[j + 3] = 1.0;
                }
            }
            return;
        }
    }
#pragma unroll
    for (int j = 0; j < VPT; ++j) F[j] = base + j < K ? 1.0 - (double)t[base + j] : 1.0;
}

// Store one thread's VPT entries (those below K) of a row.
template <int VPT>
__device__ __forceinline__ void store_chunk(float* __restrict__ o, const float (&v)[VPT], int base, int K) {
    if constexpr (VPT % 4 == 0) {
        if ((K & 3) == 0) {
#pragma unroll
            for (int j = 0; j < VPT; j += 4)
                if (base + j < K)
                    *reinterpret_cast<float4*>(o + base + j) = make_float4(v[j], v[j + 1], v[j + 2], v[j + 3]);
            return;
        }
    }
#pragma unroll
    for (int j = 0; j < VPT; ++j)
        if (base + j < K) o[base + j] = v[j];
}

template <int VPT>
__global__ __launch_bounds__(kThreads) void laws_kernel(const LawArgs a) {
    __shared__ float s_wave[kWaves];
    __shared__ double s_el[kWaves];
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int q = (int)(blockIdx.x / (unsigned)a.nbs);
    const int bi = (int)(blockIdx.x % (unsigned)a.nbs);
    const int K = a.K, C = a.C;
    const int s = a.bs[bi];
    const double w = a.width[q];
    const double d = exp(-a.b * w);
    const int base = tid * VPT;
    const size_t row0 = ((size_t)q * (size_t)a.nbs + (size_t)bi) * (size_t)C;

    // class mix and its powers at this thread's bins (padding bins: F = 1)
    double mix[VPT];
#pragma unroll
    for (int j = 0; j < VPT; ++j) mix[j] = 0.0;
    double wsum = 0.0;
    bool wbad = false;
    for (int c = 0; c < C; ++c) {
        const double wc = a.weights ? a.weights[(size_t)q * C + c] : 1.0;
        wbad |= !(wc >= 0.0) || isinf(wc);
        wsum += wc;
    }
    if (wbad || !(wsum > 0.0)) {
        if (tid == 0) atomicOr(a.err, kErrWeights);
        wsum = 1.0;
    }
    for (int c = 0; c < C; ++c) {
        const double pc = (a.weights ? a.weights[(size_t)q * C + c] : 1.0) / wsum;
        double F[VPT];
        load_cdf_chunk<VPT>(F, a.tab + (row0 + (size_t)c) * (size_t)K, base, K);
#pragma unroll
        for (int j = 0; j < VPT; ++j) mix[j] = fma(pc, F[j], mix[j]);
    }
    double pm[VPT];
    double el = 0.0;
#pragma unroll
    for (int j = 0; j < VPT; ++j) {
        pm[j] = s > 1 ? pow(mix[j], (double)(s - 1)) : 1.0;
        if (base + j < K) el += 1.0 - pm[j] * mix[j];
    }
    // model-wide E[L] = w (1/2 + sum_k (1 - F_mix^s(x_{k+1})))
    for (int o = 32; o > 0; o >>= 1) el += __shfl_xor(el, o, 64);
    if (lane == 0) s_el[wv] = el;
    __syncthreads();
    if (tid == 0) {
        double tot = 0.0;
        for (int i = 0; i < kWaves; ++i) tot += s_el[i];
        a.model_el[(size_t)q * a.nbs + bi] = (float)(w * (0.5 + tot));
    }

    // scan constants: a thread chunk spans VPT bins
    const float log2d = (float)(-a.b * w * 1.4426950408889634);
    float rp[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) rp[i] = exp2_hw(log2d * (float)(VPT << i));
    const float w15 = exp2_hw(log2d * (float)(VPT * ((lane & 15) + 1)));
    const float w31 = exp2_hw(log2d * (float)(VPT * (lane >= 32 ? lane - 31 : 0)));
    const float d_wave = exp2_hw(log2d * (float)(64 * VPT));

    for (int c = 0; c < C; ++c) {
        const size_t r = (row0 + (size_t)c) * (size_t)K;
        double g[VPT];
        load_cdf_chunk<VPT>(g, a.tab + r, base, K);
        double z = 0.0;
#pragma unroll
        for (int j = 0; j < VPT; ++j) {
            g[j] *= pm[j];
            z = fma(z, d, g[j]);
        }
        // in-wave weighted scan of the chunk totals, then across the waves
        const float A = wave_wscan((float)z, rp, w15, w31);
        if (lane == 63) s_wave[wv] = A;
        __syncthreads();
        float carry = 0.0f;   // discounted sum of the earlier waves' bins, at the end of the last one
#pragma unroll
        for (int i = 0; i < kWaves; ++i)
            if (i < wv) carry = fmaf(carry, d_wave, s_wave[i]);
        __syncthreads();
        // prefix up to the end of the previous thread chunk
        const float prev = __shfl_up(A, 1, 64);
        const float before = (lane > 0 ? prev : 0.0f) + carry * exp2_hw(log2d * (float)(VPT * lane));
        double zz = (double)before;
        float lv[VPT], dv[VPT];
#pragma unroll
        for (int j = 0; j < VPT; ++j) {
            zz = fma(zz, d, g[j]);
            lv[j] = (float)g[j];
            dv[j] = (float)zz;
        }
        store_chunk<VPT>(a.law + r, lv, base, K);
        store_chunk<VPT>(a.disc + r, dv, base, K);
    }
}

// ---------------------------------------------------------------------------
// iterate_kernel: one workgroup per model, of TH threads (256, or 1024 when
// a queue is longer than 1024 requests).  Requests are strided over the
// threads (request i on thread i mod TH).  Long queues on few models split
// the iteration in two launches: the drop phase in parts of kDropPart
// requests, one workgroup each, writing per-part counts, then the rest per
// model from those counts.  For every batch size the drop
// phase keeps a request iff its deadline lies past the left edge of its
// class's first bin with mass at that batch size (then it could finish run
// alone).  Over 32 batch sizes the model's first-bin table sits in LDS and
// each wave walks its 64 requests with the batch sizes across its lanes (one
// integer compare per pair against the request's keep edge); otherwise each
// lane takes a request and the counts and the earliest kept request come
// from wave ballots.
// Thread 0 picks the candidate batch size ((D_{Q_s}, s) descending, first
// with |Q_s| >= s).  Requests kept at the candidate size get their
// priority from the model-law tables (Eq. (2) in the scan form:
// gamma e^{-b theta w} (G_k - (1-d) Z(k-2)) + h_k psi(theta), over the
// model-wide E[L]); PopBatch takes the s largest keys (kept flag, priority,
// earlier position) in rank order: for queues up to 512 requests each key's
// rank is counted against all keys in LDS; longer queues find the s-th
// largest key by a radix select (eight 8-bit digits, an LDS histogram and a
// block suffix scan per digit) and rank the selected keys.
// ---------------------------------------------------------------------------
struct IterArgs {
    const int32_t* sup;        // [M][nbs][C][2]
    const float* law;          // [M][nbs][C][K]
    const float* disc;         // [M][nbs][C][K]
    const float* model_el;     // [M][nbs]
    const int64_t* queue_off;
    const int32_t* cls;
    const double* deadline;
    const double* now;
    const double* width;
    const double* cost;        // [N] or NULL (1)
    const int64_t* step_off;   // [N+1] or NULL (one step at the deadline)
    const double* step_dl;     // [S]
    const double* step_cost;   // [S] cumulative costs
    int32_t* timed_out;        // [N]
    float* score;              // [N]
    int32_t* cand_bs;          // [M]
    int32_t* batch;            // [M][bs_max]
    int* err;
    int32_t* part_cnt;         // [M][parts][nbs] drop-phase counts of a split launch
    int32_t* part_first;       // [M][parts][nbs] and first kept positions
    int parts;
    double b;
    int M, C, K, nbs, bs_max;
    int bs[ORLOJ_MAX_BATCH_SIZES];
};

// What one iterate_kernel launch does: the whole iteration per model, or
// the iteration split in two launches for long queues on few models: the
// drop phase over parts of kDropPart requests (one workgroup each), then
// the rest per model from the parts' counts.
constexpr int kIterWhole = 0, kIterDropPart = 1, kIterFromParts = 2;
constexpr int kDropPart = 256;

constexpr int kIterMaxBatch = 1024;      // largest batch size PopBatch orders in LDS
constexpr int kIterMaxQueue = 4096;      // longest queue one workgroup ranks
constexpr int kIterWideQueue = 1024;     // longer queues get 1024-thread workgroups
constexpr int kIterStage = 8448;         // LDS words for a model's first-bin table

// The largest k in [0, K] with (double)k * w < tau, or -1 when there is
// none (tau <= 0 or NaN); w is finite and > 0.  Products k * w rise with k,
// so for any first bin lo in [0, K]: tau > lo * w iff lo <= keep_edge.
__device__ inline int keep_edge(double tau, double w, int K) {
    if (!(tau > 0.0)) return -1;
    const double t = tau / w;
    int k = t >= (double)K ? K : (int)t;
    while (k > 0 && (double)k * w >= tau) --k;
    while (k < K && (double)(k + 1) * w < tau) ++k;
    return k;
}

template <int TH, bool STAGE, int PH>
__global__ __launch_bounds__(TH) void iterate_kernel(const IterArgs a) {
    constexpr int kW = TH / 64;                    // waves
    __shared__ int s_cnt[ORLOJ_MAX_BATCH_SIZES];
    __shared__ int s_first[ORLOJ_MAX_BATCH_SIZES];
    __shared__ int s_cand;
    __shared__ double s_cd[kW];
    __shared__ int s_cb[kW];
    __shared__ unsigned s_hist[2][256];
    __shared__ int s_wcnt[kW][ORLOJ_MAX_BATCH_SIZES];
    __shared__ int s_wfirst[kW][ORLOJ_MAX_BATCH_SIZES];
    __shared__ unsigned s_wsum[4];
    __shared__ int s_digit, s_need;
    __shared__ __align__(16) unsigned long long s_sel[kIterMaxBatch];
    __shared__ int s_nsel;
    __shared__ int s_lo[STAGE ? kIterStage + 64 : 1];   // [C][nbs + 1] first bins, 64 words of tail
    const int tid = threadIdx.x, lane = tid & 63, wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int q = PH == kIterDropPart ? (int)blockIdx.x / a.parts : (int)blockIdx.x;
    const int64_t q0 = a.queue_off[q];
    const int N = (int)(a.queue_off[q + 1] - q0);
    // the requests whose drop phase this workgroup runs
    int ib = 0, ie = N;
    if constexpr (PH == kIterDropPart) {
        ib = ((int)blockIdx.x - q * a.parts) * kDropPart;
        ie = min(N, ib + kDropPart);
        if (ib >= ie) return;
    }
    const int nbs = a.nbs, C = a.C, K = a.K;
    const double w = a.width[q];
    const double nowq = a.now[q];
    const bool wok = w > 0.0 && w < HUGE_VAL;
    if (tid == 0) { s_cand = -1; s_nsel = 0; }
    if (tid < 256) {
        s_hist[0][tid] = 0u;
        s_hist[1][tid] = 0u;
    }
    const int32_t* sup_q = a.sup + (size_t)q * (size_t)nbs * (size_t)C * 2;
    // first bin with mass of class c at batch size index bi, in [0, K) in
    // a support that orloj_build_cdfs wrote (the LDS copy below is clamped
    // to [0, K], which changes nothing there)
    auto first_bin = [&](int bi, int c) { return sup_q[((size_t)bi * C + c) * 2]; };
    // STAGE (more than 32 batch sizes, and C (nbs + 1) <= kIterStage): the
    // model's table is staged in LDS class-major (rows of nbs + 1 words, so
    // the transposing writes spread over the banks) and the drop phase runs
    // across the batch sizes in the lanes.  Fewer batch sizes would leave
    // most lanes idle that way, so there each lane takes a request instead.
    const int ldo = nbs + 1;
    constexpr bool staged = STAGE;
    if constexpr (staged)
        for (int j = tid; j < nbs * C; j += TH) {
            const int bi = j / C, c = j - bi * C;
            s_lo[c * ldo + bi] = min(max(sup_q[2 * j], 0), K);
        }
    __syncthreads();

    // drop phase: per wave, the count of kept requests and the first kept
    // position of batch size index 64 r + l sit in lane l of cntv[r] and
    // firstv[r] (no atomics); the waves are combined afterwards
    constexpr int kBR = ORLOJ_MAX_BATCH_SIZES / 64;
    int cntv[kBR], firstv[kBR];
    unsigned long long vmask[kBR];   // lanes that hold a batch size, per row
    const int nrows = (nbs + 63) / 64;
#pragma unroll
    for (int r = 0; r < kBR; ++r) {
        cntv[r] = 0;
        firstv[r] = 0x7fffffff;
        vmask[r] = __ballot(64 * r + lane < nbs);
    }
    for (int i0 = ib; i0 < (PH == kIterFromParts ? ib : ie); i0 += TH) {
        const int i = i0 + tid;
        const bool live = i < ie;
        int c = 0;
        double tau = 0.0;
        if (live) {
            c = a.cls[q0 + i];
            const double D = a.deadline[q0 + i];
            // the drop phase looks at the last step of a step cost function
            const double Dlast = a.step_off ? a.step_dl[a.step_off[q0 + i + 1] - 1] : D;
            int flag = 0;
            if (c < 0 || c >= C) { flag |= kErrClassRange; c = 0; }
            if (isnan(D)) flag |= kErrDeadlineNaN;
            if (i > 0 && D < a.deadline[q0 + i - 1]) flag |= kErrUnsorted;
            if (i == 0 && isnan(nowq)) flag |= kErrNowNaN;
            if (i == 0 && !wok) flag |= kErrWidth;
            if (flag) atomicOr(a.err, flag);
            tau = Dlast - nowq;
        }
        if constexpr (staged) {
            // the wave's 64 requests one at a time, its lanes over the batch
            // sizes: request j is kept at batch size 64 r + l iff that
            // batch size's first bin of its class is <= its keep edge (no
            // first bin is below 0, so a request with edge -1, dead lanes
            // included, is kept nowhere).  Eight requests' rows are read
            // before any is compared.
            const int kk = live && wok ? keep_edge(tau, w, K) : -1;
            const int base = i0 + wv * 64;
            const int nj = __builtin_amdgcn_readfirstlane(min(64, ie - base));
            unsigned long long anyb = 0ull;   // bit j: request base + j kept somewhere
            auto sweep = [&](auto rows) {
                constexpr int NR = decltype(rows)::value;
                for (int j0 = 0; j0 < nj; j0 += 8) {
                    int kj[8], lo[8][NR];
#pragma unroll
                    for (int jj = 0; jj < 8; ++jj) {
                        kj[jj] = __builtin_amdgcn_readlane(kk, j0 + jj);
                        const int* row = s_lo + __builtin_amdgcn_readlane(c, j0 + jj) * ldo + lane;
#pragma unroll
                        for (int r = 0; r < NR; ++r) lo[jj][r] = row[64 * r];
                    }
#pragma unroll
                    for (int jj = 0; jj < 8; ++jj) {
                        const int ij = base + j0 + jj;
                        unsigned long long hit = 0ull;
#pragma unroll
                        for (int r = 0; r < NR; ++r) {
                            const bool keep = lo[jj][r] <= kj[jj];
                            hit |= __ballot(keep) & vmask[r];
                            cntv[r] += keep ? 1 : 0;
                            firstv[r] = min(firstv[r], keep ? ij : 0x7fffffff);
                        }
                        if (hit) anyb |= 1ull << (j0 + jj);
                    }
                }
            };
            switch (nrows) {
                case 1: sweep(std::integral_constant<int, 1>{}); break;
                case 2: sweep(std::integral_constant<int, 2>{}); break;
                case 3: sweep(std::integral_constant<int, 3>{}); break;
                default: sweep(std::integral_constant<int, 4>{}); break;
            }
            if (live) {
                a.timed_out[q0 + i] = (anyb >> lane) & 1ull ? 0 : 1;
                a.score[q0 + i] = 0.0f;
            }
            continue;
        }
        bool any = false;
        // the support's first bins of a group of batch sizes are loaded
        // together, so their latencies overlap
        constexpr int kGroup = 8;
#pragma unroll
        for (int r = 0; r < kBR; ++r) {
            const int bend = min(nbs, 64 * r + 64);
            for (int b0 = 64 * r; b0 < bend; b0 += kGroup) {
                int lo[kGroup];
#pragma unroll
                for (int j = 0; j < kGroup; ++j)
                    lo[j] = first_bin(min(b0 + j, nbs - 1), c);
#pragma unroll
                for (int j = 0; j < kGroup; ++j) {
                    const int bi = b0 + j;
                    if (bi >= bend) break;
                    const bool keep = live && wok && tau > (double)lo[j] * w;
                    any |= keep;
                    const unsigned long long m = __ballot(keep);
                    const bool me = lane == (bi & 63);
                    cntv[r] += me ? __popcll(m) : 0;
                    if (me && m != 0ull && firstv[r] == 0x7fffffff)
                        firstv[r] = i0 + wv * 64 + __ffsll((long long)m) - 1;
                }
            }
        }
        if (live) {
            a.timed_out[q0 + i] = any ? 0 : 1;
            a.score[q0 + i] = 0.0f;
        }
    }
    if constexpr (PH != kIterFromParts) {
#pragma unroll
        for (int r = 0; r < kBR; ++r) {
            s_wcnt[wv][64 * r + lane] = cntv[r];
            s_wfirst[wv][64 * r + lane] = firstv[r];
        }
        __syncthreads();
    }
    for (int bi = tid; bi < nbs; bi += TH) {
        int cnt = 0, first = 0x7fffffff;
        if constexpr (PH == kIterFromParts) {
            const size_t p0 = (size_t)q * a.parts * nbs + bi;
            for (int p = 0; p * kDropPart < N; ++p) {
                cnt += a.part_cnt[p0 + (size_t)p * nbs];
                first = min(first, a.part_first[p0 + (size_t)p * nbs]);
            }
        } else {
#pragma unroll
            for (int v = 0; v < kW; ++v) {
                cnt += s_wcnt[v][bi];
                first = min(first, s_wfirst[v][bi]);
            }
        }
        if constexpr (PH == kIterDropPart) {
            const size_t o = ((size_t)blockIdx.x) * nbs + bi;   // (q parts + part) nbs + bi
            a.part_cnt[o] = cnt;
            a.part_first[o] = first;
        } else {
            s_cnt[bi] = cnt;
            s_first[bi] = first;
        }
    }
    if constexpr (PH == kIterDropPart) return;
    __syncthreads();
    // Candidate batch size: among batch sizes whose kept set holds at least
    // s requests, the largest earliest-kept deadline D_{Q_s}, ties to the
    // larger batch size (batch sizes increase with their index).  Thread bi
    // proposes batch size bi; a wave reduction, then one over the waves.
    {
        double dc = 0.0;
        int cb = -1;
        for (int bi = tid; bi < nbs; bi += TH) {
            if (s_cnt[bi] < a.bs[bi]) continue;
            const double D = a.deadline[q0 + s_first[bi]];
            if (cb < 0 || D > dc || (D == dc && bi > cb)) { dc = D; cb = bi; }
        }
        auto take = [&](double d2, int b2) {
            if (b2 >= 0 && (cb < 0 || d2 > dc || (d2 == dc && b2 > cb))) { dc = d2; cb = b2; }
        };
        for (int o = 32; o > 0; o >>= 1) {
            const double d2 = __shfl_xor(dc, o, 64);
            const int b2 = __shfl_xor(cb, o, 64);
            take(d2, b2);
        }
        if (lane == 0) { s_cd[wv] = dc; s_cb[wv] = cb; }
        __syncthreads();
        if (tid == 0) {
            for (int i = 0; i < kW; ++i) take(s_cd[i], s_cb[i]);
            s_cand = cb;
            a.cand_bs[q] = cb >= 0 ? a.bs[cb] : 0;
        }
        __syncthreads();
    }
    const int cand = s_cand;
    int32_t* bq = a.batch + (size_t)q * (size_t)a.bs_max;
    if (cand < 0) {
        for (int j = tid; j < a.bs_max; j += TH) bq[j] = -1;
        return;
    }
    const int s = a.bs[cand];

    // priorities at the candidate size; keys = kept | priority bits | ~index
    const double bw = a.b * w;
    const double gamma = -expm1(-bw) / bw;
    const double omd = -expm1(-bw);
    const float el = a.model_el[(size_t)q * nbs + cand];
    const size_t lrow0 = ((size_t)q * nbs + cand) * (size_t)C;
    constexpr int kPer = kIterMaxQueue / TH;         // keys per thread, in registers
    unsigned long long key[kPer];
#pragma unroll
    for (int j = 0; j < kPer; ++j) key[j] = 0ull;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
        const int i = j * TH + tid;
        if (i < N) {
            int c = a.cls[q0 + i];
            c = (c < 0 || c >= C) ? 0 : c;
            const double D = a.deadline[q0 + i];
            const double Dlast = a.step_off ? a.step_dl[a.step_off[q0 + i + 1] - 1] : D;
            const int lo = first_bin(cand, c);
            if (wok && Dlast - nowq > (double)lo * w) {
                const float* G = a.law + (lrow0 + c) * (size_t)K;
                const float* Z = a.disc + (lrow0 + c) * (size_t)K;
                // Eq. (2) x E[L] for one deadline, in the scan form
                auto num_at = [&](double tau) -> double {
                    if (!(tau > 0.0)) return 0.0;
                    const double u = tau / w;
                    if (u >= (double)K) {
                        const double cg = gamma * exp(-a.b * (tau - (double)K * w));
                        const double zk = K >= 2 ? (double)Z[K - 2] : 0.0;
                        return cg * (1.0 - omd * zk);
                    }
                    const int k = (int)floor(u);
                    const double th = u - (double)k;
                    const double gk = k >= 1 ? (double)G[k - 1] : 0.0;
                    const double gk1 = (double)G[k];
                    const double zk = k >= 2 ? (double)Z[k - 2] : 0.0;
                    const double cg = gamma * exp(-a.b * th * w);
                    const double psi = -expm1(-a.b * th * w) / bw;
                    return cg * (gk - omd * zk) + (gk1 - gk) * psi;
                };
                double cr = a.cost ? a.cost[q0 + i] : 1.0;
                int flag = 0;
                if (!(cr >= 0.0 && cr < HUGE_VAL)) { flag = kErrCost; cr = 0.0; }
                double num = 0.0;
                if (a.step_off) {
                    // App. B: one single step per cost increment
                    double below = 0.0, dprev = -HUGE_VAL;
                    for (int64_t st = a.step_off[q0 + i]; st < a.step_off[q0 + i + 1]; ++st) {
                        const double dj = a.step_dl[st], cj = a.step_cost[st];
                        if (!(cj >= below && cj < HUGE_VAL) || !(dj > dprev)) {
                            flag = kErrCost;
                            num = 0.0;
                            break;
                        }
                        num += (cj - below) * num_at(dj - nowq);
                        below = cj;
                        dprev = dj;
                    }
                } else {
                    num = num_at(D - nowq);
                }
                if (flag) atomicOr(a.err, flag);
                num *= cr;
                const float p = (float)(num / (double)el);
                a.score[q0 + i] = p;
                const float pp = p > 0.0f ? p : 0.0f;
                key[j] = (1ull << 63) | ((unsigned long long)__float_as_uint(pp) << 32) |
                         (unsigned long long)(0xffffffffu - (unsigned)i);
            }
        }
    }
    // Short queues: every kept key's rank is the number of larger keys
    // (keys are unique), counted over the keys staged in LDS; the s keys of
    // rank < s are the batch, in rank order.
    constexpr int kRankQueue = 512;
    constexpr int kRankSlots = (kRankQueue + TH - 1) / TH;
    static_assert(kRankQueue <= kIterMaxBatch && kRankSlots <= kPer, "s_sel holds the keys");
    if (N <= kRankQueue) {
        // staged up to a multiple of 8 with zero keys (never larger than a
        // kept key), read 16 bytes at a time
        const int N8 = (N + 7) & ~7;
#pragma unroll
        for (int j = 0; j < kRankSlots; ++j) {
            const int i = j * TH + tid;
            if (i < N8) s_sel[i] = i < N ? key[j] : 0ull;
        }
        __syncthreads();
        const ulonglong2* sel2 = reinterpret_cast<const ulonglong2*>(s_sel);
#pragma unroll
        for (int j = 0; j < kRankSlots; ++j) {
            const int i = j * TH + tid;
            if (i < N && key[j] != 0ull) {
                const unsigned long long kj = key[j];
                int rank = 0;
                for (int t = 0; t < N8 / 2; t += 4) {
                    ulonglong2 v[4];
#pragma unroll
                    for (int u = 0; u < 4; ++u) v[u] = sel2[t + u];
#pragma unroll
                    for (int u = 0; u < 4; ++u) rank += (v[u].x > kj) + (v[u].y > kj);
                }
                if (rank < s) bq[rank] = i;
            }
        }
        for (int j = s + tid; j < a.bs_max; j += TH) bq[j] = -1;
        return;
    }
    // Longer queues: the s-th largest key (at least s are non-zero, since
    // |Q_s| >= s) by a radix select, most significant digit first.  Pass by
    // pass, the keys that agree with the digits fixed so far are counted
    // per next digit; the digit is the largest whose suffix count reaches
    // the number of keys still needed, which then drops by the count of the
    // larger digits.
    unsigned long long prefix = 0ull, pmask = 0ull;
    int need = s;
    for (int shift = 56; shift >= 0; shift -= 8) {
        unsigned* hist = s_hist[(shift >> 3) & 1];    // two buffers: the other one is cleared here
        if (tid < 256) s_hist[((shift >> 3) & 1) ^ 1][tid] = 0u;
#pragma unroll
        for (int j = 0; j < kPer; ++j)
            if (key[j] != 0ull && (key[j] & pmask) == prefix)
                atomicAdd(&hist[(unsigned)(key[j] >> shift) & 255u], 1u);
        __syncthreads();
        // suffix sums over the digits: thread t < 256 holds digit 255 - t,
        // so an inclusive prefix scan over t counts the keys with digit
        // >= 255 - t (the first four waves, whole)
        const bool hw = tid < 256;
        unsigned mine = 0u, incl = 0u;
        if (hw) {
            mine = hist[255 - tid];
            incl = mine;
            for (int o = 1; o < 64; o <<= 1) {
                const unsigned up = __shfl_up(incl, o, 64);
                if (lane >= o) incl += up;
            }
            if (lane == 63) s_wsum[wv] = incl;
        }
        __syncthreads();
        if (hw) {
            for (int i = 0; i < wv; ++i) incl += s_wsum[i];
            const unsigned excl = incl - mine;
            // exactly one thread sees the crossing: keys with larger digits
            // are fewer than `need`, with this digit included they are enough
            if (excl < (unsigned)need && incl >= (unsigned)need) {
                s_digit = 255 - tid;
                s_need = need - (int)excl;
            }
        }
        __syncthreads();
        prefix |= (unsigned long long)s_digit << shift;
        pmask |= 255ull << shift;
        need = s_need;
    }
    const unsigned long long lo_k = prefix;
    // the selected keys, then each one's rank among them
#pragma unroll
    for (int j = 0; j < kPer; ++j)
        if (key[j] >= lo_k && key[j] != 0ull) {
            const int slot = atomicAdd(&s_nsel, 1);
            if (slot < kIterMaxBatch) s_sel[slot] = key[j];
        }
    __syncthreads();
    const int nsel = min(s_nsel, min(s, kIterMaxBatch));
    for (int j = tid; j < nsel; j += TH) {
        const unsigned long long kj = s_sel[j];
        int rank = 0;
        for (int i = 0; i < nsel; ++i) rank += s_sel[i] > kj;
        bq[rank] = (int32_t)(0xffffffffu - (unsigned)(kj & 0xffffffffull));
    }
    for (int j = nsel + tid; j < a.bs_max; j += TH) bq[j] = -1;
}

// ---------------------------------------------------------------------------
// accumulate_kernel: profiler feedback.  One thread per sample (grid-stride):
// validate, bin by floor(latency / w) with the last bin catching the tail,
// and add one count with a device-scope atomic.
// ---------------------------------------------------------------------------
struct AccArgs {
    const int32_t* model;
    const int32_t* bs_index;
    const int32_t* cls;
    const double* latency;
    const double* width;
    uint32_t* counts;
    unsigned long long* n_rejected;
    int64_t n;
    int M, nbs, C, K;
};

__global__ __launch_bounds__(kThreads) void accumulate_kernel(const AccArgs a) {
    unsigned long long rejected = 0;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < a.n;
         i += (int64_t)gridDim.x * kThreads) {
        const int q = a.model[i], b = a.bs_index[i], c = a.cls[i];
        const double lat = a.latency[i];
        if (q < 0 || q >= a.M || b < 0 || b >= a.nbs || c < 0 || c >= a.C ||
            !(lat >= 0.0 && lat < HUGE_VAL)) {
            ++rejected;
            continue;
        }
        const double w = a.width[q];
        if (!(w > 0.0)) {
            ++rejected;
            continue;
        }
        const double u = floor(lat / w);
        const int k = u >= (double)(a.K - 1) ? a.K - 1 : (int)u;
        atomicAdd(a.counts + (((size_t)q * a.nbs + b) * a.C + c) * (size_t)a.K + k, 1u);
    }
    if (a.n_rejected && rejected) atomicAdd(a.n_rejected, rejected);
}

}  // namespace

namespace {


int hip_fail(orloj_ctx* ctx, hipError_t e, const char* what) {
    return orloj_ctx_fail(ctx, ORLOJ_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

int check_grid(orloj_ctx* ctx, const orloj_grid* g) {
    if (!g) return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "grid is NULL");
    if (g->n_models < 0) return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "n_models < 0");
    if (g->n_classes < 1) return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "n_classes < 1");
    if (g->n_bins < 1) return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "n_bins < 1");
    if (g->n_bins > ORLOJ_MAX_BINS)
        return orloj_ctx_fail(ctx, ORLOJ_E_UNSUPPORTED, "n_bins %d > %d", g->n_bins, ORLOJ_MAX_BINS);
    if (g->n_bs < 1) return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "n_bs < 1");
    if (g->n_bs > ORLOJ_MAX_BATCH_SIZES)
        return orloj_ctx_fail(ctx, ORLOJ_E_UNSUPPORTED, "n_bs %d > %d", g->n_bs, ORLOJ_MAX_BATCH_SIZES);
    if (!g->batch_sizes) return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "batch_sizes is NULL");
    for (int i = 0; i < g->n_bs; ++i) {
        if (g->batch_sizes[i] < 1) return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "batch size < 1");
        if (i > 0 && g->batch_sizes[i] <= g->batch_sizes[i - 1])
            return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "batch sizes not strictly increasing");
    }
    if (g->n_models > 0 && !g->d_bin_width_ms)
        return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "d_bin_width_ms is NULL");
    return ORLOJ_OK;
}

int check_queues(orloj_ctx* ctx, const orloj_grid* g, const orloj_queues* qs) {
    if (!qs) return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "queues is NULL");
    if (!qs->h_queue_off) return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "h_queue_off is NULL");
    if (qs->h_queue_off[0] != 0) return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "h_queue_off[0] != 0");
    for (int q = 0; q < g->n_models; ++q)
        if (qs->h_queue_off[q + 1] < qs->h_queue_off[q])
            return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "h_queue_off decreases at model %d", q);
    if (g->n_models > 0) {
        if (!qs->d_queue_off || !qs->d_now_ms)
            return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "d_queue_off / d_now_ms is NULL");
        if (qs->h_queue_off[g->n_models] > 0 && (!qs->d_class || !qs->d_deadline_ms))
            return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "d_class / d_deadline_ms is NULL");
    }
    return ORLOJ_OK;
}

int64_t ncap_of(int64_t N, int bsz, int rect) { return rect ? N : (N < bsz ? N : (int64_t)bsz); }

int chunk_per_lane(int K) {
    int c = 1;
    while (c * kThreads < K) c <<= 1;
    return c;
}


template <int CPL, bool EXACT, int CR, bool AFF, bool ESPLIT>
hipError_t launch_score_v(const ScoreArgs& a, unsigned grid, hipStream_t st) {
    // the tabulated launches that take their E sums from emax_kernel are
    // small ones (or split into chunks): few waves per SIMD to hide a row
    // load's latency, so their ring is deeper
    constexpr int PF = (ESPLIT && !AFF) ? ORLOJ_SPLIT_PREFETCH : ORLOJ_SCORE_PREFETCH;
    const size_t sm = score_fixed_bytes<CPL>() + (size_t)a.maxcap * score_bytes_per_member();
    static size_t attr_bytes = 0;   // per template instance; device-independent
    if (sm > attr_bytes) {
        hipError_t e = hipFuncSetAttribute((const void*)score_kernel<CPL, PF, EXACT, CR, AFF, ESPLIT>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)sm);
        if (e != hipSuccess) return e;
        attr_bytes = sm;
    }
    hipLaunchKernelGGL((score_kernel<CPL, PF, EXACT, CR, AFF, ESPLIT>), dim3(grid), dim3(64), sm,
                       st, a);
    return hipGetLastError();
}

// Bins per lane chunk: panels of 64 chunks of CPL bins, at most kMaxChunk
// bins per lane (larger rows take more panels).  Wider panels spread each
// step's cross-lane reductions over more bins; narrower ones need fewer
// registers (more waves per SIMD) and re-read a repeated class's row slice
// sooner, while it may still sit in L2.  16 bins per lane (144 VGPRs, three
// waves per SIMD) balances the two on gfx950.
constexpr int kMaxChunk = 16;

int score_chunk_of(int K) {
    int c = 1;
    while (c < kMaxChunk && 64 * c < K) c <<= 1;
    return c;
}
// The affine mode's score waves read only the bins up to their members'
// deadlines (E[L_B] comes from emax_kernel), which at large batch sizes
// are a few hundred: narrower panels there mean less work per step and
// fewer registers.
#ifndef ORLOJ_AFFINE_CHUNK
#define ORLOJ_AFFINE_CHUNK 4
#endif
constexpr int kAffineChunk = ORLOJ_AFFINE_CHUNK;

int affine_chunk(int K) {
    int c = std::min(score_chunk_of(K), kAffineChunk);
    while ((K + 64 * c - 1) / (64 * c) > kMaxPanels) c <<= 1;   // a lane per panel's first member
    return c;
}

int score_chunk(int K) { return score_chunk_of(K); }

// Step carries: one register per 64 steps (longest prefix up to 64, or up to
// the compiled limit).
template <int CPL, bool EXACT, bool AFF, bool ESPLIT>
hipError_t launch_score_c(const ScoreArgs& a, unsigned grid, hipStream_t st) {
    constexpr int CRL = (ORLOJ_MAX_PREFIX + 63) / 64;
    return a.maxcap <= 64 ? launch_score_v<CPL, EXACT, 1, AFF, ESPLIT>(a, grid, st)
                          : launch_score_v<CPL, EXACT, CRL, AFF, ESPLIT>(a, grid, st);
}

template <int CPL, bool AFF, bool ESPLIT>
hipError_t launch_score_m(const ScoreArgs& a, unsigned grid, hipStream_t st) {
    return a.K % (64 * CPL) == 0 ? launch_score_c<CPL, true, AFF, ESPLIT>(a, grid, st)
                                 : launch_score_c<CPL, false, AFF, ESPLIT>(a, grid, st);
}

// Affine mode: E sums from emax_kernel.  Tabulated mode: from emax_kernel
// when the launch is split into step chunks over rows of more than two
// panels (a.psum set), else summed by the score waves themselves.
template <int CPL>
hipError_t launch_score(const ScoreArgs& a, unsigned grid, hipStream_t st) {
    if (a.c1) return launch_score_m<CPL, true, true>(a, grid, st);
    return a.psum ? launch_score_m<CPL, false, true>(a, grid, st)
                  : launch_score_m<CPL, false, false>(a, grid, st);
}

// emax_kernel: the tabulated kernel's panel width, so that its per-panel
// sums round as that kernel's do.  One wave per (pair, panel): pairs are
// models in the affine mode, (model, batch size) pairs in the tabulated one.
template <int CPL, bool AFF>
hipError_t launch_emax_m(const ScoreArgs& a, hipStream_t st) {
    const unsigned pairs = AFF ? (unsigned)a.Mg : (unsigned)a.Mg * (unsigned)a.nbs;
    const unsigned g = pairs * (unsigned)a.np_e;
    const bool exact = a.K % (64 * CPL) == 0;
    constexpr int CRL = (ORLOJ_MAX_PREFIX + 63) / 64;
    if (a.maxcap <= 64) {
        if (exact) hipLaunchKernelGGL((emax_kernel<CPL, true, 1, AFF>), dim3(g), dim3(64), 0, st, a);
        else hipLaunchKernelGGL((emax_kernel<CPL, false, 1, AFF>), dim3(g), dim3(64), 0, st, a);
    } else {
        if (exact) hipLaunchKernelGGL((emax_kernel<CPL, true, CRL, AFF>), dim3(g), dim3(64), 0, st, a);
        else hipLaunchKernelGGL((emax_kernel<CPL, false, CRL, AFF>), dim3(g), dim3(64), 0, st, a);
    }
    return hipGetLastError();
}

template <int CPL>
hipError_t launch_emax(const ScoreArgs& a, hipStream_t st) {
    return a.c1 ? launch_emax_m<CPL, true>(a, st) : launch_emax_m<CPL, false>(a, st);
}

template <int CPL, bool EXACT, int CR>
hipError_t launch_round_v(const ScoreArgs& a, unsigned n_emax, unsigned grid, hipStream_t st) {
    const size_t sm = score_fixed_bytes<CPL>() + (size_t)a.maxcap * score_bytes_per_member();
    static size_t attr_bytes = 0;   // per template instance; device-independent
    if (sm > attr_bytes) {
        hipError_t e = hipFuncSetAttribute((const void*)round_kernel<CPL, EXACT, CR>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)sm);
        if (e != hipSuccess) return e;
        attr_bytes = sm;
    }
    hipLaunchKernelGGL((round_kernel<CPL, EXACT, CR>), dim3(grid), dim3(64), sm, st, a, n_emax);
    return hipGetLastError();
}

template <int CPL>
hipError_t launch_round(const ScoreArgs& a, unsigned n_emax, unsigned grid, hipStream_t st) {
    constexpr int CRL = (ORLOJ_MAX_PREFIX + 63) / 64;
    const bool exact = a.K % (64 * CPL) == 0;
    if (a.maxcap <= 64)
        return exact ? launch_round_v<CPL, true, 1>(a, n_emax, grid, st)
                     : launch_round_v<CPL, false, 1>(a, n_emax, grid, st);
    return exact ? launch_round_v<CPL, true, CRL>(a, n_emax, grid, st)
                 : launch_round_v<CPL, false, CRL>(a, n_emax, grid, st);
}

template <int VPT>
hipError_t launch_cdf(const uint32_t* c, float* o, int32_t* sup, int64_t rows, int K, int* err,
                      hipStream_t st) {
    const int64_t cap = 1 << 20;
    const unsigned grid = (unsigned)(rows < cap ? rows : cap);
    hipLaunchKernelGGL(cdf_kernel<VPT>, dim3(grid), dim3(kThreads), 0, st, c, o, sup, rows, K, err);
    return hipGetLastError();
}

}  // namespace

// Scratch of orloj_score_candidates_affine_noalloc: the per-(model, panel,
// prefix length) sums of 1 - G that emax_kernel writes and score_kernel
// reads, in a fixed device array instead of the context's grown block.  Each
// device the library runs on holds its own copy until the process ends.  In
// host code `scratch` names a host-side stand-in: kernels are given the
// device address that hipGetSymbolAddress returns for the current device.
constexpr size_t kNoAllocScratchFloats = ORLOJ_NOALLOC_SCRATCH_FLOATS;
static __device__ __align__(256) float scratch[kNoAllocScratchFloats];

namespace {

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
bool g_scratch_done[kMaxScratchDevices];
hipError_t g_scratch_err[kMaxScratchDevices];
float* g_scratch_ptr[kMaxScratchDevices];

// Device address of `scratch` on `device`, looked up once per device with
// that device current (the caller has made it current).
float* scratch_address(int device, hipError_t* err) {
    if (device < 0 || device >= kMaxScratchDevices) {
        *err = hipErrorInvalidDevice;
        return nullptr;
    }
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_done[device]) {
        void* ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        g_scratch_err[device] = e;
        g_scratch_ptr[device] = e == hipSuccess ? static_cast<float*>(ptr) : nullptr;
        g_scratch_done[device] = true;
    }
    *err = g_scratch_err[device];
    return g_scratch_ptr[device];
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
    ctx->d_fill = nullptr;
    ctx->d_work = nullptr;
    ctx->work_bytes = 0;
    ctx->noalloc_scratch = nullptr;
    ctx->noalloc_err = hipSuccess;
    ctx->msg[0] = 0;
    int n = 0;
    if (hipGetDeviceCount(&n) != hipSuccess || hip_device < 0 || hip_device >= n) {
        delete ctx;
        return ORLOJ_E_INVALID;
    }
    float fill[kFillFloats];
    for (int i = 0; i < kFillFloats; ++i) fill[i] = i < kFillFloats / 2 ? 0.0f : 1.0f;
    hipError_t e = hipSetDevice(hip_device);
    ctx->n_cu = 0;
    ctx->chunk_pref = -1;
    if (e == hipSuccess) e = hipDeviceGetAttribute(&ctx->n_cu, hipDeviceAttributeMultiprocessorCount, hip_device);
    if (e == hipSuccess) e = hipMalloc((void**)&ctx->d_err, sizeof(int));
    if (e == hipSuccess) e = hipMemset(ctx->d_err, 0, sizeof(int));
    if (e == hipSuccess) e = hipMalloc((void**)&ctx->d_fill, sizeof fill);
    if (e == hipSuccess) e = hipMemcpy(ctx->d_fill, fill, sizeof fill, hipMemcpyHostToDevice);
    // the allocation-free scorer's scratch on this device (its failure only
    // disables that entry point)
    if (e == hipSuccess) ctx->noalloc_scratch = scratch_address(hip_device, &ctx->noalloc_err);
    if (e != hipSuccess) {
        if (ctx->d_err) (void)hipFree(ctx->d_err);
        if (ctx->d_fill) (void)hipFree(ctx->d_fill);
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
    if (ctx->d_fill) (void)hipFree(ctx->d_fill);
    if (ctx->d_work) (void)hipFree(ctx->d_work);
    delete ctx;
}

int orloj_set_score_chunk(orloj_ctx* ctx, int32_t steps) {
    if (!ctx) return ORLOJ_E_INVALID;
    if (steps < -1) return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "score chunk %d < -1", steps);
    ctx->chunk_pref = steps;
    return ORLOJ_OK;
}

int orloj_set_stream(orloj_ctx* ctx, void* hip_stream) {
    if (!ctx) return ORLOJ_E_INVALID;
    if ((hipStream_t)hip_stream != ctx->stream && ctx->d_work) {
        // calls still queued on the old stream may use the scratch
        hipError_t e = hipSetDevice(ctx->device);
        if (e == hipSuccess) e = hipStreamSynchronize(ctx->stream);
        if (e != hipSuccess) return hip_fail(ctx, e, "hipStreamSynchronize");
    }
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
        return orloj_ctx_fail(ctx, ORLOJ_E_DATA, "device data error:%s%s%s%s%s%s%s%s%s",
                    (flags & kErrEmptyHistogram) ? " histogram-with-no-samples" : "",
                    (flags & kErrClassRange) ? " class-id-out-of-range" : "",
                    (flags & kErrDeadlineNaN) ? " NaN-deadline" : "",
                    (flags & kErrUnsorted) ? " deadlines-not-sorted" : "",
                    (flags & kErrNowNaN) ? " NaN-now" : "",
                    (flags & kErrWidth) ? " bin-width-not-positive" : "",
                    (flags & kErrWeights) ? " class-weights-invalid" : "",
                    (flags & kErrCost) ? " cost-or-steps-invalid" : "",
                    (flags & kErrAffine) ? " affine-constants-invalid" : "");
    }
    return ORLOJ_OK;
}

int orloj_build_cdfs(orloj_ctx* ctx, int64_t n_rows, int32_t n_bins, const uint32_t* d_counts,
                     float* d_ccdf, int32_t* d_support) {
    if (!ctx) return ORLOJ_E_INVALID;
    if (n_rows < 0) return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "n_rows < 0");
    if (n_bins < 1) return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "n_bins < 1");
    if (n_bins > ORLOJ_MAX_BINS)
        return orloj_ctx_fail(ctx, ORLOJ_E_UNSUPPORTED, "n_bins %d > %d", n_bins, ORLOJ_MAX_BINS);
    if (n_rows == 0) return ORLOJ_OK;
    if (!d_counts || !d_ccdf) return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "NULL buffer");
    const char* cb = (const char*)d_counts;
    const char* ob = (const char*)d_ccdf;
    const size_t bytes = (size_t)n_rows * (size_t)n_bins * 4;
    if (cb < ob + bytes && ob < cb + bytes)
        return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "d_counts and d_ccdf overlap");
    if (d_support) {
        const char* sb = (const char*)d_support;
        const size_t sbytes = (size_t)n_rows * 8;
        if ((sb < ob + bytes && ob < sb + sbytes) || (sb < cb + bytes && cb < sb + sbytes))
            return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "d_support overlaps d_counts or d_ccdf");
    }
    hipError_t e = hipSetDevice(ctx->device);
    if (e != hipSuccess) return hip_fail(ctx, e, "hipSetDevice");
    const int vpt = chunk_per_lane(n_bins);
    switch (vpt) {
        case 1: e = launch_cdf<1>(d_counts, d_ccdf, d_support, n_rows, n_bins, ctx->d_err, ctx->stream); break;
        case 2: e = launch_cdf<2>(d_counts, d_ccdf, d_support, n_rows, n_bins, ctx->d_err, ctx->stream); break;
        case 4: e = launch_cdf<4>(d_counts, d_ccdf, d_support, n_rows, n_bins, ctx->d_err, ctx->stream); break;
        case 8: e = launch_cdf<8>(d_counts, d_ccdf, d_support, n_rows, n_bins, ctx->d_err, ctx->stream); break;
        case 16: e = launch_cdf<16>(d_counts, d_ccdf, d_support, n_rows, n_bins, ctx->d_err, ctx->stream); break;
        default: e = launch_cdf<32>(d_counts, d_ccdf, d_support, n_rows, n_bins, ctx->d_err, ctx->stream); break;
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

}  // extern "C"

namespace {

// Prefix steps per score workgroup.  A (model, batch size) workgroup runs
// its steps one after another, so a launch with too few workgroups to fill
// the chip lasts as long as its longest one.  Splitting the steps into
// chunks, each of which first rebuilds G over the steps before it with
// warm-up steps (about a fifth of a scored step), shortens that chain at
// the price of the warm-up work.  Only launches whose workgroups occupy
// fewer than half the SIMDs (`active` pairs with candidates against
// `simds`) and whose rows span at most two panels are split: every chunk
// repeats the product over the panels past its members' deadlines, which
// in rows of more panels costs as much as it saves.  Cost model, in scored
// steps: max(longest workgroup, all work / slots), where a SIMD is worth
// 1.5 slots (one wave alone on a SIMD runs at about half the rate three
// waves sharing it reach together); a chunk size is taken only if it is 10%
// faster than none.  Chunks of 4 only where the warm-up runs in its own
// loop with a deep prefetch ring (launches with an E pre-pass); elsewhere
// warm-up steps wait on their row loads.  Measured: this picks the fastest
// of none, 8, 16 and 32
// at configurations 1 to 3 and leaves configuration 5's saturated launch
// and scheduling-loop rounds unsplit.
int pick_chunk(const orloj_grid* g, const orloj_queues* qs, int mode, int64_t maxcap,
               int64_t active, int simds, int panels, bool warm_loop) {
    if (2 * active > simds || panels > 2) return 0;
    const double slots = 1.5 * simds;
    constexpr double kWarm = 0.2;
    constexpr int kCh[5] = {0, 32, 16, 8, 4};
    double total[5] = {0.0, 0.0, 0.0, 0.0, 0.0}, longest[5] = {0.0, 0.0, 0.0, 0.0, 0.0};
    for (int q = 0; q < g->n_models; ++q) {
        const int64_t N = qs->h_queue_off[q + 1] - qs->h_queue_off[q];
        if (N <= 0) continue;
        for (int bi = 0; bi < g->n_bs; ++bi) {
            const int64_t n = ncap_of(N, g->batch_sizes[bi], mode);
            total[0] += (double)n;
            longest[0] = fmax(longest[0], (double)n);
            for (int o = 1; o < 5; ++o) {
                const int64_t ch = kCh[o], k = (n + ch - 1) / ch;
                total[o] += (double)n + kWarm * ch * (double)(k * (k - 1) / 2);
                longest[o] = fmax(longest[o], kWarm * ch * (double)(k - 1) + (double)(n - (k - 1) * ch));
            }
        }
    }
    const double t_none = fmax(longest[0], total[0] / slots);
    double t_best = t_none;
    int best = 0;
    for (int o = 1; o < 5; ++o) {
        if (kCh[o] >= maxcap || (kCh[o] < 8 && !warm_loop)) continue;
        const double t = fmax(longest[o], total[o] / slots);
        if (t < 0.9 * t_none && t < t_best) {
            t_best = t;
            best = kCh[o];
        }
    }
    return best;
}

// The context's scratch, grown to at least `bytes`.  Work already enqueued
// on the context's stream may still use the old block, so the stream is
// drained before it is freed.
int ensure_work(orloj_ctx* ctx, size_t bytes) {
    if (bytes <= ctx->work_bytes) return ORLOJ_OK;
    hipError_t e = hipStreamSynchronize(ctx->stream);
    if (e != hipSuccess) return hip_fail(ctx, e, "hipStreamSynchronize");
    if (ctx->d_work) {
        e = hipFree(ctx->d_work);
        ctx->d_work = nullptr;
        ctx->work_bytes = 0;
        if (e != hipSuccess) return hip_fail(ctx, e, "hipFree");
    }
    e = hipMalloc(&ctx->d_work, bytes);
    if (e != hipSuccess) {
        ctx->d_work = nullptr;
        return e == hipErrorOutOfMemory
                   ? orloj_ctx_fail(ctx, ORLOJ_E_NOMEM, "scratch of %zu bytes", bytes)
                   : hip_fail(ctx, e, "hipMalloc");
    }
    ctx->work_bytes = bytes;
    return ORLOJ_OK;
}

// A scheduling round's tabulated score launch that left E[L_B] and the
// scores to the selection (orloj_internal_score_select).
struct Deferred {
    bool on = false;
    const float* psum = nullptr;
    int np_e = 0, maxcap = 0;
};

// Validation and launch shared by the tabulated and the affine scorer
// (d_c0 / d_c1 NULL: tabulated).
// fixed_psum (affine mode only): a caller-fixed block of fixed_floats
// floats for the panel sums instead of the context's grown one (no
// allocation; ORLOJ_E_UNSUPPORTED when the call needs more).
int score_common(orloj_ctx* ctx, const orloj_grid* grid, const float* d_ccdf,
                 const int32_t* d_support, const double* d_c0, const double* d_c1,
                 const orloj_queues* queues, double b_expo_per_ms, int32_t prefix_mode,
                 const int64_t* d_cand_off, const int64_t* d_prob_off, float* d_finish_prob,
                 double* d_expected_finish, float* d_expected_latency_ms, float* d_score,
                 float* fixed_psum = nullptr, size_t fixed_floats = 0,
                 Deferred* defer = nullptr) {
    if (!ctx) return ORLOJ_E_INVALID;
    int rc = check_grid(ctx, grid);
    if (rc) return rc;
    rc = check_queues(ctx, grid, queues);
    if (rc) return rc;
    if (prefix_mode != ORLOJ_PREFIX_TRIANGLE && prefix_mode != ORLOJ_PREFIX_RECT)
        return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "prefix_mode %d", prefix_mode);
    if (!(b_expo_per_ms > 0.0) || !isfinite(b_expo_per_ms))
        return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "b_expo_per_ms must be finite and > 0");
    const int M = grid->n_models;
    if (M == 0) return ORLOJ_OK;
    int64_t maxcap = 0, total = 0, active = 0;
    int n_act = 0;
    int act[kMaxActive];
    for (int q = 0; q < M; ++q) {
        const int64_t N = queues->h_queue_off[q + 1] - queues->h_queue_off[q];
        if (N <= 0) continue;
        if (n_act < kMaxActive) act[n_act] = q;
        ++n_act;
        for (int bi = 0; bi < grid->n_bs; ++bi) {
            const int64_t c = ncap_of(N, grid->batch_sizes[bi], prefix_mode);
            if (c > maxcap) maxcap = c;
            total += c;
            active += c > 0;
        }
    }
    if (maxcap > ORLOJ_MAX_PREFIX)
        return orloj_ctx_fail(ctx, ORLOJ_E_UNSUPPORTED, "prefix of %lld members > %d",
                    (long long)maxcap, ORLOJ_MAX_PREFIX);
    if (total == 0) return ORLOJ_OK;
    if (!d_ccdf || !d_cand_off || !d_prob_off || !d_finish_prob || !d_expected_finish ||
        !d_expected_latency_ms || !d_score)
        return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "NULL device buffer");
    // bins per lane of the score kernel (the affine mode reads only its
    // members' bins, in narrower panels)
    const int cpl = d_c1 ? affine_chunk(grid->n_bins) : score_chunk(grid->n_bins);
    const int panels = (grid->n_bins + 64 * cpl - 1) / (64 * cpl);
    // Tabulated rows of more than two panels, in a launch too small to fill
    // the chip or split into step chunks: every panel's E sums come from
    // emax_kernel (one wave per (model, batch size, panel), in parallel),
    // and the score waves walk only the panels that hold members (one, as
    // far as the chunk cost model knows), so chunks repeat only those.
    // Chunk setting 0 (never split) keeps the single pass.
    const int simds = 4 * (ctx->n_cu > 0 ? ctx->n_cu : 256);
    const bool esplit_ok = !d_c1 && panels > 2;
    const int chunk = ctx->chunk_pref >= 0
                          ? (ctx->chunk_pref < maxcap ? ctx->chunk_pref : 0)
                          : pick_chunk(grid, queues, prefix_mode, maxcap, active, simds,
                                       esplit_ok ? 1 : panels, esplit_ok);
    const bool esplit = esplit_ok && (chunk > 0 || (ctx->chunk_pref < 0 && 2 * active <= simds));
    const int nchunk = chunk ? (int)((maxcap + chunk - 1) / chunk) : 1;
    // only the models with a queue get workgroups, when they are few enough
    // to list
    const bool compact = n_act < M && n_act <= kMaxActive;
    const int Mg = compact ? n_act : M;
    const int64_t nblk = (int64_t)Mg * grid->n_bs * nchunk;
    if (nblk > 0x7fffffff) return orloj_ctx_fail(ctx, ORLOJ_E_UNSUPPORTED, "too many (model, batch size) pairs");

    ScoreArgs a;
    a.defer = 0;
    a.chunk = chunk;
    a.nchunk = nchunk;
    a.tab = d_ccdf;
    a.sup = d_support;
    a.c0 = d_c0;
    a.c1 = d_c1;
    a.cost = queues->d_cost;
    a.fill = ctx->d_fill;
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
    a.Mg = Mg;
    a.compact = compact ? 1 : 0;
    memset(a.bs, 0, sizeof a.bs);
    for (int i = 0; i < grid->n_bs; ++i) a.bs[i] = grid->batch_sizes[i];
    memset(a.act, 0, sizeof a.act);
    if (compact)
        for (int i = 0; i < n_act; ++i) a.act[i] = act[i];

    hipError_t e = hipSetDevice(ctx->device);
    if (e != hipSuccess) return hip_fail(ctx, e, "hipSetDevice");
    a.psum = nullptr;
    a.np_e = 0;
    // emax_kernel's panels: the score waves' own in the tabulated mode (its
    // sums must round as theirs do); in the affine mode the narrow panels of
    // the affine score waves, so that four times as many waves share the
    // products of a model's few hundred prefixes
    const int cple = d_c1 ? cpl : score_chunk(grid->n_bins);
    if (d_c1 || esplit) {
        // emax_kernel's panel sums, formed first: [pairs][panels][maxcap]
        // floats, pairs = models (affine) or (model, batch size) pairs
        const int64_t np = (grid->n_bins + 64 * cple - 1) / (64 * cple);
        const int64_t pairs = d_c1 ? (int64_t)M : (int64_t)M * grid->n_bs;
        if (pairs * np > 0x7fffffff)
            return orloj_ctx_fail(ctx, ORLOJ_E_UNSUPPORTED, "too many (pair, panel) pairs");
        const size_t need = (size_t)pairs * (size_t)np * (size_t)maxcap;
        if (fixed_psum) {
            if (need > fixed_floats)
                return orloj_ctx_fail(ctx, ORLOJ_E_UNSUPPORTED,
                                      "the call needs %zu scratch floats (models x panels x longest "
                                      "prefix), the fixed scratch holds %zu",
                                      need, fixed_floats);
            a.psum = fixed_psum;
        } else {
            rc = ensure_work(ctx, need * sizeof(float));
            if (rc) return rc;
            a.psum = (float*)ctx->d_work;
        }
        a.np_e = (int)np;
        if (defer && !d_c1 && cple == cpl) {
            // a scheduling round: emax_kernel's and score_kernel's waves in
            // one launch, E[L_B] and the scores finished by the selection
            a.defer = 1;
            const unsigned n_emax = (unsigned)(Mg * grid->n_bs) * (unsigned)np;
            const unsigned g = n_emax + (unsigned)nblk;
            switch (cpl) {
                case 1: e = launch_round<1>(a, n_emax, g, ctx->stream); break;
                case 2: e = launch_round<2>(a, n_emax, g, ctx->stream); break;
                case 4: e = launch_round<4>(a, n_emax, g, ctx->stream); break;
                case 8: e = launch_round<8>(a, n_emax, g, ctx->stream); break;
                default: e = launch_round<16>(a, n_emax, g, ctx->stream); break;
            }
            if (e != hipSuccess) return hip_fail(ctx, e, "round_kernel launch");
            defer->on = true;
            defer->psum = a.psum;
            defer->np_e = a.np_e;
            defer->maxcap = a.maxcap;
            return ORLOJ_OK;
        }
        switch (cple) {
            case 1: e = launch_emax<1>(a, ctx->stream); break;
            case 2: e = launch_emax<2>(a, ctx->stream); break;
            case 4: e = launch_emax<4>(a, ctx->stream); break;
            case 8: e = launch_emax<8>(a, ctx->stream); break;
            default: e = launch_emax<16>(a, ctx->stream); break;
        }
        if (e != hipSuccess) return hip_fail(ctx, e, "emax_kernel launch");
    }
    const unsigned g = (unsigned)nblk;
    static_assert(kMaxChunk == 16, "launch table below");
    static_assert((ORLOJ_MAX_BINS + 64 * kMaxChunk - 1) / (64 * kMaxChunk) <= kMaxPanels, "panels");
    switch (cpl) {
        case 1: e = launch_score<1>(a, g, ctx->stream); break;
        case 2: e = launch_score<2>(a, g, ctx->stream); break;
        case 4: e = launch_score<4>(a, g, ctx->stream); break;
        case 8: e = launch_score<8>(a, g, ctx->stream); break;
        default: e = launch_score<16>(a, g, ctx->stream); break;
    }
    if (e != hipSuccess) return hip_fail(ctx, e, "score_kernel launch");
    return ORLOJ_OK;
}

// orloj_select_batch, and the finishing selection of a scheduling round
// (fin->on: E[L_B] and the scores are formed here from the panel sums and
// the priority sums in d_score, and written to d_EL and d_score).
int select_common(orloj_ctx* ctx, const orloj_grid* grid, const orloj_queues* queues,
                  int32_t prefix_mode, const int64_t* d_cand_off, float* d_score,
                  int32_t* d_sel_n, int32_t* d_sel_bs, float* d_sel_score, const Deferred* fin,
                  float* d_EL, int32_t* d_done = nullptr, int32_t round = 0, int* n_groups = nullptr) {
    if (!ctx) return ORLOJ_E_INVALID;
    int rc = check_grid(ctx, grid);
    if (rc) return rc;
    rc = check_queues(ctx, grid, queues);
    if (rc) return rc;
    if (prefix_mode != ORLOJ_PREFIX_TRIANGLE && prefix_mode != ORLOJ_PREFIX_RECT)
        return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "prefix_mode %d", prefix_mode);
    const int M = grid->n_models;
    if (M == 0) return ORLOJ_OK;
    if (!d_cand_off || !d_sel_n || !d_sel_bs || !d_sel_score)
        return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "NULL device buffer");
    const int64_t total = queues->h_queue_off[M];
    if (total > 0 && !d_score) return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "d_score is NULL");
    SelectArgs a;
    a.finish = fin && fin->on ? 1 : 0;
    a.done = d_done;
    a.round = round;
    a.psum = a.finish ? fin->psum : nullptr;
    a.np_e = a.finish ? fin->np_e : 0;
    a.maxcap = a.finish ? fin->maxcap : 0;
    a.width = grid->d_bin_width_ms;
    a.EL = d_EL;
    a.queue_off = queues->d_queue_off;
    a.cand_off = d_cand_off;
    a.S = d_score;
    a.sel_n = d_sel_n;
    a.sel_bs = d_sel_bs;
    a.sel_score = d_sel_score;
    a.nbs = grid->n_bs;
    a.rect = prefix_mode;
    a.M = M;
    memset(a.bs, 0, sizeof a.bs);
    for (int i = 0; i < grid->n_bs; ++i) a.bs[i] = grid->batch_sizes[i];
    // the models with a queue, when they are few enough to list: one
    // workgroup each, and one more that clears the others
    int n_act = 0;
    for (int q = 0; q < M; ++q)
        if (queues->h_queue_off[q + 1] > queues->h_queue_off[q]) {
            if (n_act < kMaxActive) a.act[n_act] = q;
            ++n_act;
        }
    a.compact = n_act < M && n_act <= kMaxActive;
    a.n_act = n_act;
    const unsigned g = a.compact ? (unsigned)(n_act + 1) : (unsigned)M;
    if (n_groups) *n_groups = (int)g;
    hipError_t e = hipSetDevice(ctx->device);
    if (e != hipSuccess) return hip_fail(ctx, e, "hipSetDevice");
    hipLaunchKernelGGL(select_kernel, dim3(g), dim3(kSelThreads), 0, ctx->stream, a);
    e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(ctx, e, "select_kernel launch");
    return ORLOJ_OK;
}

}  // namespace

extern "C" {

int orloj_score_candidates(orloj_ctx* ctx, const orloj_grid* grid, const float* d_ccdf,
                           const int32_t* d_support, const orloj_queues* queues, double b_expo_per_ms, int32_t prefix_mode,
                           const int64_t* d_cand_off, const int64_t* d_prob_off,
                           float* d_finish_prob, double* d_expected_finish,
                           float* d_expected_latency_ms, float* d_score) {
    return score_common(ctx, grid, d_ccdf, d_support, nullptr, nullptr, queues, b_expo_per_ms,
                        prefix_mode, d_cand_off, d_prob_off, d_finish_prob, d_expected_finish,
                        d_expected_latency_ms, d_score);
}

int orloj_score_candidates_affine(orloj_ctx* ctx, const orloj_grid* grid, const float* d_ccdf,
                                  const int32_t* d_support, const double* d_c0_ms,
                                  const double* d_c1, const orloj_queues* queues,
                                  double b_expo_per_ms, int32_t prefix_mode,
                                  const int64_t* d_cand_off, const int64_t* d_prob_off,
                                  float* d_finish_prob, double* d_expected_finish,
                                  float* d_expected_latency_ms, float* d_score) {
    if (!ctx) return ORLOJ_E_INVALID;
    if (grid && grid->n_models > 0 && (!d_c0_ms || !d_c1))
        return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "d_c0_ms / d_c1 is NULL");
    return score_common(ctx, grid, d_ccdf, d_support, d_c0_ms, d_c1, queues, b_expo_per_ms,
                        prefix_mode, d_cand_off, d_prob_off, d_finish_prob, d_expected_finish,
                        d_expected_latency_ms, d_score);
}

int orloj_score_candidates_affine_noalloc(orloj_ctx* ctx, const orloj_grid* grid,
                                          const float* d_ccdf, const int32_t* d_support,
                                          const double* d_c0_ms, const double* d_c1,
                                          const orloj_queues* queues, double b_expo_per_ms,
                                          int32_t prefix_mode, const int64_t* d_cand_off,
                                          const int64_t* d_prob_off, float* d_finish_prob,
                                          double* d_expected_finish,
                                          float* d_expected_latency_ms, float* d_score) {
    if (!ctx) return ORLOJ_E_INVALID;
    if (grid && grid->n_models > 0 && (!d_c0_ms || !d_c1))
        return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "d_c0_ms / d_c1 is NULL");
    if (!ctx->noalloc_scratch)
        return orloj_ctx_fail(ctx, ORLOJ_E_HIP, "fixed scratch unavailable on device %d: %s",
                              ctx->device, hipGetErrorString(ctx->noalloc_err));
    return score_common(ctx, grid, d_ccdf, d_support, d_c0_ms, d_c1, queues, b_expo_per_ms,
                        prefix_mode, d_cand_off, d_prob_off, d_finish_prob, d_expected_finish,
                        d_expected_latency_ms, d_score, ctx->noalloc_scratch,
                        kNoAllocScratchFloats);
}

int orloj_build_model_laws(orloj_ctx* ctx, const orloj_grid* grid, const float* d_ccdf,
                           const double* d_class_weights, double b_expo_per_ms, float* d_law,
                           float* d_disc, float* d_model_el) {
    if (!ctx) return ORLOJ_E_INVALID;
    int rc = check_grid(ctx, grid);
    if (rc) return rc;
    if (!(b_expo_per_ms > 0.0) || !isfinite(b_expo_per_ms))
        return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "b_expo_per_ms must be finite and > 0");
    if (grid->n_models == 0) return ORLOJ_OK;
    if (!d_ccdf || !d_law || !d_disc || !d_model_el)
        return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "NULL device buffer");
    const int64_t nblk = (int64_t)grid->n_models * grid->n_bs;
    if (nblk > 0x7fffffff) return orloj_ctx_fail(ctx, ORLOJ_E_UNSUPPORTED, "too many (model, batch size) pairs");
    LawArgs a;
    a.tab = d_ccdf;
    a.weights = d_class_weights;
    a.width = grid->d_bin_width_ms;
    a.law = d_law;
    a.disc = d_disc;
    a.model_el = d_model_el;
    a.err = ctx->d_err;
    a.b = b_expo_per_ms;
    a.M = grid->n_models;
    a.C = grid->n_classes;
    a.K = grid->n_bins;
    a.nbs = grid->n_bs;
    memset(a.bs, 0, sizeof a.bs);
    for (int i = 0; i < grid->n_bs; ++i) a.bs[i] = grid->batch_sizes[i];
    hipError_t e = hipSetDevice(ctx->device);
    if (e != hipSuccess) return hip_fail(ctx, e, "hipSetDevice");
    const unsigned g = (unsigned)nblk;
    switch (chunk_per_lane(grid->n_bins)) {
        case 1: hipLaunchKernelGGL(laws_kernel<1>, dim3(g), dim3(kThreads), 0, ctx->stream, a); break;
        case 2: hipLaunchKernelGGL(laws_kernel<2>, dim3(g), dim3(kThreads), 0, ctx->stream, a); break;
        case 4: hipLaunchKernelGGL(laws_kernel<4>, dim3(g), dim3(kThreads), 0, ctx->stream, a); break;
        case 8: hipLaunchKernelGGL(laws_kernel<8>, dim3(g), dim3(kThreads), 0, ctx->stream, a); break;
        case 16: hipLaunchKernelGGL(laws_kernel<16>, dim3(g), dim3(kThreads), 0, ctx->stream, a); break;
        default: hipLaunchKernelGGL(laws_kernel<32>, dim3(g), dim3(kThreads), 0, ctx->stream, a); break;
    }
    e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(ctx, e, "laws_kernel launch");
    return ORLOJ_OK;
}

int orloj_iterate(orloj_ctx* ctx, const orloj_grid* grid, const int32_t* d_support,
                  const float* d_law, const float* d_disc, const float* d_model_el,
                  const orloj_queues* queues, const orloj_steps* steps, double b_expo_per_ms,
                  int32_t* d_timed_out, float* d_score, int32_t* d_cand_bs, int32_t* d_batch) {
    if (!ctx) return ORLOJ_E_INVALID;
    int rc = check_grid(ctx, grid);
    if (rc) return rc;
    rc = check_queues(ctx, grid, queues);
    if (rc) return rc;
    if (!(b_expo_per_ms > 0.0) || !isfinite(b_expo_per_ms))
        return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "b_expo_per_ms must be finite and > 0");
    const int M = grid->n_models;
    if (M == 0) return ORLOJ_OK;
    const int bs_max = grid->batch_sizes[grid->n_bs - 1];
    if (bs_max > kIterMaxBatch)
        return orloj_ctx_fail(ctx, ORLOJ_E_UNSUPPORTED, "batch size %d > %d", bs_max, kIterMaxBatch);
    int64_t longest = 0;
    for (int q = 0; q < M; ++q) {
        const int64_t N = queues->h_queue_off[q + 1] - queues->h_queue_off[q];
        longest = std::max(longest, N);
        if (N > kIterMaxQueue)
            return orloj_ctx_fail(ctx, ORLOJ_E_UNSUPPORTED, "queue of model %d holds %lld > %d requests", q,
                        (long long)N, kIterMaxQueue);
    }
    if (!d_support || !d_law || !d_disc || !d_model_el || !d_cand_bs || !d_batch)
        return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "NULL device buffer");
    if (queues->h_queue_off[M] > 0 && (!d_timed_out || !d_score))
        return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "NULL per-request output");
    if (steps) {
        const int64_t* so = steps->h_step_off;
        if (!so || !steps->d_step_off || !steps->d_step_deadline_ms || !steps->d_step_cost)
            return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "incomplete orloj_steps");
        if (so[0] != 0) return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "h_step_off[0] != 0");
        for (int64_t r = 0; r < queues->h_queue_off[M]; ++r)
            if (so[r + 1] <= so[r])
                return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "request %lld has no cost step", (long long)r);
    }
    IterArgs a;
    a.sup = d_support;
    a.law = d_law;
    a.disc = d_disc;
    a.model_el = d_model_el;
    a.queue_off = queues->d_queue_off;
    a.cls = queues->d_class;
    a.deadline = queues->d_deadline_ms;
    a.now = queues->d_now_ms;
    a.width = grid->d_bin_width_ms;
    a.cost = queues->d_cost;
    a.step_off = steps ? steps->d_step_off : nullptr;
    a.step_dl = steps ? steps->d_step_deadline_ms : nullptr;
    a.step_cost = steps ? steps->d_step_cost : nullptr;
    a.timed_out = d_timed_out;
    a.score = d_score;
    a.cand_bs = d_cand_bs;
    a.batch = d_batch;
    a.err = ctx->d_err;
    a.b = b_expo_per_ms;
    a.M = M;
    a.C = grid->n_classes;
    a.K = grid->n_bins;
    a.nbs = grid->n_bs;
    a.bs_max = bs_max;
    memset(a.bs, 0, sizeof a.bs);
    for (int i = 0; i < grid->n_bs; ++i) a.bs[i] = grid->batch_sizes[i];
    hipError_t e = hipSetDevice(ctx->device);
    if (e != hipSuccess) return hip_fail(ctx, e, "hipSetDevice");
    a.part_cnt = a.part_first = nullptr;
    a.parts = 0;
    const bool stage = a.nbs > 32 && (int64_t)a.C * (a.nbs + 1) <= kIterStage;
    // A long queue on few models leaves most of the chip idle while one
    // workgroup per model walks it: the drop phase then runs in parts of
    // kDropPart requests, one workgroup each, before the rest per model.
    const int n_cu = ctx->n_cu > 0 ? ctx->n_cu : 256;
    if (longest > kIterWideQueue && 4 * (int64_t)M <= n_cu) {
        const int P = (int)((longest + kDropPart - 1) / kDropPart);
        const size_t n = (size_t)M * (size_t)P * (size_t)a.nbs;
        int rc2 = ensure_work(ctx, 2 * n * sizeof(int32_t));
        if (rc2) return rc2;
        a.part_cnt = static_cast<int32_t*>(ctx->d_work);
        a.part_first = a.part_cnt + n;
        a.parts = P;
        const dim3 g((unsigned)(M * P));
        if (stage)
            hipLaunchKernelGGL((iterate_kernel<kThreads, true, kIterDropPart>), g, dim3(kThreads), 0, ctx->stream, a);
        else
            hipLaunchKernelGGL((iterate_kernel<kThreads, false, kIterDropPart>), g, dim3(kThreads), 0, ctx->stream, a);
        e = hipGetLastError();
        if (e != hipSuccess) return hip_fail(ctx, e, "iterate_kernel launch");
        hipLaunchKernelGGL((iterate_kernel<1024, false, kIterFromParts>), dim3(M), dim3(1024), 0, ctx->stream, a);
    } else if (longest > kIterWideQueue) {
        if (stage)
            hipLaunchKernelGGL((iterate_kernel<1024, true, kIterWhole>), dim3(M), dim3(1024), 0, ctx->stream, a);
        else
            hipLaunchKernelGGL((iterate_kernel<1024, false, kIterWhole>), dim3(M), dim3(1024), 0, ctx->stream, a);
    } else if (stage) {
        hipLaunchKernelGGL((iterate_kernel<kThreads, true, kIterWhole>), dim3(M), dim3(kThreads), 0, ctx->stream, a);
    } else {
        hipLaunchKernelGGL((iterate_kernel<kThreads, false, kIterWhole>), dim3(M), dim3(kThreads), 0, ctx->stream, a);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(ctx, e, "iterate_kernel launch");
    return ORLOJ_OK;
}

int orloj_accumulate(orloj_ctx* ctx, const orloj_grid* grid, int64_t n_samples,
                     const int32_t* d_model, const int32_t* d_bs_index, const int32_t* d_class,
                     const double* d_latency_ms, uint32_t* d_counts,
                     unsigned long long* d_n_rejected) {
    if (!ctx) return ORLOJ_E_INVALID;
    int rc = check_grid(ctx, grid);
    if (rc) return rc;
    if (n_samples < 0) return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "n_samples < 0");
    if (n_samples == 0) return ORLOJ_OK;
    if (!d_model || !d_bs_index || !d_class || !d_latency_ms || !d_counts || !grid->d_bin_width_ms)
        return orloj_ctx_fail(ctx, ORLOJ_E_INVALID, "NULL device buffer");
    AccArgs a;
    a.model = d_model;
    a.bs_index = d_bs_index;
    a.cls = d_class;
    a.latency = d_latency_ms;
    a.width = grid->d_bin_width_ms;
    a.counts = d_counts;
    a.n_rejected = d_n_rejected;
    a.n = n_samples;
    a.M = grid->n_models;
    a.nbs = grid->n_bs;
    a.C = grid->n_classes;
    a.K = grid->n_bins;
    hipError_t e = hipSetDevice(ctx->device);
    if (e != hipSuccess) return hip_fail(ctx, e, "hipSetDevice");
    const int64_t want = (n_samples + kThreads - 1) / kThreads;
    const unsigned g = (unsigned)(want < 4096 ? want : 4096);
    hipLaunchKernelGGL(accumulate_kernel, dim3(g), dim3(kThreads), 0, ctx->stream, a);
    e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(ctx, e, "accumulate_kernel launch");
    return ORLOJ_OK;
}

int orloj_select_batch(orloj_ctx* ctx, const orloj_grid* grid, const orloj_queues* queues,
                       int32_t prefix_mode, const int64_t* d_cand_off, const float* d_score,
                       int32_t* d_sel_n, int32_t* d_sel_bs, float* d_sel_score) {
    return select_common(ctx, grid, queues, prefix_mode, d_cand_off, const_cast<float*>(d_score),
                         d_sel_n, d_sel_bs, d_sel_score, nullptr, nullptr);
}

}  // extern "C"

int orloj_internal_score_select(orloj_ctx* ctx, const orloj_grid* grid, const float* d_ccdf,
                                const int32_t* d_support, const orloj_queues* queues,
                                double b_expo_per_ms, const int64_t* d_cand_off,
                                const int64_t* d_prob_off, float* d_finish_prob,
                                double* d_expected_finish, float* d_expected_latency_ms,
                                float* d_score, int32_t* d_sel_n, int32_t* d_sel_bs,
                                float* d_sel_score, int32_t* d_done, int32_t round, int* n_groups) {
    Deferred fin;
    int rc = score_common(ctx, grid, d_ccdf, d_support, nullptr, nullptr, queues, b_expo_per_ms,
                          ORLOJ_PREFIX_TRIANGLE, d_cand_off, d_prob_off, d_finish_prob,
                          d_expected_finish, d_expected_latency_ms, d_score, nullptr, 0, &fin);
    if (rc) return rc;
    return select_common(ctx, grid, queues, ORLOJ_PREFIX_TRIANGLE, d_cand_off, d_score, d_sel_n,
                         d_sel_bs, d_sel_score, &fin, d_expected_latency_ms, d_done, round, n_groups);
}
