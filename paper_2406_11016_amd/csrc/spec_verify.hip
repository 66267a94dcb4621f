// Fused speculative-sampling verification for gfx950 (MI355X): kernels and C ABI.
//
// Method: arXiv 2406.11016, Sec. 3.1 (eqs. (1)-(3)) and Sec. 3.2.2 (eqs. (4)-(5)).
//
// One launch per call.  Workgroups play one of four roles by index (see
// verify_kernel):
//   stats    (exact mode) one chunk of one logit row, streamed once with
//            128-bit non-temporal loads: the chunk's contribution to the row's
//            softmax normaliser (eq. (4)).  These move every logit byte and
//            bound the step.
//   decider  b: tau_c of eq. (1) at the drafted tokens and the
//            first-rejection scan for batch element b, made once.
//   mass     (b, tile): the weights a(x) of the final distribution (residual
//            of eqs. (2)-(3), or target row gamma) summed over the tile, one
//            sub-chunk per wave.
//   draw     b: fixed-order prefix over b's sub-chunk masses, then one
//            workgroup scan inside the sub-chunk the uniform falls in -- the
//            inverse-CDF draw of the next token.
// Sigmoid mode (eq. (5)) has no stats role: it needs no row normaliser, so
// only the logits at the drafted tokens and the row(s) the next token is
// drawn from are read.
#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <cmath>

#include "spec_verify.h"
#include "sv_device.hpp"

namespace sv {

enum : int { kResidual = 0, kTargetRow = 1 };

constexpr int kWantStatsTiles = 2048;    // enough workgroups to fill 256 CUs several times
constexpr int kWantSampleTiles = 1024;
constexpr int kStatsTileBytes = 65536;   // at most 64 KiB of one row per stats workgroup
constexpr int kSampleTileBytes = 32768;

// ---------------------------------------------------------------------------
// weights of the distribution the next token is drawn from
// ---------------------------------------------------------------------------

// zp - zq as an unevaluated sum hi + lo (Knuth's two-sum): the difference of two
// logits is not exact in fp32 when their exponents are far apart (e.g. fp16
// logits near +-65504 against logits near 1).
__device__ __forceinline__ void two_diff(float a, float b, float& hi, float& lo) {
    hi = a - b;
    const float bb = hi - a;
    lo = (a - (hi - bb)) - (b + bb);
    if (!__builtin_isfinite(hi)) lo = 0.0f;  // +-inf or NaN differences carry no low part
}

constexpr float kLn2 = 0.693147180559945309f;
constexpr float kLog2e = 1.44269504088896341f;

// 2^x with the hardware exponential (about 1 ulp; results below 2^-126 flush to 0).
__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

// e^x - 1 for 0 <= x <= 0.35 by its Taylor series to degree 7 (truncation
// below 2e-8 relative), keeping full relative precision for small x.
__device__ __forceinline__ float expm1_small(float x) {
    float p = 1.0f / 5040.0f;
    p = fmaf(p, x, 1.0f / 720.0f);
    p = fmaf(p, x, 1.0f / 120.0f);
    p = fmaf(p, x, 1.0f / 24.0f);
    p = fmaf(p, x, 1.0f / 6.0f);
    p = fmaf(p, x, 0.5f);
    p = fmaf(p, x, 1.0f);
    return p * x;
}

// Exact mode, in log2 units: log2 p(x) = z_p(x) c - Lambda_p with c = log2(e)/T
// and Lambda = k + log2(s) from the row normaliser.  The residual
// a(x) = max(0, p - q) (eqs. (2)-(3)) is formed as q (2^d - 1) with
// d = log2 p(x) - log2 q(x), so p == q cancels exactly and small differences
// keep their relative precision.
struct ExactWeights {
    int kind;
    float c;
    float kp, lp_hi, lp_lo;  // target row: reference k and log2(s) as hi + lo
    float kq, lq_hi, lq_lo;  // draft row
    float d_hi, d_lo;        // Lambda_p - Lambda_q as hi + lo
    template <int KIND>
    __device__ __forceinline__ float eval(float zp, float zq) const {
        if (KIND == kTargetRow) return exp2_hw((fmaf(zp, c, -kp) - lp_hi) - lp_lo);
        float dz, dz_lo;
        two_diff(zp, zq, dz, dz_lo);
        const float d = fmaf(dz_lo, c, fmaf(dz, c, -d_hi)) - d_lo;
        if (!(d > 0.0f)) return 0.0f;
        const float q = exp2_hw((fmaf(zq, c, -kq) - lq_hi) - lq_lo);
        if (d <= 0.5f) return q * expm1_small(d * kLn2);
        return exp2_hw((fmaf(zp, c, -kp) - lp_hi) - lp_lo) - q;
    }
};

// sigma(x) = 1 / (1 + e^-x) with the hardware exponential and reciprocal.
__device__ __forceinline__ float sigm(float x) {
    return __builtin_amdgcn_rcpf(1.0f + exp2_hw(-x * kLog2e));
}

// Sigmoid mode, eq. (5): p_hat = sigma(u_p) with u = (z/T - alpha)/(beta - alpha).
// max(0, p_hat - q_hat) is formed as q_hat (1 - p_hat) expm1(u_p - u_q), exact
// in the cancellation the +-1e3 / +-1e4 scalings produce (p_hat - q_hat ~ 1e-5).
struct SigmoidWeights {
    int kind;
    float s, s0;  // u = fma(z, s, s0)
    template <int KIND>
    __device__ __forceinline__ float eval(float zp, float zq) const {
        const float up = fmaf(zp, s, s0);
        if (KIND == kTargetRow) return sigm(up);
        if (zp != zp || zq != zq) return __builtin_nanf("");
        float dz, dz_lo;
        two_diff(zp, zq, dz, dz_lo);
        const float d = fmaf(dz, s, dz_lo * s);
        if (!(d > 0.0f)) return 0.0f;
        const float uq = fmaf(zq, s, s0);
        if (d <= 0.35f) return sigm(uq) * sigm(-up) * expm1_small(d);
        if (d <= 20.0f) return sigm(uq) * sigm(-up) * (exp2_hw(d * kLog2e) - 1.0f);
        return (up < 0.0f) ? sigm(up) - sigm(uq) : sigm(-uq) - sigm(-up);
    }
};

template <class D>
__device__ __forceinline__ bool pair_aligned(const typename D::T* rp, const typename D::T* rq, bool two_rows) {
    const uintptr_t a = reinterpret_cast<uintptr_t>(rp) | (two_rows ? reinterpret_cast<uintptr_t>(rq) : 0);
    return (a & 15u) == 0;
}

// Vectors v0 + u * vstride (u < U) from a chunk of n elements of the selected
// row pair (rp/rq point at the chunk start).  All 16-byte loads are issued
// before any is used; elements at or beyond n read as -inf (weight 0), and
// with one row the draft side is -inf.
template <class D, int U>
__device__ __forceinline__ void load_pair_u(const typename D::T* rp, const typename D::T* rq, bool two_rows,
                                            bool fast, int v0, int vstride, int n, float (&zp)[U][D::E],
                                            float (&zq)[U][D::E]) {
    constexpr int E = D::E;
    const int nfull = n / E;
    if (fast && nfull > 0) {
        u32x4 a[U], c[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            a[u] = load_vec_or_pad<D, false>(rp, v0 + u * vstride, nfull);
            if (two_rows) c[u] = load_vec_or_pad<D, false>(rq, v0 + u * vstride, nfull);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            unpack<D>(a[u], zp[u]);
            if (two_rows) unpack<D>(c[u], zq[u]);
        }
        // the partial vector at the end of a row, if this thread holds it
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int v = v0 + u * vstride;
            if (v == nfull && nfull * E < n) {
                load_elems_or_pad<D>(rp, v * E, n, zp[u]);
                if (two_rows) load_elems_or_pad<D>(rq, v * E, n, zq[u]);
            }
        }
    } else {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int v = v0 + u * vstride;
            load_elems_or_pad<D>(rp, v * E, n, zp[u]);
            if (two_rows) load_elems_or_pad<D>(rq, v * E, n, zq[u]);
        }
    }
    if (!two_rows) {
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int e = 0; e < E; ++e) zq[u][e] = -INFINITY;
    }
}

constexpr int kPassUnroll = 4;  // vectors in flight per lane in the weight pass
constexpr int kMergeCap = 1024;  // chunk log-normalisers of one batch element (2 gamma + 1 rows)
constexpr int kMaxSub = 1024;    // sub-chunk masses of one batch element (nchunk2 * kWaves)
constexpr int kMaxSpins = 1 << 17;  // bound on every wait (about 0.1 s), so every wave exits
constexpr int kDecisionWords = 5;          // L and the sentinel flag, then 8 floats of weight constants

// ---------------------------------------------------------------------------
// results passed between workgroups of one launch
//
// A result is one fp64 value published as one 64-bit word with a relaxed,
// agent-scope atomic store, bit-inverted so that the all-zero word means
// "not yet published" (NaN is canonicalised first, so no value maps to zero).
// Since every result is a single word, readers need no fence: on this
// multi-XCD part a device-scope release/acquire is an L2 writeback and
// invalidate, far costlier than the spin on a word.
// ---------------------------------------------------------------------------
__device__ __forceinline__ unsigned long long encode_word(double v) {
    if (v != v) v = __builtin_nan("");
    return ~(unsigned long long)__double_as_longlong(v);
}
__device__ __forceinline__ double decode_word(unsigned long long w) { return __longlong_as_double((long long)~w); }
__device__ __forceinline__ void publish(unsigned long long* p, double v) {
    __hip_atomic_store(p, encode_word(v), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void clear_word(unsigned long long* p) {
    __hip_atomic_store(p, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// A raw 64-bit record word (never all ones), published the same way.
__device__ __forceinline__ void publish_raw(unsigned long long* p, unsigned long long v) {
    __hip_atomic_store(p, ~v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned long long pack2(float a, float b) {
    const unsigned int ua = (a != a) ? 0x7fc00000u : __float_as_uint(a);  // canonical NaN
    const unsigned int ub = (b != b) ? 0x7fc00000u : __float_as_uint(b);
    return ((unsigned long long)ua << 32) | ub;
}
__device__ __forceinline__ float unpack_hi(unsigned long long w) { return __uint_as_float((unsigned int)(w >> 32)); }
__device__ __forceinline__ float unpack_lo(unsigned long long w) { return __uint_as_float((unsigned int)w); }

// Waits until the n raw words at p are published and copies them to dst.
__device__ __forceinline__ bool wait_raw(unsigned long long* p, int n, unsigned long long* dst) {
    for (int spin = 0;; ++spin) {
        int missing = 0;
        for (int i = threadIdx.x; i < n; i += kThreads) {
            const unsigned long long w = __hip_atomic_load(p + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (w == 0ull)
                missing = 1;
            else
                dst[i] = ~w;
        }
        if (__syncthreads_or(missing) == 0) return true;
        if (spin >= kMaxSpins) return false;
        __builtin_amdgcn_s_sleep(2);
    }
}

// Waits until the n words at p are published and copies them, decoded, to
// dst (LDS).  Called by every thread; returns false after kMaxSpins polls.
__device__ __forceinline__ bool wait_words(unsigned long long* p, int n, double* dst) {
    for (int spin = 0;; ++spin) {
        int missing = 0;
        for (int i = threadIdx.x; i < n; i += kThreads) {
            const unsigned long long w = __hip_atomic_load(p + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (w == 0ull)
                missing = 1;
            else
                dst[i] = decode_word(w);
        }
        if (__syncthreads_or(missing) == 0) return true;
        if (spin >= kMaxSpins) return false;
        __builtin_amdgcn_s_sleep(2);
    }
}

// ---------------------------------------------------------------------------
// the final-distribution pass: tile k2 of the selected row(s) covers elements
// [k2 * chunk2, min(V, (k2 + 1) * chunk2)); wave w of the tile covers the
// contiguous sub-chunk of vectors [w * q, (w + 1) * q), q = ceil(chunk2 / E / kWaves).
// Each sub-chunk mass is published; the draw scans one sub-chunk (q <= kThreads).
// ---------------------------------------------------------------------------
struct Span {
    int begin;  // first element, relative to the row
    int n;      // number of elements (may be 0)
};

__device__ __forceinline__ Span sub_chunk(int k2, int w, int chunk2, int V, int E) {
    const int q = (chunk2 / E + kWaves - 1) / kWaves;
    const int tb = k2 * chunk2;
    const int tn = min(V, tb + chunk2) - tb;
    const int b0 = min(tn, w * q * E);
    const int b1 = min(tn, (w + 1) * q * E);
    return Span{tb + b0, b1 - b0};
}

// Sum of the weights over one sub-chunk by one wave (rp/rq at the sub-chunk
// start, n elements); optionally stores every weight.  Valid in every lane.
// Lanes take vectors lane, lane + 64, ...; kPassUnroll 16-byte loads per row
// are in flight per lane, kept raw and unpacked one vector at a time.
template <class D, int KIND, class W>
__device__ __forceinline__ double wave_weight_sum_k(const typename D::T* rp, const typename D::T* rq, int n,
                                                    const W& w, float* wout) {
    constexpr int E = D::E;
    constexpr bool two_rows = (KIND == kResidual);
    const int lane = threadIdx.x % kWave;
    const int nvec = (n + E - 1) / E;
    const int nfull = n / E;
    const bool fast = pair_aligned<D>(rp, rq, two_rows) && nfull > 0;
    double acc = 0.0;
    for (int v0 = 0; v0 < nvec; v0 += kPassUnroll * kWave) {
        u32x4 ra[kPassUnroll], rb[kPassUnroll];
        if (fast) {
#pragma unroll
            for (int u = 0; u < kPassUnroll; ++u) {
                ra[u] = load_vec_or_pad<D, false>(rp, v0 + u * kWave + lane, nfull);
                if (two_rows) rb[u] = load_vec_or_pad<D, false>(rq, v0 + u * kWave + lane, nfull);
            }
        }
#pragma unroll
        for (int u = 0; u < kPassUnroll; ++u) {
            const int v = v0 + u * kWave + lane;
            if (v >= nvec) continue;
            float zp[E], zq[E];
            if (fast && v < nfull) {
                unpack<D>(ra[u], zp);
                if (two_rows) unpack<D>(rb[u], zq);
            } else {
                load_elems_or_pad<D>(rp, v * E, n, zp);
                if (two_rows) load_elems_or_pad<D>(rq, v * E, n, zq);
            }
#pragma unroll
            for (int e = 0; e < E; ++e) {
                const float a = w.template eval<KIND>(zp[e], two_rows ? zq[e] : -INFINITY);
                if (wout != nullptr && v * E + e < n) wout[v * E + e] = a;
                acc += (double)a;
            }
        }
    }
    return wave_sum(acc);
}

template <class D, class W>
__device__ double wave_weight_sum(const typename D::T* rp, const typename D::T* rq, int n, const W& w,
                                  float* wout) {
    return (w.kind == kTargetRow) ? wave_weight_sum_k<D, kTargetRow>(rp, rq, n, w, wout)
                                  : wave_weight_sum_k<D, kResidual>(rp, rq, n, w, wout);
}

// Lowest thread index whose predicate holds, or kThreads.  Valid in every thread.
__device__ __forceinline__ int block_first(bool pred, int* iscratch /* [kWaves] */) {
    const int wave = threadIdx.x / kWave;
    const int lane = threadIdx.x % kWave;
    const unsigned long long m = __ballot(pred);
    __syncthreads();
    if (lane == 0) iscratch[wave] = m ? wave * kWave + (__ffsll((long long)m) - 1) : kThreads;
    __syncthreads();
    int f = kThreads;
#pragma unroll
    for (int i = 0; i < kWaves; ++i) f = min(f, iscratch[i]);
    return f;
}

// Index (relative to the sub-chunk start) of the first element whose running
// weight sum exceeds t, or of the last positive weight if rounding leaves the
// sub-chunk total at or below t.  Thread i holds vector i (n <= kThreads * E),
// so one workgroup scan follows element order.  Valid in every thread.
template <class D, int KIND, class W>
__device__ __forceinline__ int sub_chunk_find_k(const typename D::T* rp, const typename D::T* rq, int n,
                                                const W& w, double t, double* scratch, double* incl_s,
                                                int* iscratch, int* result) {
    constexpr int E = D::E;
    constexpr bool two_rows = (KIND == kResidual);
    const int tid = threadIdx.x;
    const bool fast = pair_aligned<D>(rp, rq, two_rows);
    float zp[1][E], zq[1][E];
    load_pair_u<D, 1>(rp, rq, two_rows, fast, tid, 1, n, zp, zq);
    float a[E];
    double sum = 0.0;
#pragma unroll
    for (int e = 0; e < E; ++e) {
        a[e] = w.template eval<KIND>(zp[0][e], zq[0][e]);
        sum += (double)a[e];
    }
    if (tid == 0) *result = -1;
    double tot;
    const double incl = block_inclusive_scan(sum, scratch, &tot);
    incl_s[tid] = incl;
    const int first = block_first(incl > t, iscratch);
    if (first < kThreads) {
        if (tid == first) {
            double cum = (first == 0) ? 0.0 : incl_s[first - 1];
            int idx = -1, lastp = -1;
#pragma unroll
            for (int e = 0; e < E; ++e) {
                if (a[e] > 0.0f) lastp = e;
                cum += (double)a[e];
                if (idx < 0 && cum > t && a[e] > 0.0f) idx = e;
            }
            if (idx < 0) idx = lastp;
            *result = (idx >= 0) ? tid * E + idx : -1;
        }
    } else {
        // t lies at or beyond the sub-chunk total (rounding only): the last positive weight
        int lastp = -1;
#pragma unroll
        for (int e = 0; e < E; ++e)
            if (a[e] > 0.0f) lastp = tid * E + e;
        const int lv = wave_max_int(lastp);
        if ((tid % kWave) == 0) iscratch[tid / kWave] = lv;
        __syncthreads();
        if (tid == 0) {
            int best = -1;
            for (int i = 0; i < kWaves; ++i) best = max(best, iscratch[i]);
            *result = best;
        }
    }
    __syncthreads();
    return *result;
}

template <class D, class W>
__device__ int sub_chunk_find(const typename D::T* rp, const typename D::T* rq, int n, const W& w, double t,
                              double* scratch, double* incl_s, int* iscratch, int* result) {
    return (w.kind == kTargetRow) ? sub_chunk_find_k<D, kTargetRow>(rp, rq, n, w, t, scratch, incl_s, iscratch, result)
                                  : sub_chunk_find_k<D, kResidual>(rp, rq, n, w, t, scratch, incl_s, iscratch, result);
}

// ---------------------------------------------------------------------------
// the fused step: one launch; a workgroup's role follows from its index
//   stats (b, r, k)  exact mode: chunk k of row r of batch element b -> the
//                    chunk's log-normaliser (eq. (4)), published
//   decider (b)      b's decision -- eq. (1) at the drafted tokens and the
//                    first-rejection scan -- published as a small record
//   mass (b, k2)     the masses of the final distribution (eqs. (2)-(3) or
//                    the bonus row) over tile k2, one per wave, published
//   draw (b)         the inverse-CDF draw of b's next token; clears b's
//                    published words for the next call
// Index order runs over blocks j = 0, 1, ...; block j holds the stats tiles
// of b = j, the decider of b = j - lag[0], the mass tiles of b = j - lag[1]
// and the draw of b = j - lag[2], so each role of b comes after the roles it
// reads and the lags let the stream of later batch elements cover the
// latency of earlier ones.  A workgroup only waits on results of workgroups
// with smaller indices, and never on a returning atomic: the streaming
// workgroups publish and retire.  Each XCD dispatches its workgroups in index
// order, so the waiting workgroup with the smallest index always waits on
// workgroups that are running and do not wait, or that its XCD will dispatch
// once its running, non-waiting workgroups finish: no wait can block forever.
// Every wait is also bounded (kMaxSpins), so every wave exits regardless.
// ---------------------------------------------------------------------------
struct StepParams {
    const void* draft;
    const void* target;
    const int32_t* tokens;
    const float* uniforms;
    int B, gamma, V;
    int chunk1, nchunk1;           // exact: row chunks
    int chunk2, nchunk2;           // final-distribution tiles per batch element
    int n_stats, n_mass, n_total;  // workgroups by role
    int lag[3];                    // block lags of the decider, mass and draw roles
    float c;                       // exact: log2(e) / T
    float s, s0;                   // sigmoid: u = fma(z, s, s0)
    double temperature, alpha, beta;
    unsigned int* error;           // set to 1 if a wait ever timed out
    unsigned long long* dslot;     // [B, kDecisionWords] the published decision (exact mode)
    unsigned long long* pslot;     // [B, 2 gamma + 1, nchunk1] chunk log2-normalisers
    unsigned long long* mslot;     // [B, nchunk2, kWaves] sub-chunk masses
    int32_t* accepted_len;
    int32_t* next_token;
    double* tau_out;               // optional probes
    float* weight_out;
    double* mass_out;
    double* lognorm_out;
};

struct Smem {
    double words[kMergeCap];   // exact: b's chunk log2-normalisers
    double rowL[kMaxRows];     // exact: b's row log2-normalisers
    double tau[kMaxGamma];
    int stop[kMaxGamma];
    double sub[kMaxSub];       // draw: b's sub-chunk masses
    double incl[kThreads];
    double scratch[kWaves];
    int iscratch[kWaves];
    float sk[kWaves];
    double ss[kWaves];
    unsigned long long rec[kDecisionWords];
    int L, bad, tok_bad, timed_out, result, cross, last;
    double cross_t;
};

__device__ __forceinline__ double min1(double r) { return (r >= 1.0) ? 1.0 : r; }  // keeps NaN

__device__ __forceinline__ void split3(double v, float& hi, float& mid, float& lo) {
    hi = (float)v;
    mid = (float)(v - (double)hi);
    lo = (float)((v - (double)hi) - (double)mid);
}

// Exact mode, one chunk of one row: sum_x 2^(z c - k) in one streaming pass,
// published as the chunk's log2-normaliser k + log2(s).
template <class D>
__device__ __forceinline__ void stats_role(const StepParams& P, int tile, Smem& sm) {
    using T = typename D::T;
    constexpr int E = D::E;
    const int gamma = P.gamma, V = P.V, R = 2 * gamma + 1, nchunk = P.nchunk1, chunk = P.chunk1;
    const float c = P.c;
    const int k = tile % nchunk;
    const int rowid = tile / nchunk;  // b * R + r
    const int b = rowid / R;
    const int r = rowid - b * R;
    const T* row = (r <= gamma) ? static_cast<const T*>(P.target) + ((size_t)b * (gamma + 1) + r) * (size_t)V
                                : static_cast<const T*>(P.draft) + ((size_t)b * gamma + (r - gamma - 1)) * (size_t)V;
    const int begin = k * chunk;
    const int n = min(V, begin + chunk) - begin;
    const T* base = row + begin;
    const int nfull = n / E;            // whole 16-byte vectors
    const int nvec = (n + E - 1) / E;   // plus a partial one at the end of a row
    const bool aligned = (reinterpret_cast<uintptr_t>(base) & 15u) == 0;

    // Thread t takes whole vectors t, t + kThreads, ... in blocks of kUnroll;
    // all loads of a block are issued before any is used, and the block shares
    // one update of the running reference.  A partial vector at the end of a
    // row is absorbed after the loop by the thread that would own it.  The
    // assignment and order depend only on element indices, never on the
    // row's address, so equal rows give bit-identical normalisers.
    Lse st{-INFINITY, 0.0};
    if (nfull > 0) {
        for (int v0 = 0; v0 < nfull; v0 += kUnroll * kThreads) {
            float x[kUnroll][E];
            if (aligned) {
                u32x4 raw[kUnroll];
#pragma unroll
                for (int u = 0; u < kUnroll; ++u)
                    raw[u] = load_vec_or_pad<D, true>(base, v0 + u * kThreads + (int)threadIdx.x, nfull);
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) unpack<D>(raw[u], x[u]);
            } else {
                // rows that are not 16-byte aligned (e.g. odd V in fp32)
#pragma unroll
                for (int u = 0; u < kUnroll; ++u)
                    load_elems_or_pad<D>(base, (v0 + u * kThreads + (int)threadIdx.x) * E, nfull * E, x[u]);
            }
            lse_absorb_block<kUnroll, E>(st, x, c);
        }
    }
    if (nvec > nfull && (int)threadIdx.x == nfull % kThreads) {
        float x[1][E];
        load_elems_or_pad<D>(base, nfull * E, n, x[0]);
        lse_absorb_block<1, E>(st, x, c);
    }
    const Lse blk = block_lse(st, sm.sk, sm.ss);
    if (threadIdx.x == 0) publish(P.pslot + tile, (double)blk.k + log2(blk.s));
}

struct Decision {
    int L;        // accepted length, in [0, gamma]
    bool bad;     // sentinel
    bool ok;      // false if a wait timed out
    ExactWeights ew;
    SigmoidWeights sw;
};

// The decision for batch element b: eq. (1) at the drafted tokens and the
// first-rejection scan, plus the weights of the final distribution.  Every
// workgroup that needs it computes it the same way, so they all agree.
template <class D, bool kExact>
__device__ __forceinline__ Decision decide(const StepParams& P, int b, Smem& sm) {
    using T = typename D::T;
    const int gamma = P.gamma, V = P.V, R = 2 * gamma + 1;
    const int tid = threadIdx.x;
    const T* draft = static_cast<const T*>(P.draft) + (size_t)b * gamma * V;
    const T* target = static_cast<const T*>(P.target) + (size_t)b * (gamma + 1) * V;

    // independent loads first: tokens, uniforms and the drafted-token logits
    int x = 0;
    double r = 0.0;
    bool tok_ok = true;
    float zp = 0.0f, zq = 0.0f;
    if (tid == 0) sm.tok_bad = 0;
    if (tid < gamma) {
        x = P.tokens[(size_t)b * gamma + tid];
        r = (double)P.uniforms[(size_t)b * (gamma + 1) + tid];
        tok_ok = (x >= 0 && x < V);
        const int xs = tok_ok ? x : 0;
        zp = to_f32(target[(size_t)tid * V + xs]);
        zq = to_f32(draft[(size_t)tid * V + xs]);
    }

    Decision d{};
    d.ok = true;
    if (kExact) {
        // b's chunk log2-normalisers, then each row's, merged in chunk order
        const int nc1 = P.nchunk1;
        d.ok = wait_words(P.pslot + (size_t)b * R * nc1, R * nc1, sm.words);
        for (int i = tid; i < R; i += kThreads) {
            double m = -INFINITY;
            bool nan = false;
            for (int k = 0; k < nc1; ++k) {
                const double l = sm.words[i * nc1 + k];
                nan |= (l != l);
                m = fmax(m, l);
            }
            double sum = 0.0;
            if (!nan && m != -INFINITY)
                for (int k = 0; k < nc1; ++k) sum += exp2(sm.words[i * nc1 + k] - m);
            sm.rowL[i] = nan ? __builtin_nan("") : ((m == -INFINITY) ? -INFINITY : m + log2(sum));
        }
    }
    __syncthreads();

    if (tid < gamma) {
        if (!tok_ok) sm.tok_bad = 1;
        double tau;
        bool row_ok;
        if (kExact) {
            const double lam_p = sm.rowL[tid];
            const double lam_q = sm.rowL[gamma + 1 + tid];
            row_ok = isfinite(lam_p) && isfinite(lam_q);
            if (zq == -INFINITY) {
                tau = 1.0;  // q(x) = 0
            } else {
                const double l2 = ((double)zp - (double)zq) * (double)P.c - (lam_p - lam_q);
                tau = min1(exp2(l2));
            }
        } else {
            const double span = P.beta - P.alpha;
            const double up = ((double)zp / P.temperature - P.alpha) / span;
            const double uq = ((double)zq / P.temperature - P.alpha) / span;
            const double ph = 1.0 / (1.0 + exp(-up));
            const double qh = 1.0 / (1.0 + exp(-uq));
            tau = (qh > 0.0) ? min1(ph / qh) : 1.0;
            row_ok = isfinite(tau);
        }
        sm.tau[tid] = tau;
        sm.stop[tid] = !row_ok ? 2 : ((r <= tau) ? 0 : 1);
    }
    __syncthreads();
    if (tid == 0) {
        int L = gamma, bad = sm.tok_bad;
        for (int c = 0; c < gamma; ++c) {
            if (sm.stop[c] != 0) {
                L = c;
                if (sm.stop[c] == 2) bad = 1;
                break;
            }
        }
        if (kExact && !bad && L == gamma && !isfinite(sm.rowL[gamma])) bad = 1;
        sm.L = L;
        sm.bad = bad;
    }
    __syncthreads();
    d.L = sm.L;
    d.bad = sm.bad != 0 || !d.ok;
    const bool two_rows = d.L < gamma;
    if (kExact && !d.bad) {
        const double lp = sm.rowL[min(d.L, gamma)];
        const double lq = sm.rowL[gamma + 1 + min(d.L, gamma - 1)];
        d.ew.kind = two_rows ? kResidual : kTargetRow;
        d.ew.c = P.c;
        split3(lp, d.ew.kp, d.ew.lp_hi, d.ew.lp_lo);
        split3(lq, d.ew.kq, d.ew.lq_hi, d.ew.lq_lo);
        float dummy;
        split3(lp - lq, d.ew.d_hi, d.ew.d_lo, dummy);
    }
    if (!kExact) {
        d.sw.kind = two_rows ? kResidual : kTargetRow;
        d.sw.s = P.s;
        d.sw.s0 = P.s0;
    }
    return d;
}

// b's decision, made once by b's decider workgroup and published as a small
// record for b's mass and draw workgroups; it also writes the tau / normaliser
// probes.
template <class D, bool kExact>
__device__ __forceinline__ void decider_role(const StepParams& P, int b, Smem& sm) {
    const int gamma = P.gamma, R = 2 * gamma + 1;
    const int tid = threadIdx.x;
    const Decision d = decide<D, kExact>(P, b, sm);
    if (!d.ok && tid == 0) __hip_atomic_store(P.error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (P.tau_out != nullptr && tid < gamma) P.tau_out[(size_t)b * gamma + tid] = sm.tau[tid];
    if (kExact && P.lognorm_out != nullptr)
        for (int i = tid; i < R; i += kThreads)
            P.lognorm_out[(size_t)b * R + i] = sm.rowL[i] * 0.693147180559945309417;
    if (tid == 0) {
        unsigned long long* rec = P.dslot + (size_t)b * kDecisionWords;
        publish_raw(rec + 1, pack2(d.ew.kp, d.ew.lp_hi));
        publish_raw(rec + 2, pack2(d.ew.lp_lo, d.ew.kq));
        publish_raw(rec + 3, pack2(d.ew.lq_hi, d.ew.lq_lo));
        publish_raw(rec + 4, pack2(d.ew.d_hi, d.ew.d_lo));
        publish_raw(rec + 0, (unsigned long long)(d.L & 0xffff) | ((unsigned long long)(d.bad ? 1 : 0) << 16) |
                                 (1ull << 32));
    }
}

// b's published decision (in b's mass and draw workgroups).
__device__ __forceinline__ Decision read_decision(const StepParams& P, int b, bool exact, Smem& sm) {
    Decision d{};
    d.ok = wait_raw(P.dslot + (size_t)b * kDecisionWords, kDecisionWords, sm.rec);
    const unsigned long long w0 = sm.rec[0];
    d.L = d.ok ? (int)(w0 & 0xffff) : 0;
    d.bad = ((w0 >> 16) & 1) != 0 || !d.ok;
    const int kind = (d.L < P.gamma) ? kResidual : kTargetRow;
    if (exact) {
        d.ew.kind = kind;
        d.ew.c = P.c;
        d.ew.kp = unpack_hi(sm.rec[1]);
        d.ew.lp_hi = unpack_lo(sm.rec[1]);
        d.ew.lp_lo = unpack_hi(sm.rec[2]);
        d.ew.kq = unpack_lo(sm.rec[2]);
        d.ew.lq_hi = unpack_hi(sm.rec[3]);
        d.ew.lq_lo = unpack_lo(sm.rec[3]);
        d.ew.d_hi = unpack_hi(sm.rec[4]);
        d.ew.d_lo = unpack_lo(sm.rec[4]);
    } else {
        d.sw.kind = kind;
        d.sw.s = P.s;
        d.sw.s0 = P.s0;
    }
    return d;
}

template <class D, bool kExact>
__device__ __forceinline__ void mass_role(const StepParams& P, int b, int k2, Smem& sm) {
    using T = typename D::T;
    constexpr int E = D::E;
    const int gamma = P.gamma, V = P.V;
    const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
    const Decision d = read_decision(P, b, kExact, sm);
    if (!d.ok && tid == 0) __hip_atomic_store(P.error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const Span sp = sub_chunk(k2, wave, P.chunk2, V, E);
    double m = 0.0;
    if (!d.ok) {
        m = __builtin_nan("");
    } else if (!d.bad && sp.n > 0) {
        const T* rp = static_cast<const T*>(P.target) + ((size_t)b * (gamma + 1) + min(d.L, gamma)) * V + sp.begin;
        const T* rq = static_cast<const T*>(P.draft) + ((size_t)b * gamma + min(d.L, gamma - 1)) * V + sp.begin;
        float* wout = (P.weight_out != nullptr) ? P.weight_out + (size_t)b * V + sp.begin : nullptr;
        m = kExact ? wave_weight_sum<D>(rp, rq, sp.n, d.ew, wout) : wave_weight_sum<D>(rp, rq, sp.n, d.sw, wout);
    }
    if (lane == 0) publish(P.mslot + ((size_t)b * P.nchunk2 + k2) * kWaves + wave, m);
}

// The inverse-CDF draw for b, by b's draw workgroup, once b's mass tiles have
// published.
template <class D, bool kExact>
__device__ __forceinline__ void draw_role(const StepParams& P, int b, Smem& sm) {
    using T = typename D::T;
    constexpr int E = D::E;
    const int gamma = P.gamma, V = P.V, R = 2 * gamma + 1;
    const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
    const int M = P.nchunk2 * kWaves;
    Decision d = read_decision(P, b, kExact, sm);
    unsigned long long* ms = P.mslot + (size_t)b * M;
    const bool got = d.ok && wait_words(ms, M, sm.sub);
    if (!got && tid == 0) __hip_atomic_store(P.error, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const double u = (double)P.uniforms[(size_t)b * (gamma + 1) + gamma];
    const T* rp = static_cast<const T*>(P.target) + ((size_t)b * (gamma + 1) + min(d.L, gamma)) * V;
    const T* rq = static_cast<const T*>(P.draft) + ((size_t)b * gamma + min(d.L, gamma - 1)) * V;
    float* wrow = (P.weight_out != nullptr) ? P.weight_out + (size_t)b * V : nullptr;
    const int L = d.L;
    bool bad = d.bad || !got;
    int idx = -1;
    double total = __builtin_nan("");
    for (int pass = 0; pass < 2 && !bad; ++pass) {
        // fixed-order prefix over the sub-chunk masses: 4 consecutive per thread
        double loc[4];
        double ls = 0.0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int j = tid * 4 + i;
            loc[i] = (j < M) ? sm.sub[j] : 0.0;
            ls += loc[i];
        }
        double tot;
        const double incl = block_inclusive_scan(ls, sm.scratch, &tot);
        sm.incl[tid] = incl;
        total = tot;
        if (!(isfinite(total) && total >= 0.0)) {
            bad = true;
            break;
        }
        if (total == 0.0) {
            if (pass == 0 && L < gamma) {
                // no residual mass (possible in sigmoid mode): draw from target row L
                d.ew.kind = kTargetRow;
                d.sw.kind = kTargetRow;
                __syncthreads();
                for (int k2 = 0; k2 < P.nchunk2; ++k2) {
                    const Span sp = sub_chunk(k2, wave, P.chunk2, V, E);
                    double m = 0.0;
                    if (sp.n > 0)
                        m = kExact ? wave_weight_sum<D>(rp + sp.begin, rq + sp.begin, sp.n, d.ew, wrow ? wrow + sp.begin : nullptr)
                                   : wave_weight_sum<D>(rp + sp.begin, rq + sp.begin, sp.n, d.sw, wrow ? wrow + sp.begin : nullptr);
                    if (lane == 0) sm.sub[k2 * kWaves + wave] = m;
                }
                __syncthreads();
                continue;
            }
            bad = true;
            break;
        }
        const double t = u * total;
        const int first = block_first(incl > t, sm.iscratch);
        if (tid == 0) {
            sm.cross = -1;
            sm.cross_t = 0.0;
        }
        __syncthreads();
        if (first < kThreads && tid == first) {
            double cum = (first == 0) ? 0.0 : sm.incl[first - 1];
            int j = -1;
            double before = cum;
            int lastp = -1;
            double lastp_before = 0.0;
            for (int i = 0; i < 4; ++i) {
                if (loc[i] > 0.0) {
                    lastp = tid * 4 + i;
                    lastp_before = cum;
                }
                if (j < 0 && cum + loc[i] > t && loc[i] > 0.0) {
                    j = tid * 4 + i;
                    before = cum;
                }
                cum += loc[i];
            }
            if (j < 0) {
                j = lastp;
                before = lastp_before;
            }
            sm.cross = j;
            sm.cross_t = t - before;
        }
        if (first >= kThreads && tid == 0) {
            // rounding only: the last positive weight of the last sub-chunk with mass
            for (int j = M - 1; j >= 0; --j)
                if (sm.sub[j] > 0.0) {
                    sm.cross = j;
                    sm.cross_t = sm.sub[j];
                    break;
                }
        }
        __syncthreads();
        const int j = sm.cross;
        if (j < 0) {
            bad = true;
            break;
        }
        const Span sp = sub_chunk(j / kWaves, j % kWaves, P.chunk2, V, E);
        const int local = kExact ? sub_chunk_find<D>(rp + sp.begin, rq + sp.begin, sp.n, d.ew, sm.cross_t, sm.scratch, sm.incl, sm.iscratch, &sm.result)
                                 : sub_chunk_find<D>(rp + sp.begin, rq + sp.begin, sp.n, d.sw, sm.cross_t, sm.scratch, sm.incl, sm.iscratch, &sm.result);
        idx = (local >= 0) ? sp.begin + local : -1;
        if (idx < 0) bad = true;
        break;
    }
    if (tid == 0) {
        P.accepted_len[b] = bad ? -1 : L;
        P.next_token[b] = bad ? -1 : idx;
        if (P.mass_out != nullptr) P.mass_out[b] = bad ? __builtin_nan("") : total;
    }
    // every workgroup of b is done with b's published words: clear them for the next call
    __syncthreads();
    if (kExact)
        for (int i = tid; i < R * P.nchunk1; i += kThreads) clear_word(P.pslot + (size_t)b * R * P.nchunk1 + i);
    if (tid < kDecisionWords) clear_word(P.dslot + (size_t)b * kDecisionWords + tid);
    for (int i = tid; i < M; i += kThreads) clear_word(ms + i);
}

// Workgroups before block j (see the layout comment of StepParams).
__device__ __forceinline__ long long block_offset(long long j, long long B, long long S, long long Mt, const int* lag) {
    auto clampb = [&](long long x) { return x < 0 ? 0 : (x > B ? B : x); };
    return S * clampb(j) + clampb(j - lag[0]) + Mt * clampb(j - lag[1]) + clampb(j - lag[2]);
}

template <class D, bool kExact>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4))) void verify_kernel(StepParams P) {
    __shared__ Smem sm;
    const long long id = blockIdx.x;
    const long long B = P.B;
    const long long S = kExact ? (long long)(2 * P.gamma + 1) * P.nchunk1 : 0;  // stats tiles per element
    const long long Mt = P.nchunk2;                                            // mass tiles per element
    // block j holds, in this order: the stats tiles of b = j, the decider of
    // b = j - lag[0], the mass tiles of b = j - lag[1], the draw of b = j - lag[2]
    long long lo = 0, hi = B + P.lag[2];  // the block containing id: offset(j) <= id < offset(j + 1)
    while (hi - lo > 1) {
        const long long mid = (lo + hi) / 2;
        if (block_offset(mid, B, S, Mt, P.lag) <= id) lo = mid; else hi = mid;
    }
    const long long j = lo;
    long long r = id - block_offset(j, B, S, Mt, P.lag);
    if (j < B) {
        if (r < S) {
            stats_role<D>(P, (int)(j * S + r), sm);
            return;
        }
        r -= S;
    }
    const long long bd = j - P.lag[0];
    if (bd >= 0 && bd < B) {
        if (r == 0) {
            decider_role<D, kExact>(P, (int)bd, sm);
            return;
        }
        r -= 1;
    }
    const long long bm = j - P.lag[1];
    if (bm >= 0 && bm < B) {
        if (r < Mt) {
            mass_role<D, kExact>(P, (int)bm, (int)r, sm);
            return;
        }
        r -= Mt;
    }
    draw_role<D, kExact>(P, (int)(j - P.lag[2]), sm);
}

__global__ void fill_zero_kernel(uint32_t* p, size_t n) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        p[i] = 0u;
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
struct Plan {
    int E;
    int chunk1, nchunk1;
    int chunk2, nchunk2;
    long long n_stats, n_mass, n_total;
    size_t off_dslot, off_pslot, off_mslot, bytes;
};

static inline long long ceil_div(long long a, long long b) { return (a + b - 1) / b; }
static inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

static bool valid_dtype(sv_dtype_t dt) { return dt == SV_F32 || dt == SV_F16 || dt == SV_BF16; }

// Work decomposition; the workspace size depends only on (B, gamma, V, dtype).
static bool make_plan(int32_t B, int32_t gamma, int32_t V, sv_dtype_t dt, Plan* p) {
    if (B < 1 || gamma < 1 || gamma > kMaxGamma || V < 1 || !valid_dtype(dt)) return false;
    const int E = (dt == SV_F32) ? 4 : 8;
    const int s = (dt == SV_F32) ? 4 : 2;
    const long long R = 2LL * gamma + 1;
    if ((long long)B * (gamma + 1) * (long long)V > (1LL << 40)) return false;
    const long long min_elems = (long long)kThreads * E;
    const long long max_cells = std::max<long long>(1, ceil_div(V, min_elems));

    // row chunks: enough workgroups to fill the GPU, at most 64 KiB each
    long long nc = ceil_div(kWantStatsTiles, B * R);
    nc = std::max(nc, ceil_div(V, kStatsTileBytes / s));
    nc = std::min(nc, max_cells);
    nc = std::min(nc, std::max<long long>(1, kMergeCap / R));
    const long long chunk = ceil_div(ceil_div(V, nc), E) * E;
    p->chunk1 = (int)chunk;
    p->nchunk1 = (int)ceil_div(V, chunk);
    if (R * p->nchunk1 > kMergeCap) return false;

    // final-distribution tiles: a sub-chunk (a quarter tile) must fit one
    // vector per thread, and b's sub-chunk masses must fit kMaxSub
    const long long max_tile_vecs = (long long)kWaves * kThreads;
    long long nc2 = ceil_div(kWantSampleTiles, B);
    nc2 = std::max(nc2, ceil_div(V, kSampleTileBytes / s));
    nc2 = std::min(nc2, max_cells);
    nc2 = std::max(nc2, ceil_div(V, max_tile_vecs * E));
    const long long chunk2 = ceil_div(ceil_div(V, nc2), E) * E;
    p->chunk2 = (int)chunk2;
    p->nchunk2 = (int)ceil_div(V, chunk2);
    if ((long long)p->nchunk2 * kWaves > kMaxSub || chunk2 / E > max_tile_vecs) return false;
    p->E = E;

    p->n_stats = (long long)B * R * p->nchunk1;
    p->n_mass = (long long)B * p->nchunk2;
    p->n_total = p->n_stats + p->n_mass + 2LL * B;  // plus a decider and a draw per batch element
    if (p->n_total > 0x7fffffffLL) return false;

    size_t off = 256;  // header: the error flag at byte offset 4
    p->off_dslot = off;
    off = align256(off + sizeof(unsigned long long) * (size_t)B * kDecisionWords);
    p->off_pslot = off;
    off = align256(off + sizeof(unsigned long long) * (size_t)p->n_stats);
    p->off_mslot = off;
    off = align256(off + sizeof(unsigned long long) * (size_t)p->n_mass * kWaves);
    p->bytes = off;
    return true;
}

// Block lags (in batch elements) of the decider, mass and draw roles.  The
// decider of b follows b's stats tiles at once; mass and draw workgroups come
// after the whole stream: interleaving them into it was measured to cost more
// (their latency-bound lifetimes hold dispatch slots the stream needs) than
// the overlap gains.
static void set_lags(long long B, int* lag) {
    lag[0] = 1;
    lag[1] = (int)B;
    lag[2] = (int)B + 1;
}

struct Call {
    const void* draft;
    const void* target;
    sv_dtype_t dt;
    const int32_t* tokens;
    const float* uniforms;
    int32_t B, gamma, V;
    float temperature, alpha, beta;
    int32_t* accepted_len;
    int32_t* next_token;
    void* ws;
    size_t ws_bytes;
    hipStream_t stream;
    double* tau_out;
    float* weight_out;
    double* mass_out;
    double* lognorm_out;
};

template <class D>
static sv_status_t launch(const Call& a, bool exact, const Plan& pl) {
    char* ws = static_cast<char*>(a.ws);
    StepParams P{};
    P.draft = a.draft;
    P.target = a.target;
    P.tokens = a.tokens;
    P.uniforms = a.uniforms;
    P.B = a.B;
    P.gamma = a.gamma;
    P.V = a.V;
    P.chunk1 = pl.chunk1;
    P.nchunk1 = pl.nchunk1;
    P.chunk2 = pl.chunk2;
    P.nchunk2 = pl.nchunk2;
    P.n_stats = exact ? (int)pl.n_stats : 0;
    P.n_mass = (int)pl.n_mass;
    P.n_total = P.n_stats + P.n_mass + 2 * a.B;
    set_lags(a.B, P.lag);
    P.temperature = (double)a.temperature;
    P.alpha = (double)a.alpha;
    P.beta = (double)a.beta;
    P.c = (float)(1.4426950408889634074 / (double)a.temperature);
    P.s = (float)(1.0 / ((double)a.temperature * ((double)a.beta - (double)a.alpha)));
    P.s0 = (float)(-(double)a.alpha / ((double)a.beta - (double)a.alpha));
    P.error = reinterpret_cast<unsigned int*>(ws) + 1;
    P.dslot = reinterpret_cast<unsigned long long*>(ws + pl.off_dslot);
    P.pslot = reinterpret_cast<unsigned long long*>(ws + pl.off_pslot);
    P.mslot = reinterpret_cast<unsigned long long*>(ws + pl.off_mslot);
    P.accepted_len = a.accepted_len;
    P.next_token = a.next_token;
    P.tau_out = a.tau_out;
    P.weight_out = a.weight_out;
    P.mass_out = a.mass_out;
    P.lognorm_out = a.lognorm_out;
    if (exact)
        hipLaunchKernelGGL((verify_kernel<D, true>), dim3(P.n_total), dim3(kThreads), 0, a.stream, P);
    else
        hipLaunchKernelGGL((verify_kernel<D, false>), dim3(P.n_total), dim3(kThreads), 0, a.stream, P);
    return hipGetLastError() == hipSuccess ? SV_OK : SV_ERR_HIP;
}

static sv_status_t run(const Call& a, bool exact) {
    if (a.draft == nullptr || a.target == nullptr || a.tokens == nullptr || a.uniforms == nullptr ||
        a.accepted_len == nullptr || a.next_token == nullptr || a.ws == nullptr)
        return SV_ERR_NULL;
    if (!valid_dtype(a.dt)) return SV_ERR_DTYPE;
    Plan pl;
    if (!make_plan(a.B, a.gamma, a.V, a.dt, &pl)) return SV_ERR_SHAPE;
    if (!(std::isfinite(a.temperature) && a.temperature > 0.0f)) return SV_ERR_PARAM;
    const double c = 1.4426950408889634074 / (double)a.temperature;
    if (!(std::isfinite((float)c) && (float)c > 0.0f)) return SV_ERR_PARAM;
    if (!exact) {
        if (!(std::isfinite(a.alpha) && std::isfinite(a.beta) && a.alpha < a.beta)) return SV_ERR_PARAM;
        const double s = 1.0 / ((double)a.temperature * ((double)a.beta - (double)a.alpha));
        if (!(std::isfinite((float)s) && (float)s > 0.0f)) return SV_ERR_PARAM;
    }
    if (a.ws_bytes < pl.bytes || (reinterpret_cast<uintptr_t>(a.ws) & 15u) != 0) return SV_ERR_WORKSPACE;
    switch (a.dt) {
        case SV_F32: return launch<F32>(a, exact, pl);
        case SV_F16: return launch<F16>(a, exact, pl);
        case SV_BF16: return launch<BF16>(a, exact, pl);
    }
    return SV_ERR_DTYPE;
}

}  // namespace sv

// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------
extern "C" {

size_t spec_verify_workspace_bytes(int32_t batch, int32_t gamma, int32_t vocab, sv_dtype_t dtype) {
    sv::Plan pl;
    return sv::make_plan(batch, gamma, vocab, dtype, &pl) ? pl.bytes : 0;
}

sv_status_t spec_verify_workspace_init(void* workspace, size_t workspace_bytes, hipStream_t stream) {
    if (workspace == nullptr) return SV_ERR_NULL;
    if ((reinterpret_cast<uintptr_t>(workspace) & 15u) != 0 || workspace_bytes % 4 != 0) return SV_ERR_WORKSPACE;
    const size_t n = workspace_bytes / 4;
    if (n == 0) return SV_OK;
    const unsigned int blocks = (unsigned int)std::min<size_t>(1024, (n + 255) / 256);
    hipLaunchKernelGGL(sv::fill_zero_kernel, dim3(blocks), dim3(256), 0, stream, static_cast<uint32_t*>(workspace), n);
    return hipGetLastError() == hipSuccess ? SV_OK : SV_ERR_HIP;
}

sv_status_t spec_verify_exact(const void* draft_logits, const void* target_logits, sv_dtype_t dtype,
                              const int32_t* draft_tokens, const float* uniforms, int32_t batch, int32_t gamma,
                              int32_t vocab, float temperature, int32_t* accepted_len, int32_t* next_token,
                              void* workspace, size_t workspace_bytes, hipStream_t stream) {
    sv::Call a{draft_logits, target_logits, dtype, draft_tokens, uniforms, batch, gamma, vocab, temperature,
               0.0f, 0.0f, accepted_len, next_token, workspace, workspace_bytes, stream,
               nullptr, nullptr, nullptr, nullptr};
    return sv::run(a, true);
}

sv_status_t spec_verify_sigmoid(const void* draft_logits, const void* target_logits, sv_dtype_t dtype,
                                const int32_t* draft_tokens, const float* uniforms, int32_t batch, int32_t gamma,
                                int32_t vocab, float temperature, float alpha, float beta, int32_t* accepted_len,
                                int32_t* next_token, void* workspace, size_t workspace_bytes, hipStream_t stream) {
    sv::Call a{draft_logits, target_logits, dtype, draft_tokens, uniforms, batch, gamma, vocab, temperature,
               alpha, beta, accepted_len, next_token, workspace, workspace_bytes, stream,
               nullptr, nullptr, nullptr, nullptr};
    return sv::run(a, false);
}

sv_status_t spec_verify_exact_probe(const void* draft_logits, const void* target_logits, sv_dtype_t dtype,
                                    const int32_t* draft_tokens, const float* uniforms, int32_t batch, int32_t gamma,
                                    int32_t vocab, float temperature, int32_t* accepted_len, int32_t* next_token,
                                    void* workspace, size_t workspace_bytes, hipStream_t stream, double* tau_out,
                                    float* weight_out, double* mass_out, double* lognorm_out) {
    sv::Call a{draft_logits, target_logits, dtype, draft_tokens, uniforms, batch, gamma, vocab, temperature,
               0.0f, 0.0f, accepted_len, next_token, workspace, workspace_bytes, stream,
               tau_out, weight_out, mass_out, lognorm_out};
    return sv::run(a, true);
}

sv_status_t spec_verify_sigmoid_probe(const void* draft_logits, const void* target_logits, sv_dtype_t dtype,
                                      const int32_t* draft_tokens, const float* uniforms, int32_t batch,
                                      int32_t gamma, int32_t vocab, float temperature, float alpha, float beta,
                                      int32_t* accepted_len, int32_t* next_token, void* workspace,
                                      size_t workspace_bytes, hipStream_t stream, double* tau_out,
                                      float* weight_out, double* mass_out) {
    sv::Call a{draft_logits, target_logits, dtype, draft_tokens, uniforms, batch, gamma, vocab, temperature,
               alpha, beta, accepted_len, next_token, workspace, workspace_bytes, stream,
               tau_out, weight_out, mass_out, nullptr};
    return sv::run(a, false);
}

const char* spec_verify_status_string(sv_status_t status) {
    switch (status) {
        case SV_OK: return "ok";
        case SV_ERR_NULL: return "a required pointer is NULL";
        case SV_ERR_SHAPE: return "invalid sizes (batch, gamma or vocab)";
        case SV_ERR_DTYPE: return "unknown logit dtype";
        case SV_ERR_PARAM: return "invalid temperature or sigmoid scaling constants";
        case SV_ERR_WORKSPACE: return "workspace too small or misaligned";
        case SV_ERR_HIP: return "HIP launch failed";
    }
    return "unknown status";
}

}  // extern "C"
