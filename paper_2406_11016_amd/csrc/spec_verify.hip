// Fused speculative-sampling verification for gfx950 (MI355X): kernels and C ABI.
//
// Method: arXiv 2406.11016, Sec. 3.1 (eqs. (1)-(3)) and Sec. 3.2.2 (eqs. (4)-(5)).
//
// One launch per call.  Workgroups play one of five roles by index (see
// verify_kernel):
//   stats    (exact mode) one chunk of one logit row, streamed once with
//            128-bit non-temporal loads: the chunk's contribution to the row's
//            softmax normaliser (eq. (4)).  These move every logit byte and
//            bound the step.
//   decider  b: tau_c of eq. (1) at the drafted tokens and the
//            first-rejection scan for batch element b, made once (exact
//            mode; in the sigmoid mode every reader makes it itself).
//   mass     (b, tile): the weights a(x) of the final distribution (residual
//            of eqs. (2)-(3), or target row gamma) summed over the tile, one
//            sub-chunk per wave.
//   draw     b: fixed-order prefix over b's sub-chunk masses, then one
//            workgroup scan inside the sub-chunk the uniform falls in -- the
//            inverse-CDF draw of the next token.
//   bonus    b: when every draft is accepted, the draw from target row
//            gamma straight from that row's normaliser partials (exact
//            mode) or its sums of p_hat (sigmoid mode), prepared without
//            waiting for the decision.
// Sigmoid mode (eq. (5)) has no stats role: it needs no row normaliser, so
// it reads the logits at the drafted tokens, target row gamma (summed for
// the bonus draw before the decision is known) and, after a rejection, the
// two rows the residual is drawn from.
#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <cmath>
#include <mutex>

#include "spec_verify.h"
#include "sv_device.hpp"

namespace sv {

enum : int { kResidual = 0, kTargetRow = 1 };

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
// keep their relative precision.  kFlat evaluates both forms and selects
// (the same values, without a divergent branch per element: quicker where a
// workgroup's chain is the step's critical path, slower where the residual
// pass shares the GPU with the stream and most weights are 0).
struct ExactWeights {
    int kind;
    float c;
    float kp, lp_hi, lp_lo;  // target row: reference k and log2(s) as hi + lo
    float kq, lq_hi, lq_lo;  // draft row
    float d_hi, d_lo;        // Lambda_p - Lambda_q as hi + lo
    template <int KIND, bool kFlat = false>
    __device__ __forceinline__ float eval(float zp, float zq) const {
        if (KIND == kTargetRow) return exp2_hw((fmaf(zp, c, -kp) - lp_hi) - lp_lo);
        float dz, dz_lo;
        two_diff(zp, zq, dz, dz_lo);
        const float d = fmaf(dz_lo, c, fmaf(dz, c, -d_hi)) - d_lo;
        if constexpr (kFlat) {
            const float q = exp2_hw((fmaf(zq, c, -kq) - lq_hi) - lq_lo);
            const float near = q * expm1_small(d * kLn2);
            const float far = exp2_hw((fmaf(zp, c, -kp) - lp_hi) - lp_lo) - q;
            return (d > 0.0f) ? ((d <= 0.5f) ? near : far) : 0.0f;  // NaN d: 0
        }
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
    template <int KIND, bool kFlat = false>
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
    return (a & 3u) == 0;
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

// A workgroup barrier for LDS data only: it waits for the workgroup's LDS
// (and scalar) accesses but not for its global loads and stores in flight,
// which __syncthreads would.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Sleep between the two polls in flight of a wait, in s_sleep units of 64
// clocks: none (gaps of 1, 2 and 4 units, and the 10 of a first version,
// measured slower: the second poll is best issued at once).
constexpr int kPollGap = 0;

// Waits until the n words at p are published, handing each to take(i, w)
// (w the raw, still inverted word).  Called by every thread; returns false
// after `limit` polls.  Each poll issues NV loads per thread before it
// looks at any (indices clamped into range), so a poll costs one memory
// round trip for up to NV * kThreads words.  With kPipe (the launch of short
// streams, whose steps are a chain of such waits) and up to NV * kThreads
// words, two polls are in flight at once, the second issued a fraction of a
// round trip after the first, so a word is seen sooner after it lands; the
// workgroup then agrees on "all present" through LDS flags (a
// __syncthreads_or would also wait for the other poll's loads).
template <int NV, bool kPipe = false, class A, class F>
__device__ __forceinline__ bool poll_at(int n, A addr, F take, int limit) {
    if (!kPipe || n > NV * kThreads) {
        for (int spin = 0;; ++spin) {
            int missing = 0;
            for (int i0 = 0; i0 < n; i0 += NV * kThreads) {
                unsigned long long w[NV];
#pragma unroll
                for (int u = 0; u < NV; ++u) {
                    const int i = min(i0 + u * kThreads + (int)threadIdx.x, n - 1);
                    w[u] = __hip_atomic_load(addr(i), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                }
#pragma unroll
                for (int u = 0; u < NV; ++u) {
                    const int i = i0 + u * kThreads + (int)threadIdx.x;
                    if (i < n) {
                        if (w[u] == 0ull)
                            missing = 1;
                        else
                            take(i, w[u]);
                    }
                }
            }
            if (__syncthreads_or(missing) == 0) return true;
            if (spin >= limit) return false;
            __builtin_amdgcn_s_sleep(2);
        }
    }
    __shared__ int pflag[2][kWaves];  // "a word is missing", per wave, for two rounds
    const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
    unsigned long long a[NV], c[NV];
    auto issue = [&](unsigned long long (&w)[NV]) {
#pragma unroll
        for (int u = 0; u < NV; ++u)
            w[u] = __hip_atomic_load(addr(min(u * kThreads + tid, n - 1)), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    };
    auto check = [&](unsigned long long (&w)[NV], int round) {
        bool missing = false;
#pragma unroll
        for (int u = 0; u < NV; ++u) {
            const int i = u * kThreads + tid;
            if (i < n) {
                if (w[u] == 0ull)
                    missing = true;
                else
                    take(i, w[u]);
            }
        }
        const unsigned long long m = __ballot(missing);
        if (lane == 0) pflag[round & 1][wave] = (m != 0ull) ? 1 : 0;
        lds_barrier();
        int any = 0;
#pragma unroll
        for (int w2 = 0; w2 < kWaves; ++w2) any |= pflag[round & 1][w2];
        return any == 0;
    };
    issue(a);
    for (int round = 0;; round += 2) {
        if constexpr (kPollGap > 0) __builtin_amdgcn_s_sleep(kPollGap);
        issue(c);
        if (check(a, round)) return true;
        if (round + 1 >= limit) return false;
        if constexpr (kPollGap > 0) __builtin_amdgcn_s_sleep(kPollGap);
        issue(a);
        if (check(c, round + 1)) return true;
        if (round + 2 >= limit) return false;
    }
}

template <int NV, bool kPipe = false, class F>
__device__ __forceinline__ bool poll_words(unsigned long long* p, int n, F take, int limit) {
    return poll_at<NV, kPipe>(n, [&](int i) { return p + i; }, take, limit);
}

// The n (<= kThreads) raw record words at p, copied to dst.
template <bool kPipe = false>
__device__ __forceinline__ bool wait_raw(unsigned long long* p, int n, unsigned long long* dst, int limit) {
    return poll_words<1, kPipe>(p, n, [&](int i, unsigned long long w) { dst[i] = ~w; }, limit);
}

// The n words at p, decoded to dst (LDS).
template <bool kPipe = false>
__device__ __forceinline__ bool wait_words(unsigned long long* p, int n, double* dst, int limit) {
    return poll_words<4, kPipe>(p, n, [&](int i, unsigned long long w) { dst[i] = decode_word(w); }, limit);
}

// The n (K, S) word pairs at p, decoded to K[i] (float) and S[i] (LDS).
template <bool kPipe = false>
__device__ __forceinline__ bool wait_ks(unsigned long long* p, int n, float* K, double* S, int limit) {
    return poll_words<4, kPipe>(p, 2 * n, [&](int i, unsigned long long w) {
        if (i & 1)
            S[i >> 1] = decode_word(w);
        else
            K[i >> 1] = (float)decode_word(w);
    }, limit);
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
template <class D, int KIND, bool kFlat, class W>
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
                const float a = w.template eval<KIND, kFlat>(zp[e], two_rows ? zq[e] : -INFINITY);
                if (wout != nullptr && v * E + e < n) wout[v * E + e] = a;
                acc += (double)a;
            }
        }
    }
    return wave_sum(acc);
}

template <class D, bool kFlat = false, class W>
__device__ double wave_weight_sum(const typename D::T* rp, const typename D::T* rq, int n, const W& w,
                                  float* wout) {
    return (w.kind == kTargetRow) ? wave_weight_sum_k<D, kTargetRow, kFlat>(rp, rq, n, w, wout)
                                  : wave_weight_sum_k<D, kResidual, kFlat>(rp, rq, n, w, wout);
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
// sub-chunk total at or below t.  Thread i holds vectors i NV .. i NV + NV - 1
// (n <= kThreads * NV * E), so one workgroup scan follows element order.
// Valid in every thread.
template <class D, int KIND, int NV, bool kFlat, class W>
__device__ __forceinline__ int sub_chunk_find_k(const typename D::T* rp, const typename D::T* rq, int n,
                                                const W& w, double t, double* scratch, double* incl_s,
                                                int* iscratch, int* result) {
    constexpr int E = D::E;
    constexpr int NE = NV * E;
    constexpr bool two_rows = (KIND == kResidual);
    const int tid = threadIdx.x;
    const bool fast = pair_aligned<D>(rp, rq, two_rows);
    float zp[NV][E], zq[NV][E];
    load_pair_u<D, NV>(rp, rq, two_rows, fast, tid * NV, 1, n, zp, zq);
    float a[NE];
    double sum = 0.0;
#pragma unroll
    for (int u = 0; u < NV; ++u)
#pragma unroll
        for (int e = 0; e < E; ++e) {
            a[u * E + e] = w.template eval<KIND, kFlat>(zp[u][e], zq[u][e]);
            sum += (double)a[u * E + e];
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
            for (int e = 0; e < NE; ++e) {
                if (a[e] > 0.0f) lastp = e;
                cum += (double)a[e];
                if (idx < 0 && cum > t && a[e] > 0.0f) idx = e;
            }
            if (idx < 0) idx = lastp;
            *result = (idx >= 0) ? tid * NE + idx : -1;
        }
    } else {
        // t lies at or beyond the sub-chunk total (rounding only): the last positive weight
        int lastp = -1;
#pragma unroll
        for (int e = 0; e < NE; ++e)
            if (a[e] > 0.0f) lastp = tid * NE + e;
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

template <class D, bool kFlat = false, class W>
__device__ int sub_chunk_find(const typename D::T* rp, const typename D::T* rq, int n, const W& w, double t,
                              double* scratch, double* incl_s, int* iscratch, int* result) {
    return (w.kind == kTargetRow)
               ? sub_chunk_find_k<D, kTargetRow, 1, kFlat>(rp, rq, n, w, t, scratch, incl_s, iscratch, result)
               : sub_chunk_find_k<D, kResidual, 1, kFlat>(rp, rq, n, w, t, scratch, incl_s, iscratch, result);
}

// sub_chunk_find by one wave when the sub-chunk has at most kWave vectors:
// lane i holds vector i, as thread i does there, with the same sums, scan and
// crossing rule, so the same index, without the workgroup barriers.  Valid in
// every lane of the calling wave.
template <class D, int KIND, bool kFlat, class W>
__device__ __forceinline__ int wave_sub_chunk_find_k(const typename D::T* rp, const typename D::T* rq, int n,
                                                     const W& w, double t) {
    constexpr int E = D::E;
    constexpr bool two_rows = (KIND == kResidual);
    const int lane = threadIdx.x % kWave;
    const bool fast = pair_aligned<D>(rp, rq, two_rows);
    float zp[1][E], zq[1][E];
    load_pair_u<D, 1>(rp, rq, two_rows, fast, lane, 1, n, zp, zq);
    float a[E];
    double sum = 0.0;
#pragma unroll
    for (int e = 0; e < E; ++e) {
        a[e] = w.template eval<KIND, kFlat>(zp[0][e], zq[0][e]);
        sum += (double)a[e];
    }
    const double incl = wave_inclusive_scan(sum);
    const unsigned long long over = __ballot(incl > t);
    if (over) {
        const int f = __ffsll((long long)over) - 1;
        const double before = (f == 0) ? 0.0 : lane_f64(incl, f - 1);
        int mine = -1;
        if (lane == f) {
            double cum = before;
            int idx = -1, lastp = -1;
#pragma unroll
            for (int e = 0; e < E; ++e) {
                if (a[e] > 0.0f) lastp = e;
                cum += (double)a[e];
                if (idx < 0 && cum > t && a[e] > 0.0f) idx = e;
            }
            if (idx < 0) idx = lastp;
            mine = (idx >= 0) ? lane * E + idx : -1;
        }
        return __builtin_amdgcn_readlane(mine, f);
    }
    // t lies at or beyond the sub-chunk total (rounding only): the last positive weight
    int lastp = -1;
#pragma unroll
    for (int e = 0; e < E; ++e)
        if (a[e] > 0.0f) lastp = lane * E + e;
    return wave_max_int(lastp);
}

template <class D, bool kFlat = false, class W>
__device__ __forceinline__ int wave_sub_chunk_find(const typename D::T* rp, const typename D::T* rq, int n, const W& w,
                                                   double t) {
    return (w.kind == kTargetRow) ? wave_sub_chunk_find_k<D, kTargetRow, kFlat>(rp, rq, n, w, t)
                                  : wave_sub_chunk_find_k<D, kResidual, kFlat>(rp, rq, n, w, t);
}

// ---------------------------------------------------------------------------
// the fused step: one launch; a workgroup's role follows from its index
//   stats (b, s, k)  exact mode: chunk k of stats slot s of batch element b
//                    (slot_row); each wave publishes its contiguous
//                    quarter's normaliser terms (eq. (4)) as a (K, S) pair
//   decider (b)      b's decision -- eq. (1) at the drafted tokens and the
//                    first-rejection scan -- published as a small record,
//                    one copy per reader (exact mode; in the sigmoid mode,
//                    and in the exact mode's short streams with few pairs to
//                    copy, the mass workgroups decide for themselves)
//   mass (b, k2)     the masses of the final distribution (eqs. (2)-(3), or
//                    the target row) over tile k2, one per wave, published
//   draw (b)         the inverse-CDF draw of b's next token
//   bonus (b)        if every draft is accepted, the draw from target row
//                    gamma straight from that row's stats sums (exact mode;
//                    no second pass over the row) or from its sums of p_hat
//                    published by the sigmoid row tiles (see bonus_role)
// Index order: units u = 0, 1, ...: unit u holds the stats tiles of the rows
// b = u's decision reads and then b's decider (for u < B), followed by the
// mass tiles and then the draw of b = u - lagM (for u >= lagM); then the
// tiles of every target row gamma (stats tiles in the exact mode, sigmoid row
// tiles in the sigmoid mode; when the bonus role draws); then the mass and
// draw roles of the last lagM batch elements; then the bonus workgroups.
// (The sigmoid mode streams nothing for its decisions: its units hold only
// the deciders, and every element's mass and draw roles come after the row
// tiles.)  Decisions and the residual draws of most batch
// elements so finish while the stream still runs, and the stream ends with
// rows whose only remaining work is one scan each.
//
// Each role of b comes after the roles it reads.  A workgroup only waits on
// results of workgroups with smaller indices, and never on a returning
// atomic: the streaming workgroups publish and retire.  Each XCD dispatches
// its workgroups in index order, so the waiting workgroup with the smallest
// index always waits on workgroups that are running and do not wait, or that
// its XCD will dispatch once its running, non-waiting workgroups finish: no
// wait can block forever.  Every wait is also bounded (kMaxSpins), so every
// wave exits regardless.
//
// Segments have uniform unit sizes, so a workgroup finds its role with at
// most one division, from kernel arguments that sit in the first cache lines
// of the argument block together with everything the stats role reads: a
// stats workgroup starts its stream after a single argument fetch.
// ---------------------------------------------------------------------------
struct StepParams {
    Layout y;
    const void* draft;
    const void* target;
    unsigned long long* pslot;     // [B, 2 gamma + 1 slots, nchunk1, kWaves, 2] stats (K, S) pairs
    int B, gamma, V;
    int chunk1, nchunk1;           // exact: row chunks
    int chunkg, nchunkg;           // exact: chunks of target row gamma when the bonus role draws
    float c;                       // exact: log2(e) / T
    int chunk2, nchunk2;           // final-distribution tiles per batch element
    float s, s0;                   // sigmoid: u = fma(z, s, s0)
    int ncopy;                     // copies of each decision record (one per reader)
    int pstride;                   // stats words per batch element
    unsigned long long* qslot;     // short streams: [B, nchunk2, qstride] the mass workgroups' copies of the pairs
    int qstride;
    const int32_t* tokens;
    const float* uniforms;
    const int32_t* gammas;         // ragged variant: drafts of each batch element (1 .. gamma)
    double temperature, alpha, beta;
    unsigned int* header;          // workspace header: [1] sticky error flag, [2] spin limit (0: default)
    unsigned long long* dslot;     // [B, ncopy, kDecisionWords] copies of the published decision
    unsigned long long* mslot;     // [B, nchunk2, kWaves] sub-chunk masses
    int32_t* accepted_len;
    int32_t* next_token;
    double* tau_out;               // optional probes
    float* weight_out;
    double* mass_out;
    double* lognorm_out;
    // row-staged early exit (staged_kernel) only
    unsigned long long* gslot;     // [B, gstride]: gate words of stages 0 .. gamma, then the row deciders' states
    int gate;                      // stages s >= gate wait for the word of row decider s - gate
    int gwords;                    // gate words per stage: max(2 nchunk1, nchunkg)
    int gstride;                   // (gamma + 1) gwords + gamma
};

struct Smem {
    float K[kMaxStatsSub];     // exact: b's stats chunk references
    double S[kMaxStatsSub];    //        and sums
    double rowL[kMaxRows];     // exact: log2-normaliser of each stats slot
    double tau[kMaxGamma];
    double sub[kMaxSub];       // sub-chunk masses of a draw
    double incl[kThreads];
    double scratch[kWaves];
    int iscratch[kWaves];
    float sk[kWaves];
    double ss[kWaves];
    unsigned long long rec[kDecisionWords];
    int result, cross;
    float kmax;
    unsigned long long flags[kWaves][3];
    double cross_t, cross_tot;
};

// The workspace header: word 1 is the sticky error flag (a wait of this or an
// earlier call on the workspace timed out), word 2 the bound on each wait in
// polls (0: kMaxSpins; a test hook).  Both are read once per role; the flag
// only reflects earlier calls there (a later call's outputs are sentinels
// until the workspace is re-initialised), since the kernel boundary orders
// them.
__device__ __forceinline__ int spin_limit(const StepParams& P) {
    const unsigned int v = P.header[2];
    return (v == 0u) ? kMaxSpins : (int)min(v, (unsigned int)kMaxSpins);
}
__device__ __forceinline__ bool sticky_error(const StepParams& P) { return P.header[1] != 0u; }
__device__ __forceinline__ void set_error(const StepParams& P) {
    __hip_atomic_store(P.header + 1, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Stats slots of a batch element: the rows its decision reads first (target
// rows 0 .. gamma - 1, then draft rows 0 .. gamma - 1), target row gamma last.
__device__ __forceinline__ int slot_row(int s, int gamma) { return s < gamma ? s : (s < 2 * gamma ? s + 1 : gamma); }

// The number of drafts of batch element b: gamma, or in the ragged variant
// gammas[b] when it lies in 1 .. gamma (otherwise gamma, and *bad is set: the
// element's outputs are sentinels).
template <bool kRagged>
__device__ __forceinline__ int elem_gamma(const StepParams& P, int b, bool* bad) {
    *bad = false;
    if constexpr (!kRagged) return P.gamma;
    // a scalar load through the constant address space (b is the same in the
    // whole workgroup and gammas is read-only): after the first workgroup of
    // a CU it comes from the scalar cache, not through the stream's memory queue
    const int g = ((const __attribute__((address_space(4))) int32_t*)P.gammas)[b];
    *bad = !(g >= 1 && g <= P.gamma);
    return *bad ? P.gamma : g;
}

__device__ __forceinline__ double min1(double r) { return (r >= 1.0) ? 1.0 : r; }  // keeps NaN

__device__ __forceinline__ void split3(double v, float& hi, float& mid, float& lo) {
    hi = (float)v;
    mid = (float)(v - (double)hi);
    lo = (float)((v - (double)hi) - (double)mid);
}

// The lane's whole vectors l, l + 64, ... of a chunk of nfull vectors at
// base, absorbed in blocks of U (all loads of a block issued before any is
// used, the block sharing one update of the running reference).
template <int U, class D>
__device__ __forceinline__ void stats_stream(const typename D::T* base, int nfull, bool aligned, int lane, float c,
                                             Lse& st) {
    constexpr int E = D::E;
    for (int v0 = 0; v0 < nfull; v0 += U * kWave) {
        float x[U][E];
        if (aligned) {
            u32x4 raw[U];
#pragma unroll
            for (int u = 0; u < U; ++u) raw[u] = load_vec_or_pad<D, true>(base, v0 + u * kWave + lane, nfull);
#pragma unroll
            for (int u = 0; u < U; ++u) unpack<D>(raw[u], x[u]);
        } else {
            // rows that are not 4-byte aligned (16-bit logits with odd V)
#pragma unroll
            for (int u = 0; u < U; ++u) load_elems_or_pad<D>(base, (v0 + u * kWave + lane) * E, nfull * E, x[u]);
        }
        lse_absorb_block<U, E>(st, x, c);
    }
}

// Exact mode, one chunk of one row: sum_x 2^(z c - K) in one streaming pass,
// published as the pair (K, S): K an integral reference (or -inf), S the fp64
// sum of 2^(z c - K) over the chunk, so sum_x e^(z/T) = sum over chunks of
// S 2^K, merged later by exact power-of-two scaling.  Wave w streams the
// contiguous quarter sub_chunk(k, w, ...) of the chunk; the quarters merge
// in wave order.
template <class D, bool kRagged, bool kPipe = false>
__device__ __forceinline__ void stats_role(const StepParams& P, int b, int slot, int k, Smem& sm) {
    static_assert(!(kPipe && kRagged), "the short-stream launch is not ragged");
    using T = typename D::T;
    constexpr int E = D::E;
    const int gamma = P.gamma, V = P.V;
    const float c = P.c;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    int r = slot_row(slot, gamma);
    if constexpr (kRagged) {
        // element b drafts gb tokens: its rows are target 0 .. gb - 1, draft
        // 0 .. gb - 1 and target gb (in the slot of target row gamma); the
        // other slots publish an empty pair without reading anything
        bool gbad;
        const int gb = elem_gamma<true>(P, b, &gbad);
        if (slot == 2 * gamma) {
            r = gb;
        } else if ((slot < gamma) ? (slot >= gb) : (slot - gamma >= gb)) {
            if (threadIdx.x == 0) {
                unsigned long long* out = P.pslot + (size_t)b * P.pstride + ((size_t)slot * P.nchunk1 + k) * 2;
                publish(out, -INFINITY);
                publish(out + 1, 0.0);
            }
            return;
        }
    }
    const int chunk = (slot == 2 * gamma) ? P.chunkg : P.chunk1;
    const T* row = (r <= gamma) ? static_cast<const T*>(P.target) + ((size_t)b * (gamma + 1) + r) * (size_t)V
                                : static_cast<const T*>(P.draft) + ((size_t)b * gamma + (r - gamma - 1)) * (size_t)V;
    const Span sp = sub_chunk(k, wave, chunk, V, E);
    const T* base = row + sp.begin;
    const int n = sp.n;
    const int nfull = n / E;  // whole vectors of E elements
    const bool aligned = vec_loadable(base);

    // Lane l takes whole vectors l, l + 64, ... of the quarter in blocks of
    // kUnroll; all loads of a block are issued before any is used, and the
    // block shares one update of the running reference.  A partial vector at
    // the end of a row is absorbed after the loop.  The assignment and order
    // depend only on element indices, never on the row's address, so equal
    // rows give bit-identical sums.
    Lse st{-INFINITY, 0.0};
    if constexpr (kPipe) {
        // short streams: blocks no deeper than the lane's vectors (short
        // chunks hold one or two per lane)
        const int per_lane = (nfull + kWave - 1) / kWave;
        if (per_lane <= 1)
            stats_stream<1, D>(base, nfull, aligned, lane, c, st);
        else if (per_lane <= 2)
            stats_stream<2, D>(base, nfull, aligned, lane, c, st);
        else if (per_lane <= 4)
            stats_stream<4, D>(base, nfull, aligned, lane, c, st);
        else
            stats_stream<kUnroll, D>(base, nfull, aligned, lane, c, st);
    } else {
        for (int v0 = 0; v0 < nfull; v0 += kUnroll * kWave) {
            float x[kUnroll][E];
            if (aligned) {
                u32x4 raw[kUnroll];
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) raw[u] = load_vec_or_pad<D, true>(base, v0 + u * kWave + lane, nfull);
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) unpack<D>(raw[u], x[u]);
            } else {
                // rows that are not 4-byte aligned (16-bit logits with odd V)
#pragma unroll
                for (int u = 0; u < kUnroll; ++u)
                    load_elems_or_pad<D>(base, (v0 + u * kWave + lane) * E, nfull * E, x[u]);
            }
            lse_absorb_block<kUnroll, E>(st, x, c);
        }
    }
    if (n > nfull * E && lane == nfull % kWave) {
        float x[1][E];
        load_elems_or_pad<D>(base, nfull * E, n, x[0]);
        lse_absorb_block<1, E>(st, x, c);
    }
    if (slot == 2 * gamma) {
        // target row gamma: one pair per wave, so the bonus draw scans a
        // single quarter (one vector per thread)
        const Lse w = wave_lse(st);
        if (lane == 0) {
            unsigned long long* out =
                P.pslot + (size_t)b * P.pstride + ((size_t)slot * P.nchunk1 + (size_t)k * kWaves + wave) * 2;
            publish(out, (double)w.k);
            publish(out + 1, w.s);
        }
        return;
    }
    if constexpr (kPipe) {
        // short streams: the pair goes to b's decider and, where b's mass
        // workgroups decide for themselves (qstride > 0), to each of them,
        // one copy per thread
        const Lse t = block_lse_all(st, sm.sk, sm.ss);
        const size_t at = ((size_t)slot * P.nchunk1 + k) * 2;
        const int ncp = (P.qstride > 0) ? P.nchunk2 : 0;
        for (int j = threadIdx.x; j <= ncp; j += kThreads) {
            unsigned long long* out = (j == 0) ? P.pslot + (size_t)b * P.pstride + at
                                               : P.qslot + ((size_t)b * P.nchunk2 + (j - 1)) * P.qstride + at;
            publish(out, (double)t.k);
            publish(out + 1, t.s);
        }
        return;
    }
    const Lse t = block_lse(st, sm.sk, sm.ss);
    if (threadIdx.x == 0) {
        unsigned long long* out = P.pslot + (size_t)b * P.pstride + ((size_t)slot * P.nchunk1 + k) * 2;
        publish(out, (double)t.k);
        publish(out + 1, t.s);
    }
}

// The target-row weights of a bonus draw: exact mode 2^(z c - kq) on the
// scale of a quarter with reference kq (eq. (4) before normalisation),
// sigmoid mode sigma(u(z)) (eq. (5), unnormalised).
template <bool kExact>
struct BonusWeights;
template <>
struct BonusWeights<true> {
    static __device__ __forceinline__ ExactWeights of(const StepParams& P, float kq) {
        ExactWeights w{};
        w.kind = kTargetRow;
        w.c = P.c;
        w.kp = kq;
        return w;
    }
};
template <>
struct BonusWeights<false> {
    static __device__ __forceinline__ SigmoidWeights of(const StepParams& P, float) {
        SigmoidWeights w{};
        w.kind = kTargetRow;
        w.s = P.s;
        w.s0 = P.s0;
        return w;
    }
};

// Sigmoid mode, tile k of the row the next token is drawn from when every
// draft is accepted (target row gamma, or gammas[b]): the masses
// sum_x sigma(u(x)) of its quarters (eq. (5), unnormalised), one per wave,
// published as pairs (0, S) in the slots of the exact mode's row-gamma pairs,
// so that the bonus role draws from them the same way.  It waits for nothing:
// the row needs no normaliser, so the draw need not wait for the decision.
template <class D, bool kRagged>
__device__ __forceinline__ void sigmoid_row_role(const StepParams& P, int b, int k) {
    using T = typename D::T;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    bool gbad;
    const int gb = elem_gamma<kRagged>(P, b, &gbad);
    const T* row = static_cast<const T*>(P.target) + ((size_t)b * (P.gamma + 1) + gb) * (size_t)P.V;
    const Span sp = sub_chunk(k, wave, P.chunkg, P.V, D::E);
    const SigmoidWeights w = BonusWeights<false>::of(P, 0.0f);
    const double m = (sp.n > 0) ? wave_weight_sum<D>(row + sp.begin, row + sp.begin, sp.n, w, nullptr) : 0.0;
    if (lane == 0) {
        unsigned long long* out =
            P.pslot + (size_t)b * P.pstride + ((size_t)2 * P.gamma * P.nchunk1 + (size_t)k * kWaves + wave) * 2;
        publish(out, 0.0);
        publish(out + 1, m);
    }
}

// log2(s) for a finite s > 0, to about 1.3e-7 absolute: s = M 2^e exactly
// (M in [1, 2)), log2(M) from the hardware fp32 logarithm of M rounded to
// fp32 (within an ulp of log2(M) < 1, i.e. 1.2e-7) plus the first-order term
// of the rounding, (M - m) / (m ln 2).  The decision margin the parity bar
// allows is 1e-6, and the one-pass fp64 chain this replaces was a long
// dependent path on the step's critical chain.
__device__ __forceinline__ double log2_pos(double s) {
    int e;
    const double M = 2.0 * frexp(s, &e);  // [1, 2)
    const float m = (float)M;
    return (double)(e - 1) + (double)__builtin_amdgcn_logf(m) + (M - (double)m) / ((double)m * 0.6931471805599453094);
}

// log2_pos with the correction term in fp32 (it is below 9e-8, so its fp32
// rounding is far below the decision margin): no fp64 division on the chain.
__device__ __forceinline__ double log2_pos_fast(double s) {
    int e;
    const double M = 2.0 * frexp(s, &e);  // [1, 2)
    const float m = (float)M;
    const float corr = (float)(M - (double)m) * __builtin_amdgcn_rcpf(m) * kLog2e;
    return (double)(e - 1) + (double)__builtin_amdgcn_logf(m) + (double)corr;
}

// 2^l for l <= 0 (larger l return 1, the clamp of eq. (1)), to about 1.5e-7
// relative: 2^floor(l) exactly times the hardware fp32 2^f of the fraction
// f = l - floor(l) in [0, 1) (its fp32 rounding adds under 3e-8).
__device__ __forceinline__ double exp2_nonpos(double l) {
    if (!(l < 0.0)) return (l == l) ? 1.0 : l;
    if (l < -1074.0) return 0.0;
    const double fl = floor(l);
    return ldexp((double)__builtin_amdgcn_exp2f((float)(l - fl)), (int)fl);
}

// Row log2-normalisers Lambda = Kmax + log2(sum S 2^(K - Kmax)) of R rows
// from the (K, S) pairs of their W sub-chunks in LDS, into sm.rowL: row i
// belongs to an aligned group of G lanes (the largest power of two <= 16 with
// R G <= kThreads, rows beyond kThreads in further rounds); lane g of the
// group takes pairs g, g + G, ... in order, and a DPP butterfly combines the
// group in a fixed order, so equal rows give equal bits.  The group's first
// lane takes the logarithm.  Ends with a workgroup barrier.
// The group size follows from Rg if given (else R): merging fewer rows with
// the group size of Rg rows gives each row the same bits as the larger merge.
// kFast (the short-stream launch, where the merge is on the step's critical
// chain): a lane's pairs are read from LDS up to four at a time with their
// loads issued together and kept in registers for the sum, and the logarithm
// takes log2_pos_fast.  The sums run in the same order, so only the last bits
// of the logarithm differ from the plain merge.
template <bool kFast = false>
__device__ __forceinline__ void merge_rows(Smem& sm, int R, int W, int Rg = 0) {
    const int Rs = (Rg > 0) ? Rg : R;
    const int G = (Rs <= 16) ? 16 : (Rs <= 32) ? 8 : (Rs <= 64) ? 4 : (Rs <= 128) ? 2 : 1;
    const int g = threadIdx.x % G;
    for (int i0 = 0; i0 < R; i0 += kThreads / G) {
        const int i = i0 + (int)threadIdx.x / G;
        const bool row = i < R;
        const float* K = sm.K + (size_t)i * W;
        const double* S = sm.S + (size_t)i * W;
        float m = -INFINITY;
        double sum = 0.0;
        if constexpr (kFast) {
            constexpr int kBatch = 4;
            if (W <= kBatch * G) {
                float kb[kBatch];
                double sb[kBatch];
#pragma unroll
                for (int u = 0; u < kBatch; ++u) {
                    const int j = g + u * G;
                    kb[u] = (row && j < W) ? K[j] : -INFINITY;
                    sb[u] = (row && j < W) ? S[j] : 0.0;
                }
#pragma unroll
                for (int u = 0; u < kBatch; ++u) m = fmaxf(m, kb[u]);
                m = group_max(m, G);
#pragma unroll
                for (int u = 0; u < kBatch; ++u)
                    if (row && g + u * G < W) sum += ldexp(sb[u], exp_delta(kb[u] - m));
            } else {
                if (row)
                    for (int j = g; j < W; j += G) m = fmaxf(m, K[j]);
                m = group_max(m, G);
                if (row)
                    for (int j = g; j < W; j += G) sum += ldexp(S[j], exp_delta(K[j] - m));
            }
        } else {
            if (row)
                for (int j = g; j < W; j += G) m = fmaxf(m, K[j]);
            m = group_max(m, G);
            if (row)
                for (int j = g; j < W; j += G) sum += ldexp(S[j], exp_delta(K[j] - m));
        }
        sum = group_sum(sum, G);
        // a NaN logit makes S NaN; a +inf logit makes K +inf and S NaN
        if (row && g == 0)
            sm.rowL[i] = (sum != sum) ? __builtin_nan("")
                         : ((m == -INFINITY) ? -INFINITY
                                             : (double)m + ((sum > 0.0 && sum < INFINITY)
                                                                ? (kFast ? log2_pos_fast(sum) : log2_pos(sum))
                                                                : log2(sum)));
    }
    __syncthreads();
}

// The short streams' wait for the R decision rows' pairs at p (W per row)
// and their merge into sm.rowL, with no LDS staging: thread (i, g) of the
// merge (row i = tid / G, lane g of the row's group of G, G as in
// merge_rows) polls the words of its own pairs g, g + G, g + 2G, g + 3G
// directly (two polls in flight), the workgroup agrees through LDS flags
// that every pair is in, and the merge then runs on the registers: the same
// values, order and group butterfly as merge_rows<true>, so the same bits.
// Needs W <= 4 G (the caller checks).  Ends with a workgroup barrier.
__device__ __forceinline__ bool wait_merge_rows(const unsigned long long* p, int R, int W, Smem& sm, int limit) {
    constexpr int kB = 4;
    const int G = (R <= 16) ? 16 : (R <= 32) ? 8 : (R <= 64) ? 4 : (R <= 128) ? 2 : 1;
    const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
    const int i = tid / G, g = tid % G;
    const int nu = (W + G - 1) / G;  // pairs per lane (uniform)
    const bool row = i < R;
    const int ic = min(i, R - 1);
    bool have[kB];
    const unsigned long long* q[kB];
#pragma unroll
    for (int u = 0; u < kB; ++u) {
        const int j = g + u * G;
        have[u] = row && j < W;
        q[u] = p + 2 * ((size_t)ic * W + min(j, W - 1));
    }
    __shared__ int mflag[2][kWaves];
    unsigned long long a[2 * kB], c[2 * kB];
    auto issue = [&](unsigned long long (&w)[2 * kB]) {
#pragma unroll
        for (int u = 0; u < kB; ++u) {
            if (u < nu) {
                w[2 * u] = __hip_atomic_load(q[u], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                w[2 * u + 1] = __hip_atomic_load(q[u] + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            } else {
                w[2 * u] = w[2 * u + 1] = 0ull;
            }
        }
    };
    auto check = [&](const unsigned long long (&w)[2 * kB], int round) {
        bool missing = false;
#pragma unroll
        for (int u = 0; u < kB; ++u) missing |= have[u] && (w[2 * u] == 0ull || w[2 * u + 1] == 0ull);
        const unsigned long long m = __ballot(missing);
        if (lane == 0) mflag[round & 1][wave] = (m != 0ull) ? 1 : 0;
        lds_barrier();
        int any = 0;
#pragma unroll
        for (int w2 = 0; w2 < kWaves; ++w2) any |= mflag[round & 1][w2];
        return any == 0;
    };
    unsigned long long w[2 * kB];
    bool ok = false;
    issue(a);
    for (int round = 0;; round += 2) {
        issue(c);
        if (check(a, round)) {
#pragma unroll
            for (int k = 0; k < 2 * kB; ++k) w[k] = a[k];
            ok = true;
            break;
        }
        if (round + 1 >= limit) break;
        issue(a);
        if (check(c, round + 1)) {
#pragma unroll
            for (int k = 0; k < 2 * kB; ++k) w[k] = c[k];
            ok = true;
            break;
        }
        if (round + 2 >= limit) break;
    }
    if (!ok) {
#pragma unroll
        for (int k = 0; k < 2 * kB; ++k) w[k] = 0ull;  // decodes as a NaN pair: the caller reports the timeout
    }
    float kb[kB];
    double sb[kB];
#pragma unroll
    for (int u = 0; u < kB; ++u) {
        kb[u] = have[u] ? (float)decode_word(w[2 * u]) : -INFINITY;
        sb[u] = have[u] ? decode_word(w[2 * u + 1]) : 0.0;
    }
    float m = -INFINITY;
#pragma unroll
    for (int u = 0; u < kB; ++u) m = fmaxf(m, kb[u]);
    m = group_max(m, G);
    double sum = 0.0;
#pragma unroll
    for (int u = 0; u < kB; ++u)
        if (have[u]) sum += ldexp(sb[u], exp_delta(kb[u] - m));
    sum = group_sum(sum, G);
    if (row && g == 0)
        sm.rowL[i] = (sum != sum) ? __builtin_nan("")
                     : ((m == -INFINITY) ? -INFINITY
                                         : (double)m + ((sum > 0.0 && sum < INFINITY) ? log2_pos_fast(sum) : log2(sum)));
    __syncthreads();
    return ok;
}

// For the drafts c < gamma (thread c holds stop_c: 0 accepted, 1 rejected, 2
// unreadable, and tok_ok): the first c with stop_c != 0 (kThreads if none),
// whether that one is unreadable, and whether any drafted token is out of
// range.  One workgroup barrier.
__device__ __forceinline__ void scan_stops(int stop, bool tok_ok, Smem& sm, int* first, bool* first_bad,
                                           bool* tok_bad) {
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const unsigned long long rej = __ballot(stop != 0);
    const unsigned long long unr = __ballot(stop == 2);
    const unsigned long long tok = __ballot(!tok_ok);
    if (lane == 0) {
        sm.flags[wave][0] = rej;
        sm.flags[wave][1] = unr;
        sm.flags[wave][2] = tok;
    }
    __syncthreads();
    int f = kThreads;
    bool fb = false, tb = false;
#pragma unroll
    for (int w = kWaves - 1; w >= 0; --w) {
        const unsigned long long r = sm.flags[w][0];
        if (r != 0) {
            const int l = __ffsll((long long)r) - 1;
            f = w * kWave + l;
            fb = ((sm.flags[w][1] >> l) & 1ull) != 0;
        }
        tb |= sm.flags[w][2] != 0;
    }
    *first = f;
    *first_bad = fb;
    *tok_bad = tb;
}

// The largest of one row's W sub-chunk references (valid in every thread).
__device__ __forceinline__ float row_kmax(Smem& sm, const float* K, int W) {
    const int tid = threadIdx.x;
    float m = -INFINITY;
    for (int j = tid; j < W; j += kThreads) m = fmaxf(m, K[j]);
    m = wave_max(m);
    if (tid % kWave == 0) sm.sk[tid / kWave] = m;
    __syncthreads();
    if (tid == 0) {
        float mm = sm.sk[0];
        for (int w = 1; w < kWaves; ++w) mm = fmaxf(mm, sm.sk[w]);
        sm.kmax = mm;
    }
    __syncthreads();
    return sm.kmax;
}

struct Decision {
    int L;        // accepted length, in [0, gb]
    int gb;       // the element's number of drafts
    bool bad;     // sentinel
    bool ok;      // false if a wait timed out
    ExactWeights ew;
    SigmoidWeights sw;
};

// The decision for batch element b: eq. (1) at the drafted tokens and the
// first-rejection scan, plus the weights of the final distribution.
template <class D, bool kExact, bool kRagged, bool kPipe = false>
__device__ __forceinline__ Decision decide(const StepParams& P, int b, Smem& sm, unsigned long long* ks = nullptr) {
    using T = typename D::T;
    const int gamma = P.gamma, V = P.V;
    const int tid = threadIdx.x;
    bool gbad;
    const int gb = elem_gamma<kRagged>(P, b, &gbad);
    const T* draft = static_cast<const T*>(P.draft) + (size_t)b * gamma * V;
    const T* target = static_cast<const T*>(P.target) + (size_t)b * (gamma + 1) * V;

    // independent loads first: tokens, uniforms and the drafted-token logits.
    // In the short-stream launch with at most kWave drafts every wave takes
    // all drafts (lane c draft c), so that eq. (1) and the first-rejection
    // scan need no exchange between waves.
    const bool inwave = kPipe && gb <= kWave;
    const int c = inwave ? tid % kWave : tid;
    int x = 0;
    double r = 0.0;
    bool tok_ok = true;
    float zp = 0.0f, zq = 0.0f;
    if (c < gb) {
        x = P.tokens[(size_t)b * gamma + c];
        r = (double)P.uniforms[(size_t)b * (gamma + 1) + c];
        tok_ok = (x >= 0 && x < V);
        const int xs = tok_ok ? x : 0;
        zp = to_f32(target[(size_t)c * V + xs]);
        zq = to_f32(draft[(size_t)c * V + xs]);
    }

    Decision d{};
    d.ok = true;
    if (kExact) {
        // the stats slots the decision reads, merged into log2-normalisers
        // max K + log2(sum S 2^(K - max K)) by exact power-of-two scaling
        const int W = P.nchunk1;  // chunks per row
        unsigned long long* src = (ks != nullptr) ? ks : P.pslot + (size_t)b * P.pstride;
        const int R = 2 * gamma;
        const int G = (R <= 16) ? 16 : (R <= 32) ? 8 : (R <= 64) ? 4 : (R <= 128) ? 2 : 1;
        if (kPipe && W <= 4 * G) {
            d.ok = wait_merge_rows(src, R, W, sm, spin_limit(P));
        } else {
            d.ok = wait_ks<kPipe>(src, R * W, sm.K, sm.S, spin_limit(P));
            merge_rows<kPipe>(sm, R, W);
        }
    }

    int stop = 0;
    if (c < gb) {
        double tau;
        bool row_ok;
        if (kExact) {
            const double lam_p = sm.rowL[c];          // target row c
            const double lam_q = sm.rowL[gamma + c];  // draft row c
            row_ok = isfinite(lam_p) && isfinite(lam_q);
            if (zq == -INFINITY) {
                tau = 1.0;  // q(x) = 0
            } else {
                const double l2 = ((double)zp - (double)zq) * (double)P.c - (lam_p - lam_q);
                tau = exp2_nonpos(l2);
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
        if (c == tid) sm.tau[c] = tau;
        stop = !row_ok ? 2 : ((r <= tau) ? 0 : 1);
    }
    // the first draft that is rejected (or unreadable) ends the accepted prefix
    int first;
    bool first_bad, tok_bad;
    if (inwave) {
        const unsigned long long rej = __ballot(stop != 0);
        const unsigned long long unr = __ballot(stop == 2);
        const int l = rej ? __ffsll((long long)rej) - 1 : 0;
        first = rej ? l : kThreads;
        first_bad = rej && ((unr >> l) & 1ull) != 0;
        tok_bad = __ballot(!tok_ok) != 0ull;
    } else {
        scan_stops(stop, tok_ok, sm, &first, &first_bad, &tok_bad);
    }
    d.L = min(first, gb);
    d.gb = gb;
    // target row gb is the bonus role's business (it sentinels a non-finite
    // row itself)
    d.bad = gbad || tok_bad || first_bad || !d.ok;
    const bool two_rows = d.L < gb;
    if (kExact && !d.bad && two_rows) {
        const double lp = sm.rowL[d.L];
        const double lq = sm.rowL[gamma + d.L];
        d.ew.kind = kResidual;
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

// Fixed-order prefix over M (<= 4 kThreads) masses m[] in LDS, four
// consecutive ones per thread: loc receives the thread's masses, sm.incl[tid]
// its inclusive prefix.  Returns the total, valid in every thread.
__device__ __forceinline__ double mass_prefix(const double* m, int M, Smem& sm, double (&loc)[4]) {
    const int tid = threadIdx.x;
    double ls = 0.0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int j = tid * 4 + i;
        loc[i] = (j < M) ? m[j] : 0.0;
        ls += loc[i];
    }
    double tot;
    sm.incl[tid] = block_inclusive_scan(ls, sm.scratch, &tot);
    return tot;
}

// After mass_prefix: the index of the mass in which the running sum first
// exceeds t (or the last positive one, if rounding leaves the total at or
// below t), with t minus the running sum before it in *t_local; -1 if no
// mass is positive.  Valid in every thread.
__device__ __forceinline__ int mass_locate(const double* m, int M, double t, const double (&loc)[4], Smem& sm,
                                           double* t_local) {
    const int tid = threadIdx.x;
    const int first = block_first(sm.incl[tid] > t, sm.iscratch);
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
        // rounding only: the last positive weight of the last mass with weight
        for (int j = M - 1; j >= 0; --j)
            if (m[j] > 0.0) {
                sm.cross = j;
                sm.cross_t = m[j];
                break;
            }
    }
    __syncthreads();
    *t_local = sm.cross_t;
    return sm.cross;
}

// Inverse-CDF locate over at most kWave masses by one wave (all its lanes
// call this; lane l holds mass l, 0 beyond the last): sm.cross receives the
// first mass at which the running sum exceeds t = u * total -- or the last
// positive mass, if rounding leaves t at or beyond the total; -1 if no mass
// is positive -- sm.cross_t the part of t inside it and sm.cross_tot the
// total.  The caller's barrier publishes them.
// (wave_locate_r returns the results in registers, valid in every lane of the
// wave, so that one wave can finish a draw without a workgroup barrier.)
struct Located {
    double tot;      // the total of the masses
    int j;           // the mass the draw falls in, or -1
    double t_local;  // the part of u * tot inside mass j
};

__device__ __forceinline__ Located wave_locate_r(double m, double u) {
    const double incl = wave_inclusive_scan(m);
    const double tot = lane_f64(incl, kWave - 1);
    const double t = u * tot;
    const unsigned long long over = __ballot(incl > t && m > 0.0);
    const unsigned long long pos = __ballot(m > 0.0);
    const int j = over ? __ffsll((long long)over) - 1 : (pos ? 63 - __clzll((long long)pos) : -1);
    const int jc = max(j, 0);
    const double before = lane_f64(incl, max(jc - 1, 0));
    const double mj = lane_f64(m, jc);
    return Located{tot, j, over ? t - ((jc == 0) ? 0.0 : before) : mj};
}

__device__ __forceinline__ void wave_locate(double m, double u, Smem& sm) {
    const Located r = wave_locate_r(m, u);
    if (threadIdx.x % kWave == 0) {
        sm.cross_tot = r.tot;
        sm.cross = r.j;
        sm.cross_t = r.t_local;
    }
}

// mass_prefix + mass_locate by one wave when M <= 4 kWave: lane l holds
// masses 4 l .. 4 l + 3, as thread l does there, with the same sums, scan and
// crossing rule, so the same total, mass and remainder, left in
// sm.cross_tot, sm.cross (-1 if none) and sm.cross_t as wave_locate leaves
// them; the caller's barrier publishes them.  Called by the lanes of one wave.
__device__ __forceinline__ void wave_locate4(const double* m, int M, double u, Smem& sm) {
    const int lane = threadIdx.x % kWave;
    double loc[4];
    double ls = 0.0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int k = lane * 4 + i;
        loc[i] = (k < M) ? m[k] : 0.0;
        ls += loc[i];
    }
    const double incl = wave_inclusive_scan(ls);
    const double tot = lane_f64(incl, kWave - 1);
    int j = -1;
    double tl = 0.0;
    if (isfinite(tot) && tot > 0.0) {
        const double t = u * tot;
        const unsigned long long over = __ballot(incl > t);
        if (over) {
            const int f = __ffsll((long long)over) - 1;
            const double cum0 = (f == 0) ? 0.0 : lane_f64(incl, f - 1);
            int jl = -1;
            double rem = 0.0;
            if (lane == f) {
                double cum = cum0, before = cum0, lastp_before = 0.0;
                int lastp = -1;
                for (int i = 0; i < 4; ++i) {
                    if (loc[i] > 0.0) {
                        lastp = lane * 4 + i;
                        lastp_before = cum;
                    }
                    if (jl < 0 && cum + loc[i] > t && loc[i] > 0.0) {
                        jl = lane * 4 + i;
                        before = cum;
                    }
                    cum += loc[i];
                }
                if (jl < 0) {
                    jl = lastp;
                    before = lastp_before;
                }
                rem = t - before;
            }
            j = __builtin_amdgcn_readlane(jl, f);
            tl = lane_f64(rem, f);
        } else {
            // rounding only: the last positive mass, whole
            int lp = -1;
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (loc[i] > 0.0) lp = lane * 4 + i;
            j = wave_max_int(lp);
            tl = (j >= 0) ? m[j] : 0.0;
        }
    }
    if (lane == 0) {
        sm.cross_tot = tot;
        sm.cross = j;
        sm.cross_t = tl;
    }
}



// b's decision, made once by b's decider workgroup and, in the exact mode,
// published as a small record, one copy per reader (each mass workgroup, the
// draw, the bonus workgroup; only the last two when the mass workgroups
// decide for themselves), which that reader clears once it has read it.
// Copies before `first` are not written.
// The decider also writes the tau / normaliser probes and clears the stats
// words it read (it is their only reader).
// The P.ncopy copies of b's decision record (L, the sentinel flag, gb and the
// residual's constants), written by every thread of the workgroup.
__device__ __forceinline__ void publish_decision(const StepParams& P, int b, const Decision& d, int first = 0) {
    const unsigned long long rec[kDecisionWords] = {
        (unsigned long long)(d.L & 0xffff) | ((unsigned long long)(d.bad ? 1 : 0) << 16) | (1ull << 32) |
            ((unsigned long long)(d.gb & 0xffff) << 40),
        pack2(d.ew.kp, d.ew.lp_hi), pack2(d.ew.lp_lo, d.ew.kq), pack2(d.ew.lq_hi, d.ew.lq_lo),
        pack2(d.ew.d_hi, d.ew.d_lo)};
    unsigned long long* dst = P.dslot + (size_t)b * P.ncopy * kDecisionWords;
    for (int i = first * kDecisionWords + (int)threadIdx.x; i < P.ncopy * kDecisionWords; i += kThreads) {
        const int w = i % kDecisionWords;
        unsigned long long v = rec[0];
#pragma unroll
        for (int k = 1; k < kDecisionWords; ++k) v = (w == k) ? rec[k] : v;
        publish_raw(dst + i, v);
    }
}

template <class D, bool kExact, bool kRagged, bool kPipe = false>
__device__ __forceinline__ void decider_role(const StepParams& P, int b, Smem& sm) {
    const int gamma = P.gamma, R = 2 * gamma + 1;
    const int tid = threadIdx.x;
    const Decision d = decide<D, kExact, kRagged, kPipe>(P, b, sm);
    if (!d.ok && tid == 0) set_error(P);
    // (sigmoid mode and the short streams' mass workgroups decide for
    // themselves: the sigmoid mode's only copy is the bonus workgroup's, the
    // short streams' are the draw's and the bonus workgroup's)
    publish_decision(P, b, d, (kPipe && kExact && P.qstride > 0) ? P.nchunk2 : 0);
    if (P.tau_out != nullptr && tid < gamma) P.tau_out[(size_t)b * gamma + tid] = sm.tau[tid];
    if (kExact) {
        const int W = P.nchunk1;
        if (P.lognorm_out != nullptr)
            for (int i = tid; i < 2 * gamma; i += kThreads)
                P.lognorm_out[(size_t)b * R + slot_row(i, gamma)] = sm.rowL[i] * 0.693147180559945309417;
        for (int i = tid; i < 4 * gamma * W; i += kThreads) clear_word(P.pslot + (size_t)b * P.pstride + i);
    }
}

// The decision held in a record's five words (rec, as published), with ok
// false when the wait for them timed out.
__device__ __forceinline__ Decision decode_record(const StepParams& P, const unsigned long long* rec, bool ok,
                                                  bool exact);

// Copy `copy` of b's published decision (in b's mass, draw and bonus
// workgroups), cleared once read.
template <bool kPipe = false>
__device__ __forceinline__ Decision read_decision(const StepParams& P, int b, int copy, bool exact, Smem& sm) {
    unsigned long long* src = P.dslot + ((size_t)b * P.ncopy + copy) * kDecisionWords;
    const bool ok = wait_raw<kPipe>(src, kDecisionWords, sm.rec, spin_limit(P));
    if ((int)threadIdx.x < kDecisionWords) clear_word(src + threadIdx.x);
    return decode_record(P, sm.rec, ok, exact);
}

// The record's words (raw, as published) by one wave on its own: lanes
// 0 .. 4 poll them with two polls in flight and the wave goes on as soon as
// it has all five, with no exchange with the other waves of its workgroup
// (which poll their own).  rec receives the words in every lane.  The caller
// clears the record once every wave has read it.
__device__ __forceinline__ bool wave_wait_record(const unsigned long long* src, unsigned long long* rec, int limit) {
    const int lane = threadIdx.x % kWave;
    const unsigned long long* p = src + min(lane, kDecisionWords - 1);
    const bool mine = lane < kDecisionWords;
    unsigned long long a = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT), c = 0ull, w = 0ull;
    bool ok = false;
    for (int round = 0;; round += 2) {
        c = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (__ballot(mine && a == 0ull) == 0ull) {
            w = a;
            ok = true;
            break;
        }
        if (round + 1 >= limit) break;
        a = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (__ballot(mine && c == 0ull) == 0ull) {
            w = c;
            ok = true;
            break;
        }
        if (round + 2 >= limit) break;
    }
#pragma unroll
    for (int k = 0; k < kDecisionWords; ++k) rec[k] = ~lane_u64(w, k);
    return ok;
}

__device__ __forceinline__ Decision decode_record(const StepParams& P, const unsigned long long* rec, bool ok,
                                                  bool exact) {
    Decision d{};
    d.ok = ok;
    const unsigned long long w0 = rec[0];
    d.L = d.ok ? (int)(w0 & 0xffff) : 0;
    d.gb = d.ok ? (int)((w0 >> 40) & 0xffff) : P.gamma;
    d.bad = ((w0 >> 16) & 1) != 0 || !d.ok;
    // a record from this call always has 0 <= L <= gb <= gamma; anything else
    // is left over from a call whose wait timed out (the workspace is then
    // dirty): a sentinel, and indices kept in range
    if (d.gb < 1 || d.gb > P.gamma || d.L > d.gb) {
        d.bad = true;
        d.gb = P.gamma;
        d.L = 0;
    }
    const int kind = (d.L < d.gb) ? kResidual : kTargetRow;
    if (exact) {
        d.ew.kind = kind;
        d.ew.c = P.c;
        d.ew.kp = unpack_hi(rec[1]);
        d.ew.lp_hi = unpack_lo(rec[1]);
        d.ew.lp_lo = unpack_hi(rec[2]);
        d.ew.kq = unpack_lo(rec[2]);
        d.ew.lq_hi = unpack_hi(rec[3]);
        d.ew.lq_lo = unpack_lo(rec[3]);
        d.ew.d_hi = unpack_hi(rec[4]);
        d.ew.d_lo = unpack_lo(rec[4]);
    } else {
        d.sw.kind = kind;
        d.sw.s = P.s;
        d.sw.s0 = P.s0;
    }
    return d;
}

// Index (relative to rp) of the first element of target-row weights
// w(z) = 2^(z c - kp) over n elements whose running sum exceeds t, or of the
// last positive weight if rounding leaves the total at or below t; -1 if no
// weight is positive.  One wave: lane l holds vectors 4 l .. 4 l + 3
// (n <= 4 kWave E), so lane order is element order and no workgroup barrier
// is needed.  Every lane returns the same value.
template <class D, class Wt>
__device__ __forceinline__ int wave_find_target(const typename D::T* rp, int n, const Wt& w, double t) {
    constexpr int E = D::E;
    constexpr int NV = 4;
    constexpr int NE = NV * E;
    const int lane = threadIdx.x % kWave;
    const bool fast = vec_loadable(rp);
    float z[NV][E], zq[NV][E];
    load_pair_u<D, NV>(rp, rp, false, fast, lane * NV, 1, n, z, zq);
    // the weights are recomputed where needed rather than kept (registers)
    double sum = 0.0;
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int e = 0; e < E; ++e) sum += (double)w.template eval<kTargetRow>(z[v][e], -INFINITY);
    const double incl = wave_inclusive_scan(sum);
    const unsigned long long over = __ballot(incl > t);
    int mine = -1;
    if (over) {
        // the crossing lane f's NE elements, one per lane (lanes below NE
        // read element f NE + lane again, now from cache), weighed and
        // scanned across the wave on top of the mass before lane f
        static_assert(NE <= kWave, "one element per lane");
        const int f = __ffsll((long long)over) - 1;
        const double before = (f == 0) ? 0.0 : lane_f64(incl, f - 1);
        const int i = f * NE + lane;
        const bool mine_el = lane < NE && i < n;
        const float a = mine_el ? w.template eval<kTargetRow>(to_f32(rp[max(min(i, n - 1), 0)]), -INFINITY) : 0.0f;
        const double cum = before + wave_inclusive_scan((double)a);
        const unsigned long long hit = __ballot(mine_el && cum > t && a > 0.0f);
        const unsigned long long pos = __ballot(mine_el && a > 0.0f);
        const int idx = hit ? __ffsll((long long)hit) - 1 : (pos ? 63 - __clzll((long long)pos) : -1);
        return (idx >= 0) ? f * NE + idx : -1;
    }
    // t lies at or beyond the total (rounding only): the last positive weight
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int e = 0; e < E; ++e)
            if (w.template eval<kTargetRow>(z[v][e], -INFINITY) > 0.0f) mine = lane * NE + v * E + e;
    return wave_max_int(mine);
}

// Probe outputs of a bonus draw: the draw's total (exact mode in units of the
// row normaliser, 1 up to rounding; sigmoid mode the plain sum of p_hat) and
// the row's weights (exact p(x), sigmoid p_hat(x)).
template <class D, bool kExact>
__device__ __forceinline__ void bonus_probes(const StepParams& P, int b, int gb, float km, double total, bool bad,
                                             int t0, int nt) {
    using T = typename D::T;
    const int gamma = P.gamma, V = P.V;
    auto lam = [&]() { return (double)km + log2(total); };  // exact: the row's log2-normaliser
    if (P.mass_out != nullptr && (int)threadIdx.x == 0)
        P.mass_out[b] = bad ? __builtin_nan("") : (kExact ? total * exp2((double)km - lam()) : total);
    if (P.weight_out != nullptr && !bad) {
        const T* rp = static_cast<const T*>(P.target) + ((size_t)b * (gamma + 1) + gb) * V;
        if constexpr (kExact) {
            ExactWeights w{};
            w.kind = kTargetRow;
            w.c = P.c;
            split3(lam(), w.kp, w.lp_hi, w.lp_lo);
            for (int x = t0; x < V; x += nt) P.weight_out[(size_t)b * V + x] = w.template eval<kTargetRow>(to_f32(rp[x]), -INFINITY);
        } else {
            const SigmoidWeights w = BonusWeights<false>::of(P, 0.0f);
            for (int x = t0; x < V; x += nt) P.weight_out[(size_t)b * V + x] = w.template eval<kTargetRow>(to_f32(rp[x]), -INFINITY);
        }
    }
}

// The bonus draw of b by one wave, when target row gamma has at most kWave
// quarters (see bonus_role): the same steps as the workgroup version, with
// every value in registers and no workgroup barrier, since this chain ends
// the step.  The other waves of the workgroup return at once.
template <class D, bool kExact, bool kRagged, bool kPipe = false>
__device__ __forceinline__ void bonus_wave_role(const StepParams& P, int b) {
    using T = typename D::T;
    if (threadIdx.x >= kWave) return;
    const int gamma = P.gamma, V = P.V, R = 2 * gamma + 1;
    const int lane = threadIdx.x;
    const int W = kWaves * P.nchunkg;  // quarters of the row's tiles, <= kWave
    bool gbad;
    const int gb = elem_gamma<kRagged>(P, b, &gbad);
    const double u = (double)P.uniforms[(size_t)b * (gamma + 1) + gb];
    unsigned long long* rec = P.dslot + ((size_t)b * P.ncopy + P.ncopy - 1) * kDecisionWords;
    unsigned long long* words = P.pslot + (size_t)b * P.pstride + (size_t)2 * gamma * P.nchunk1 * 2;
    const int limit = spin_limit(P);
    const bool sticky = sticky_error(P);
    // lane l < W: the (K, S) words of quarter l
    const int q = min(lane, W - 1);
    unsigned long long wk = 0ull, ws = 0ull;
    bool ok = false;
    if constexpr (!kPipe) {
        for (int spin = 0;; ++spin) {
            wk = __hip_atomic_load(words + 2 * q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            ws = __hip_atomic_load(words + 2 * q + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (__ballot(lane < W && (wk == 0ull || ws == 0ull)) == 0ull) {
                ok = true;
                break;
            }
            if (spin >= limit) break;
            __builtin_amdgcn_s_sleep(2);
        }
    } else {
        // two polls in flight, as in poll_at
        unsigned long long ka, sa, kb, sb;
        ka = __hip_atomic_load(words + 2 * q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        sa = __hip_atomic_load(words + 2 * q + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        for (int spin = 0;; spin += 2) {
            if constexpr (kPollGap > 0) __builtin_amdgcn_s_sleep(kPollGap);
            kb = __hip_atomic_load(words + 2 * q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            sb = __hip_atomic_load(words + 2 * q + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (__ballot(lane < W && (ka == 0ull || sa == 0ull)) == 0ull) {
                wk = ka;
                ws = sa;
                ok = true;
                break;
            }
            if (spin + 1 >= limit) break;
            if constexpr (kPollGap > 0) __builtin_amdgcn_s_sleep(kPollGap);
            ka = __hip_atomic_load(words + 2 * q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            sa = __hip_atomic_load(words + 2 * q + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (__ballot(lane < W && (kb == 0ull || sb == 0ull)) == 0ull) {
                wk = kb;
                ws = sb;
                ok = true;
                break;
            }
            if (spin + 2 >= limit) break;
        }
    }
    // the decision copy, in flight during the draw
    unsigned long long rw = 0ull;
    if (lane < kDecisionWords) rw = __hip_atomic_load(rec + lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    // the masses S 2^(K - Kmax) of the quarters, their total and the quarter
    // the uniform falls in
    const float K = (ok && lane < W) ? (float)decode_word(wk) : -INFINITY;
    const double S = (ok && lane < W) ? decode_word(ws) : 0.0;
    const float km = wave_max(K);
    const Located loc = wave_locate_r(ldexp(S, exp_delta(K - km)), u);
    const double total = loc.tot;
    if (kExact && P.lognorm_out != nullptr && lane == 0)
        P.lognorm_out[(size_t)b * R + gb] = ((double)km + log2(total)) * 0.693147180559945309417;
    // a NaN logit makes the total NaN, an all -inf row makes it 0: sentinel
    int idx = -1;
    if (ok && isfinite(total) && total > 0.0 && loc.j >= 0) {
        const Span sp = sub_chunk(loc.j / kWaves, loc.j % kWaves, P.chunkg, V, D::E);
        const T* rp = static_cast<const T*>(P.target) + ((size_t)b * (gamma + 1) + gb) * V + sp.begin;
        // on the quarter's own scale 2^K: its largest weight is at least 1/2,
        // so a quarter with positive mass has a positive fp32 weight
        const float kj = lane_f32(K, loc.j);
        const int local = wave_find_target<D>(rp, sp.n, BonusWeights<kExact>::of(P, kj),
                                              ldexp(loc.t_local, exp_delta(km - kj)));
        idx = (local >= 0) ? sp.begin + local : -1;
    }
    // b's decision: the outputs are this workgroup's if every draft was
    // accepted (otherwise b's draw workgroup writes them), and also if the
    // decision never arrives (a timed-out wait: then they are sentinels)
    bool rok = true;
    if (__ballot(lane < kDecisionWords && rw == 0ull) != 0ull) {
        rok = false;
        for (int spin = 0; spin < limit; ++spin) {
            __builtin_amdgcn_s_sleep(2);
            if (lane < kDecisionWords) rw = __hip_atomic_load(rec + lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (__ballot(lane < kDecisionWords && rw == 0ull) == 0ull) {
                rok = true;
                break;
            }
        }
    }
    // this workgroup is the only reader of these words: cleared on the way out
    if (lane < W) {
        clear_word(words + 2 * lane);
        clear_word(words + 2 * lane + 1);
    }
    if (lane < kDecisionWords) clear_word(rec + lane);
    if (!(ok && rok) && lane == 0) set_error(P);
    const unsigned long long w0 = ~lane_u64(rw, 0);
    const bool draw = !rok || (((w0 >> 16) & 1) == 0 && (int)(w0 & 0xffff) == gb);
    if (!draw) return;
    const bool bad = !(ok && rok) || sticky || idx < 0;
    if (lane == 0) {
        P.accepted_len[b] = bad ? -1 : gb;
        P.next_token[b] = bad ? -1 : idx;
    }
    bonus_probes<D, kExact>(P, b, gb, km, total, bad, lane, kWave);
}

// b's bonus workgroup: waits for target row gamma's stats (exact mode; they
// stream last) or its sigmoid row tiles (sigmoid mode), draws the next token
// from that row, then reads its copy of b's decision and, if every draft was
// accepted, writes b's outputs.  The masses of the inverse-CDF draw are the
// sums S 2^(K - Kmax) of the row's tile quarters (K = 0 in the sigmoid mode),
// so the draw scans only the one quarter the uniform falls in.
// With at most kWave quarters one wave does all of it (bonus_wave_role);
// otherwise the workgroup, one vector per thread.  It is the only reader of
// row gamma's words and of its decision copy, and clears them.
template <class D, bool kExact, bool kRagged, bool kPipe = false>
__device__ __forceinline__ void bonus_role(const StepParams& P, int b, Smem& sm) {
    using T = typename D::T;
    const int gamma = P.gamma, V = P.V, R = 2 * gamma + 1;
    const int tid = threadIdx.x;
    const int W = kWaves * P.nchunkg;  // quarters of the row's tiles
    if (W <= kWave) {
        bonus_wave_role<D, kExact, kRagged, kPipe>(P, b);
        return;
    }
    bool gbad;
    const int gb = elem_gamma<kRagged>(P, b, &gbad);  // the row drawn from: target row gb
    const double u = (double)P.uniforms[(size_t)b * (gamma + 1) + gb];
    unsigned long long* rec = P.dslot + ((size_t)b * P.ncopy + P.ncopy - 1) * kDecisionWords;
    unsigned long long* words = P.pslot + (size_t)b * P.pstride + (size_t)2 * gamma * P.nchunk1 * 2;
    const int limit = spin_limit(P);
    const bool sticky = sticky_error(P);
    // the row's (K, S) pairs first: the draw does not depend on the decision,
    // so it runs while b's decider may still be at work (the last elements'
    // decisions publish after the stream has ended), and the decision is read
    // only before the outputs are written
    const bool ok = poll_at<4, kPipe>(2 * W, [&](int i) { return words + i; }, [&](int i, unsigned long long w) {
        if (i & 1)
            sm.S[i >> 1] = decode_word(w);
        else
            sm.K[i >> 1] = (float)decode_word(w);
    }, limit);
    for (int i = tid; i < 2 * W; i += kThreads) clear_word(words + i);
    // a first look at the decision, in flight during the draw (it is usually
    // published by now; if not, it is polled for after the draw)
    unsigned long long rw = 0ull;
    if (tid < kDecisionWords) rw = __hip_atomic_load(rec + tid, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);

    float km = 0.0f;
    double total = __builtin_nan("");
    int idx = -1;
    if (ok) {  // (uniform over the workgroup)
        // the masses S 2^(K - Kmax) of the row's chunks, their total and the
        // chunk the uniform falls in
        km = row_kmax(sm, sm.K, W);
        for (int i = tid; i < W; i += kThreads) sm.sub[i] = ldexp(sm.S[i], exp_delta(sm.K[i] - km));
        __syncthreads();
        double loc[4];
        total = mass_prefix(sm.sub, W, sm, loc);
        double t_local = 0.0;
        const int j = mass_locate(sm.sub, W, u * total, loc, sm, &t_local);
        // the row's log2-normaliser, a probe output only (an fp64 logarithm
        // is long on the step's last dependent chain)
        if (kExact && P.lognorm_out != nullptr && tid == 0)
            P.lognorm_out[(size_t)b * R + gb] = ((double)km + log2(total)) * 0.693147180559945309417;
        // a NaN logit makes the total NaN, an all -inf row makes it 0: sentinel
        if (isfinite(total) && total > 0.0 && j >= 0) {
            const Span sp = sub_chunk(j / kWaves, j % kWaves, P.chunkg, V, D::E);
            const int begin = sp.begin;
            const int n = sp.n;
            const T* rp = static_cast<const T*>(P.target) + ((size_t)b * (gamma + 1) + gb) * V + begin;
            // scan on the quarter's own scale 2^K: its largest weight is at
            // least 1/2, so a quarter with positive mass has a positive weight
            const int local = sub_chunk_find_k<D, kTargetRow, 1, false>(
                rp, rp, n, BonusWeights<kExact>::of(P, sm.K[j]), ldexp(t_local, exp_delta(km - sm.K[j])),
                sm.scratch, sm.incl, sm.iscratch, &sm.result);
            idx = (local >= 0) ? begin + local : -1;
        }
    }
    // b's decision (its copy for this workgroup, cleared once read): the
    // outputs are this workgroup's if every draft was accepted (otherwise b's
    // draw workgroup writes them), and also if the decision never arrives (a
    // timed-out wait: then they are sentinels)
    bool rok = true;
    if (__syncthreads_and(tid >= kDecisionWords || rw != 0ull)) {
        if (tid < kDecisionWords) sm.rec[tid] = ~rw;
        __syncthreads();
    } else {
        rok = wait_raw<kPipe>(rec, kDecisionWords, sm.rec, limit);
    }
    if (tid < kDecisionWords) clear_word(rec + tid);
    if (!(ok && rok) && tid == 0) set_error(P);
    const unsigned long long w0 = sm.rec[0];
    const bool draw = !rok || (((w0 >> 16) & 1) == 0 && (int)(w0 & 0xffff) == gb);
    if (!draw) return;
    const bool bad = !(ok && rok) || sticky || idx < 0;
    if (tid == 0) {
        P.accepted_len[b] = bad ? -1 : gb;
        P.next_token[b] = bad ? -1 : idx;
    }
    bonus_probes<D, kExact>(P, b, gb, km, total, bad, tid, kThreads);
}

// b's decision for a mass or draw workgroup: in the exact mode the copy
// `copy` of the decider's record; in the sigmoid mode the workgroup makes it
// itself (eq. (5) at the 2 gamma drafted-token logits needs no row
// normaliser, and the decision code is deterministic, so every workgroup of b
// reaches the same one), which spares the hand-off from the decider.
template <class D, bool kExact, bool kRagged, bool kPipe = false>
__device__ __forceinline__ Decision decision_of(const StepParams& P, int b, int copy, Smem& sm) {
    if constexpr (kExact) return read_decision<kPipe>(P, b, copy, true, sm);
    return decide<D, false, kRagged>(P, b, sm);
}

// Touches one element in each 128-byte line of rows p and q, elements
// [0, n) each (lines j0, j0 + stride, ...; up to 8 per row in flight), so
// that later loads of them hit the L2 of this workgroup's XCD.  Waits for
// the loads.
template <class T>
__device__ __forceinline__ void touch_rows(const T* p, const T* q, int n, int j0, int stride) {
    constexpr int kStep = 128 / (int)sizeof(T);
    const int nl = (n + kStep - 1) / kStep;
    float t = 0.0f;
    for (int l0 = j0; l0 < nl; l0 += 8 * stride) {
        float a[8], c[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int i = min((l0 + u * stride) * kStep, n - 1);
            a[u] = to_f32(p[i]);
            c[u] = to_f32(q[i]);
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) t += a[u] + c[u];
    }
    asm volatile("" ::"v"(t));
}

template <class D, bool kExact, bool kRagged, bool kPipe = false>
__device__ __forceinline__ void mass_role(const StepParams& P, int b, int k2, Smem& sm) {
    using T = typename D::T;
    constexpr int E = D::E;
    const int gamma = P.gamma, V = P.V;
    const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
    // short streams: each wave waits for the decision on its own (the record
    // is cleared at the end, once every wave has read it)
    constexpr bool kOwn = kPipe && kExact;
    unsigned long long* ks = P.qslot + ((size_t)b * P.nchunk2 + k2) * P.qstride;
    Decision d;
    unsigned long long* src = P.dslot + ((size_t)b * P.ncopy + k2) * kDecisionWords;
    if (kOwn && P.qstride > 0) {
        d = decide<D, true, kRagged, true>(P, b, sm, ks);
        if (!d.ok && tid == 0) set_error(P);
    } else if (kOwn) {
        unsigned long long rec[kDecisionWords];
        const bool ok = wave_wait_record(src, rec, spin_limit(P));
        d = decode_record(P, rec, ok, true);
        if (!d.ok && lane == 0) set_error(P);
    } else {
        d = decision_of<D, kExact, kRagged, kPipe>(P, b, k2, sm);
        if (!d.ok && tid == 0) set_error(P);
    }
    // b's bonus workgroup draws when every draft is accepted: nothing to do here
    const bool drawn = !d.bad && d.L == d.gb;
    if (!drawn) {
        const Span sp = sub_chunk(k2, wave, P.chunk2, V, E);
        double m = 0.0;
        if (!d.ok) {
            m = __builtin_nan("");
        } else if (!d.bad && sp.n > 0) {
            const T* rp = static_cast<const T*>(P.target) + ((size_t)b * (gamma + 1) + min(d.L, gamma)) * V + sp.begin;
            const T* rq = static_cast<const T*>(P.draft) + ((size_t)b * gamma + min(d.L, gamma - 1)) * V + sp.begin;
            float* wout = (P.weight_out != nullptr) ? P.weight_out + (size_t)b * V + sp.begin : nullptr;
            m = kExact ? wave_weight_sum<D, kPipe>(rp, rq, sp.n, d.ew, wout) : wave_weight_sum<D>(rp, rq, sp.n, d.sw, wout);
        }
        if (lane == 0) publish(P.mslot + ((size_t)b * P.nchunk2 + k2) * kWaves + wave, m);
    }
    if (kOwn && P.qstride > 0) {
        for (int i = tid; i < P.qstride; i += kThreads) clear_word(ks + i);
    } else if (kOwn) {
        __syncthreads();
        if (tid < kDecisionWords) clear_word(src + tid);
    }
}

// The inverse-CDF draw for b, by b's draw workgroup, once b's mass tiles have
// published (unless b's bonus workgroup draws); then clears b's mass words
// for the next call.
template <class D, bool kExact, bool kRagged, bool kPipe = false>
__device__ __forceinline__ void draw_role(const StepParams& P, int b, Smem& sm) {
    using T = typename D::T;
    constexpr int E = D::E;
    const int gamma = P.gamma, V = P.V;
    const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
    const int M = P.nchunk2 * kWaves;
    const bool sticky = sticky_error(P);
    Decision d = decision_of<D, kExact, kRagged, kPipe>(P, b, P.nchunk2, sm);
    // b's bonus workgroup writes the outputs when every draft is accepted
    const bool drawn = !d.bad && d.L == d.gb;
    if (!d.ok && tid == 0) set_error(P);
    if (drawn) return;
    if (kPipe && kExact && 2LL * V * (long long)sizeof(T) <= (128ll << 10))
        touch_rows(static_cast<const T*>(P.target) + ((size_t)b * (gamma + 1) + min(d.L, gamma)) * V,
                   static_cast<const T*>(P.draft) + ((size_t)b * gamma + min(d.L, gamma - 1)) * V, V, tid, kThreads);
    unsigned long long* ms = P.mslot + (size_t)b * M;
    const bool got = d.ok && wait_words<kPipe>(ms, M, sm.sub, spin_limit(P));
    if (d.ok && !got && tid == 0) set_error(P);
    const double u = (double)P.uniforms[(size_t)b * (gamma + 1) + d.gb];
    const T* rp = static_cast<const T*>(P.target) + ((size_t)b * (gamma + 1) + min(d.L, gamma)) * V;
    const T* rq = static_cast<const T*>(P.draft) + ((size_t)b * gamma + min(d.L, gamma - 1)) * V;
    float* wrow = (P.weight_out != nullptr) ? P.weight_out + (size_t)b * V : nullptr;
    const int L = d.L;
    bool bad = d.bad || !got || sticky;
    int idx = -1;
    double total = __builtin_nan("");
    for (int pass = 0; pass < 2 && !bad; ++pass) {
        // the mass the uniform falls in: one wave when there are at most 64
        double t_local = 0.0;
        int j = -1;
        if (M <= kWave) {
            if (tid < kWave) wave_locate((tid < M) ? sm.sub[tid] : 0.0, u, sm);
            __syncthreads();
            total = sm.cross_tot;
            j = sm.cross;
            t_local = sm.cross_t;
        } else if (kPipe && M <= 4 * kWave) {
            if (tid < kWave) wave_locate4(sm.sub, M, u, sm);
            __syncthreads();
            total = sm.cross_tot;
            j = sm.cross;
            t_local = sm.cross_t;
        } else {
            double loc[4];
            total = mass_prefix(sm.sub, M, sm, loc);
            if (isfinite(total) && total > 0.0) j = mass_locate(sm.sub, M, u * total, loc, sm, &t_local);
        }
        if (!(isfinite(total) && total >= 0.0)) {
            bad = true;
            break;
        }
        if (total == 0.0) {
            if (pass == 0 && L < d.gb) {
                // no residual mass (possible in sigmoid mode): draw from target row L
                d.ew.kind = kTargetRow;
                d.sw.kind = kTargetRow;
                __syncthreads();
                for (int k2 = 0; k2 < P.nchunk2; ++k2) {
                    const Span sp = sub_chunk(k2, wave, P.chunk2, V, E);
                    double m = 0.0;
                    if (sp.n > 0)
                        m = kExact ? wave_weight_sum<D, kPipe>(rp + sp.begin, rq + sp.begin, sp.n, d.ew, wrow ? wrow + sp.begin : nullptr)
                                   : wave_weight_sum<D>(rp + sp.begin, rq + sp.begin, sp.n, d.sw, wrow ? wrow + sp.begin : nullptr);
                    if (lane == 0) sm.sub[k2 * kWaves + wave] = m;
                }
                __syncthreads();
                continue;
            }
            bad = true;
            break;
        }
        if (j < 0) {
            bad = true;
            break;
        }
        const Span sp = sub_chunk(j / kWaves, j % kWaves, P.chunk2, V, E);
        int local = -1;
        if (kPipe && kExact && (sp.n + E - 1) / E <= kWave) {
            // one wave scans (the outputs are thread 0's to write; the other
            // waves go on to the clears)
            if (tid < kWave) local = wave_sub_chunk_find<D, kPipe>(rp + sp.begin, rq + sp.begin, sp.n, d.ew, t_local);
        } else {
            local = kExact ? sub_chunk_find<D, kPipe>(rp + sp.begin, rq + sp.begin, sp.n, d.ew, t_local, sm.scratch, sm.incl, sm.iscratch, &sm.result)
                           : sub_chunk_find<D>(rp + sp.begin, rq + sp.begin, sp.n, d.sw, t_local, sm.scratch, sm.incl, sm.iscratch, &sm.result);
        }
        idx = (local >= 0) ? sp.begin + local : -1;
        if (idx < 0) bad = true;
        break;
    }
    if (tid == 0) {
        P.accepted_len[b] = bad ? -1 : L;
        P.next_token[b] = bad ? -1 : idx;
        if (P.mass_out != nullptr) P.mass_out[b] = bad ? __builtin_nan("") : total;
    }
    // the draw is the only reader of b's mass words: clear them for the next call
    for (int i = tid; i < M; i += kThreads) clear_word(ms + i);
}

// ---------------------------------------------------------------------------
// Row-staged early exit (exact mode, staged_kernel).  The decision rows of
// every batch element stream in draft order, one stage per draft position c
// (target row c and draft row c of every element, then target row gamma),
// and each (b, c) has a row decider that evaluates eq. (1) at x_c as soon as
// those two rows' normalisers are in.  The first rejection at L ends b's
// decision: the rows of b's later stages are not needed by the method
// (Sec. 3.1 stops at the first rejection), so a tile of stage s >= gate
// first reads one gate word from row decider (b, s - gate) and publishes an
// empty pair instead of streaming its row when b has already rejected a
// draft.  The row decider that settles b (at the rejection, or at c =
// gamma - 1 when every draft is accepted) publishes the decision record that
// the mass, draw and bonus workgroups read, the gate words of every later
// gated stage of b and the state words of every later row decider of b,
// which then only consume their pairs; a row decider that accepts x_c
// without settling b hands "running" to row decider c + 1 and "stream" to
// the tiles of stage c + gate.  Every word still has one writer and one
// reader, which clears it.  The merges, eq. (1) and the record are those of
// the single-pass decider; the decision rows stream in chunks twice as long
// as verify_kernel's (fewer workgroups to dispatch when most rows are
// skipped), so the normalisers, and with them the outputs, can differ from
// verify_kernel's only by rounding in the last bits.
// ---------------------------------------------------------------------------
enum : unsigned long long { kStateRunning = 1, kStateSettled = 2, kGateStream = 1, kGateSkip = 2 };

__device__ __forceinline__ unsigned long long* gate_word(const StepParams& P, int b, int s, int j) {
    return P.gslot + (size_t)b * P.gstride + (size_t)s * P.gwords + j;
}
__device__ __forceinline__ unsigned long long* state_word(const StepParams& P, int b, int c) {
    return P.gslot + (size_t)b * P.gstride + (size_t)(P.gamma + 1) * P.gwords + c;
}

// Tile j of stage s of batch element b: for s < gamma the chunks of target
// row s (j < nchunk1) and draft row s, for s == gamma the short tiles of
// target row gamma.
template <class D>
__device__ __forceinline__ void staged_tile_role(const StepParams& P, int b, int s, int j, Smem& sm) {
    const int gamma = P.gamma, W = P.nchunk1;
    const int slot = (s == gamma) ? 2 * gamma : ((j < W) ? s : gamma + s);
    const int k = (s == gamma || j < W) ? j : j - W;
    if (s >= P.gate) {
        unsigned long long* gw = gate_word(P, b, s, j);
        const bool ok = wait_raw(gw, 1, sm.rec, spin_limit(P));
        if (threadIdx.x == 0) {
            clear_word(gw);
            if (!ok) set_error(P);
        }
        if (ok && sm.rec[0] == kGateSkip) {
            // b rejected a draft at least `gate` positions earlier: an empty
            // pair per quarter (target row gamma) or per tile, nothing read
            const int n = (s == gamma) ? kWaves : 1;
            const size_t first = (s == gamma) ? (size_t)slot * W + (size_t)k * kWaves : (size_t)slot * W + k;
            if ((int)threadIdx.x < n) {
                unsigned long long* out = P.pslot + (size_t)b * P.pstride + (first + threadIdx.x) * 2;
                publish(out, -INFINITY);
                publish(out + 1, 0.0);
            }
            return;
        }
    }
    stats_role<D, false>(P, b, slot, k, sm);
}

// Row decider (b, c).
template <class D>
__device__ __forceinline__ void row_decider_role(const StepParams& P, int b, int c, Smem& sm) {
    using T = typename D::T;
    const int gamma = P.gamma, V = P.V, W = P.nchunk1;
    const int tid = threadIdx.x;
    const T* draft = static_cast<const T*>(P.draft) + (size_t)b * gamma * V;
    const T* target = static_cast<const T*>(P.target) + (size_t)b * (gamma + 1) * V;

    // independent loads first: every drafted token (the decider that settles
    // b checks them all) and, in thread c, x_c's uniform and logits
    int x = 0;
    bool tok_ok = true;
    double r = 0.0;
    float zp = 0.0f, zq = 0.0f;
    if (tid < gamma) {
        x = P.tokens[(size_t)b * gamma + tid];
        tok_ok = (x >= 0 && x < V);
    }
    if (tid == c) {
        const int xs = tok_ok ? x : 0;
        r = (double)P.uniforms[(size_t)b * (gamma + 1) + c];
        zp = to_f32(target[(size_t)c * V + xs]);
        zq = to_f32(draft[(size_t)c * V + xs]);
    }

    // the pairs of target row c (slot c) and draft row c (slot gamma + c):
    // row 0 and row 1 of the merge
    unsigned long long* ps = P.pslot + (size_t)b * P.pstride;
    unsigned long long* pp = ps + (size_t)c * 2 * W;
    unsigned long long* pq = ps + (size_t)(gamma + c) * 2 * W;
    const int limit = spin_limit(P);
    bool ok = poll_at<1>(4 * W, [&](int i) { return (i < 2 * W) ? pp + i : pq + (i - 2 * W); },
                         [&](int i, unsigned long long w) {
                             if (i & 1)
                                 sm.S[i >> 1] = decode_word(w);
                             else
                                 sm.K[i >> 1] = (float)decode_word(w);
                         }, limit);
    for (int i = tid; i < 2 * W; i += kThreads) {
        clear_word(pp + i);
        clear_word(pq + i);
    }
    unsigned long long state = kStateRunning;
    bool state_ok = true;
    if (c > 0) {
        unsigned long long* sw = state_word(P, b, c);
        state_ok = wait_raw(sw, 1, sm.rec, limit);
        state = sm.rec[0];
        if (tid == 0) clear_word(sw);
    }
    if (!(ok && state_ok) && tid == 0) set_error(P);
    // Without the state of row decider c - 1 this one cannot know whether b is
    // still undecided: it publishes nothing, so that b's record keeps a single
    // writer (row decider c - 1 may still settle b; if nothing does, b's
    // readers give up and write the sentinel).  An earlier row decider that
    // settled b has its words for this one's successors out already.
    if (!state_ok || state == kStateSettled) return;

    // the two rows' log2-normalisers, with the group size of the single-pass
    // decider's 2 gamma-row merge (equal bits)
    merge_rows(sm, 2, W, 2 * gamma);
    if (tid == c) {
        const double lam_p = sm.rowL[0], lam_q = sm.rowL[1];
        const bool row_ok = isfinite(lam_p) && isfinite(lam_q);
        double tau = 1.0;  // q(x) = 0
        if (zq != -INFINITY) tau = exp2_nonpos(((double)zp - (double)zq) * (double)P.c - (lam_p - lam_q));
        sm.result = !row_ok ? 2 : ((r <= tau) ? 0 : 1);
    }
    const bool tok_bad = __syncthreads_or(!tok_ok) != 0;
    const int stop = sm.result;
    const bool settles = stop != 0 || c == gamma - 1 || !ok;
    if (!settles) {
        // x_c accepted: row decider c + 1 runs, stage c + gate streams
        if (tid == 0) publish_raw(state_word(P, b, c + 1), kStateRunning);
        const int s = c + P.gate;
        if (s <= gamma) {
            const int n = (s < gamma) ? 2 * W : P.nchunkg;
            for (int j = tid; j < n; j += kThreads) publish_raw(gate_word(P, b, s, j), kGateStream);
        }
        return;
    }
    Decision d{};
    d.ok = ok;
    d.gb = gamma;
    d.L = (stop != 0) ? c : gamma;
    d.bad = tok_bad || stop == 2 || !ok;
    if (!d.bad && d.L < gamma) {
        d.ew.kind = kResidual;
        d.ew.c = P.c;
        split3(sm.rowL[0], d.ew.kp, d.ew.lp_hi, d.ew.lp_lo);
        split3(sm.rowL[1], d.ew.kq, d.ew.lq_hi, d.ew.lq_lo);
        float dummy;
        split3(sm.rowL[0] - sm.rowL[1], d.ew.d_hi, d.ew.d_lo, dummy);
    }
    publish_decision(P, b, d);
    // the later row deciders of b only consume their pairs; the later gated
    // stages skip their rows unless every draft was accepted
    for (int i = c + 1 + tid; i < gamma; i += kThreads) publish_raw(state_word(P, b, i), kStateSettled);
    const unsigned long long g = (d.bad || d.L < gamma) ? kGateSkip : kGateStream;
    const int s0 = c + P.gate;
    if (s0 <= gamma) {
        const int nrows = (gamma - s0) * 2 * W;  // words of stages s0 .. gamma - 1, then nchunkg of stage gamma
        for (int i = tid; i < nrows + P.nchunkg; i += kThreads) {
            const int s = (i < nrows) ? s0 + i / (2 * W) : gamma;
            publish_raw(gate_word(P, b, s, (i < nrows) ? i - (s - s0) * 2 * W : i - nrows), g);
        }
    }
}

template <class D, bool kExact, bool kRagged, bool kPipe = false>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4))) void verify_kernel(StepParams P) {
    __shared__ Smem sm;
    // one argument fetch for the role split and the stats role (see Layout)
    asm volatile("" ::"s"(P.y.d0.m), "s"(P.y.d0.sh), "s"(P.y.d1.m), "s"(P.y.d1.sh), "s"(P.y.dc1.m),
                 "s"(P.y.dc1.sh), "s"(P.y.end0), "s"(P.y.end1), "s"(P.y.endg), "s"(P.y.end2), "s"(P.y.size0),
                 "s"(P.y.size1), "s"(P.y.size2), "s"(P.y.lagM), "s"(P.y.b2), "s"(P.y.S), "s"(P.y.Mt),
                 "s"(P.draft), "s"(P.target), "s"(P.pslot), "s"(P.B), "s"(P.gamma), "s"(P.V), "s"(P.chunk1),
                 "s"(P.nchunk1), "s"(P.chunkg), "s"(P.nchunkg), "s"(P.c));
    // the role split of role_at (plan.hpp), spelled out so that each branch
    // calls its role directly
    const Layout& Y = P.y;
    const unsigned int id = blockIdx.x;
    unsigned int r;
    int bs = 0, bm = 0;
    if (id < Y.end0) {
        const unsigned int k = div_of(Y.d0, id);
        r = id - k * Y.size0;
        bs = (int)k;
    } else if (id < Y.end1) {
        const unsigned int loc = id - Y.end0;
        const unsigned int k = div_of(Y.d1, loc);
        r = loc - k * Y.size1;
        bs = Y.lagM + (int)k;
        bm = (int)k;
    } else if (id < Y.endg) {
        const GTile g = g_tile(Y.dcg, Y.end1, Y.end2, P.B, P.nchunkg, (int)(id - Y.end1));
        if (kExact)
            stats_role<D, kRagged>(P, g.b, 2 * P.gamma, g.k, sm);
        else
            sigmoid_row_role<D, kRagged>(P, g.b, g.k);
        return;
    } else if (id < Y.end2) {
        const unsigned int loc = id - Y.endg;
        const unsigned int k = div_of(Y.d2, loc);
        r = loc - k * Y.size2 + (unsigned int)Y.S + 1u;
        bm = Y.b2 + (int)k;
    } else {
        bonus_role<D, kExact, kRagged, kPipe>(P, (int)(id - Y.end2), sm);
        return;
    }
    const unsigned int S = (unsigned int)Y.S;
    if (r < S) {
        const int slot = (int)div_of(Y.dc1, r);
        stats_role<D, kRagged, kPipe>(P, bs, slot, (int)r - slot * P.nchunk1, sm);
        return;
    }
    if (r == S) {
        decider_role<D, kExact, kRagged, kPipe>(P, bs, sm);
        return;
    }
    r -= S + 1u;
    if (r < (unsigned int)Y.Mt) {
        mass_role<D, kExact, kRagged, kPipe>(P, bm, (int)r, sm);
        return;
    }
    draw_role<D, kExact, kRagged, kPipe>(P, bm, sm);
}

// Exact mode with the row-staged early exit (see row_decider_role).  Index
// order: units (c, b) for c = 0 .. gamma - 1, b = 0 .. B - 1, each the
// 2 nchunk1 tiles of target row c and draft row c of b and then row decider
// (b, c - 1) (none in the units of stage 0: a row decider runs a stage behind
// its rows, so that it does not poll while they stream); the row deciders
// (b, gamma - 1); the tiles of every target row gamma; the mass tiles and the
// draw of every b; the bonus workgroups.  Every wait is on a smaller index: a
// gated tile of stage s on row decider s - gate of its element, which sits
// among the units of stage s - gate + 1 < s (gate >= 2); a row decider on its
// own rows' tiles and on row decider c - 1; the rest as in verify_kernel.
template <class D>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4))) void staged_kernel(StepParams P) {
    __shared__ Smem sm;
    const Layout& Y = P.y;
    const unsigned int id = blockIdx.x;
    if (id < Y.end0) {
        const unsigned int u = div_of(Y.d0, id);  // unit c B + b
        const unsigned int r = id - u * Y.size0;
        const unsigned int c = div_of(Y.d1, u);
        const int b = (int)(u - c * (unsigned int)P.B);
        if (r + 1u < Y.size0)
            staged_tile_role<D>(P, b, (int)c, (int)r, sm);
        else if (c > 0)
            row_decider_role<D>(P, b, (int)c - 1, sm);
    } else if (id < Y.end1) {
        row_decider_role<D>(P, (int)(id - Y.end0), P.gamma - 1, sm);
    } else if (id < Y.endg) {
        const int t = (int)(id - Y.end1);
        const int b = (int)div_of(Y.dcg, (unsigned int)t);
        staged_tile_role<D>(P, b, P.gamma, t - b * P.nchunkg, sm);
    } else if (id < Y.end2) {
        const unsigned int loc = id - Y.endg;
        const unsigned int b = div_of(Y.d2, loc);
        const unsigned int r = loc - b * Y.size2;
        if (r < (unsigned int)Y.Mt)
            mass_role<D, true, false>(P, (int)b, (int)r, sm);
        else
            draw_role<D, true, false>(P, (int)b, sm);
    } else {
        bonus_role<D, true, false>(P, (int)(id - Y.end2), sm);
    }
}

__global__ void fill_zero_kernel(uint32_t* p, size_t n) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        p[i] = 0u;
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
template <class D>
static sv_status_t launch(const Call& a, bool exact, const Plan& pl) {
    char* ws = static_cast<char*>(a.ws);
    StepParams P{};
    P.draft = a.draft;
    P.target = a.target;
    P.tokens = a.tokens;
    P.uniforms = a.uniforms;
    P.gammas = a.gammas;
    P.B = a.B;
    P.gamma = a.gamma;
    P.V = a.V;
    P.chunk1 = pl.chunk1;
    P.nchunk1 = pl.nchunk1;
    P.chunk2 = pl.chunk2;
    P.nchunk2 = pl.nchunk2;
    P.chunkg = pl.chunkg;
    P.nchunkg = pl.nchunkg;
    P.ncopy = decision_copies(exact, pl);
    P.pstride = (int)pl.pstride;
    P.qstride = (int)pl.qstride;
    P.qslot = reinterpret_cast<unsigned long long*>(ws + pl.off_qslot);
    P.y = single_pass_layout(a.B, a.gamma, a.V, a.dt, exact, pl);
    const long long n_total = (long long)P.y.end2 + a.B;
    P.temperature = (double)a.temperature;
    P.alpha = (double)a.alpha;
    P.beta = (double)a.beta;
    P.c = (float)(1.4426950408889634074 / (double)a.temperature);
    P.s = (float)(1.0 / ((double)a.temperature * ((double)a.beta - (double)a.alpha)));
    P.s0 = (float)(-(double)a.alpha / ((double)a.beta - (double)a.alpha));
    P.header = reinterpret_cast<unsigned int*>(ws);
    P.dslot = reinterpret_cast<unsigned long long*>(ws + pl.off_dslot);
    P.pslot = reinterpret_cast<unsigned long long*>(ws + pl.off_pslot);
    P.mslot = reinterpret_cast<unsigned long long*>(ws + pl.off_mslot);
    P.accepted_len = a.accepted_len;
    P.next_token = a.next_token;
    P.tau_out = a.tau_out;
    P.weight_out = a.weight_out;
    P.mass_out = a.mass_out;
    P.lognorm_out = a.lognorm_out;
    if (exact && a.staged && a.gammas == nullptr && staged_workgroups(a.B, a.gamma, a.V, a.dt, pl) > 0) {
        // the row-staged early exit (staged_kernel).  The single pass serves
        // (same results) past 2^31 workgroups and when the stream is too
        // short for any decision row to be gated (gate >= gamma): then the
        // staged order could skip nothing and only lengthens the chain of
        // decisions.
        P.gslot = reinterpret_cast<unsigned long long*>(ws + pl.off_gslot);
        P.gwords = pl.gwords;
        P.gstride = (int)pl.gstride;
        P.gate = gate_stages(a.B, a.V, bytes_per_logit(a.dt));
        P.chunk1 = pl.chunk1s;
        P.nchunk1 = pl.nchunk1s;
        P.y = make_staged_layout(a.B, a.gamma, pl.nchunk1s, pl.nchunkg, pl.nchunk2);
        const dim3 sgrid((unsigned int)((long long)P.y.end2 + a.B)), sblock(kThreads);
        hipLaunchKernelGGL((staged_kernel<D>), sgrid, sblock, 0, a.stream, P);
        return hipGetLastError() == hipSuccess ? SV_OK : SV_ERR_HIP;
    }
    const dim3 grid((unsigned int)n_total), block(kThreads);
    if (a.gammas == nullptr) {
        if (exact && pipelined_waits(a.B, a.gamma, a.V, a.dt))
            hipLaunchKernelGGL((verify_kernel<D, true, false, true>), grid, block, 0, a.stream, P);
        else if (exact)
            hipLaunchKernelGGL((verify_kernel<D, true, false>), grid, block, 0, a.stream, P);
        else
            hipLaunchKernelGGL((verify_kernel<D, false, false>), grid, block, 0, a.stream, P);
    } else {
        if (exact)
            hipLaunchKernelGGL((verify_kernel<D, true, true>), grid, block, 0, a.stream, P);
        else
            hipLaunchKernelGGL((verify_kernel<D, false, true>), grid, block, 0, a.stream, P);
    }
    return hipGetLastError() == hipSuccess ? SV_OK : SV_ERR_HIP;
}

// ---------------------------------------------------------------------------
// The static workspace of spec_verify_exact_static (for callers that cannot
// allocate): one array per GPU in the library's code object, never allocated
// or freed.  In host code `scratch` only names the symbol; its device address
// on the current device comes from hipGetSymbolAddress, looked up once per
// device (which also zero-fills it) and kept until the process ends.
// ---------------------------------------------------------------------------
static __device__ __align__(256) unsigned char scratch[SV_STATIC_WORKSPACE_BYTES];

constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mutex;
static void* g_scratch_ptr[kMaxDevices] = {};

static void launch_fill(void* p, size_t bytes, hipStream_t stream) {
    const size_t n = bytes / 4;
    const unsigned int blocks = (unsigned int)std::min<size_t>(1024, (n + 255) / 256);
    hipLaunchKernelGGL(fill_zero_kernel, dim3(blocks), dim3(256), 0, stream, static_cast<uint32_t*>(p), n);
}

// The current device's static workspace (zero-filled on `stream` the first
// time a device asks), or nullptr with *st set on a HIP error.
static void* static_workspace(hipStream_t stream, sv_status_t* st) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
        *st = SV_ERR_HIP;
        return nullptr;
    }
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (g_scratch_ptr[dev] == nullptr) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) {
            *st = SV_ERR_HIP;
            return nullptr;
        }
        launch_fill(ptr, SV_STATIC_WORKSPACE_BYTES, stream);
        if (hipGetLastError() != hipSuccess) {
            *st = SV_ERR_HIP;
            return nullptr;
        }
        g_scratch_ptr[dev] = ptr;
    }
    *st = SV_OK;
    return g_scratch_ptr[dev];
}

static sv_status_t run(const Call& a, bool exact) {
    Plan pl;
    const sv_status_t st = validate(a, exact, &pl);
    if (st != SV_OK) return st;
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

sv_status_t spec_verify_workspace_check(const void* workspace, size_t workspace_bytes, hipStream_t stream) {
    if (workspace == nullptr) return SV_ERR_NULL;
    if ((reinterpret_cast<uintptr_t>(workspace) & 15u) != 0 || workspace_bytes < sv::kHeaderBytes)
        return SV_ERR_WORKSPACE;
    uint32_t flag = 0;
    if (hipMemcpyAsync(&flag, static_cast<const char*>(workspace) + sv::kErrorFlagOffset, sizeof(flag),
                       hipMemcpyDeviceToHost, stream) != hipSuccess ||
        hipStreamSynchronize(stream) != hipSuccess)
        return SV_ERR_HIP;
    return flag != 0 ? SV_ERR_TIMEOUT : SV_OK;
}

sv_status_t spec_verify_exact(const void* draft_logits, const void* target_logits, sv_dtype_t dtype,
                              const int32_t* draft_tokens, const float* uniforms, int32_t batch, int32_t gamma,
                              int32_t vocab, float temperature, int32_t* accepted_len, int32_t* next_token,
                              void* workspace, size_t workspace_bytes, hipStream_t stream) {
    sv::Call a{draft_logits, target_logits, dtype, draft_tokens, uniforms, batch, gamma, vocab, temperature,
               0.0f, 0.0f, accepted_len, next_token, workspace, workspace_bytes, stream,
               nullptr, nullptr, nullptr, nullptr, nullptr};
    return sv::run(a, true);
}

sv_status_t spec_verify_exact_static(const void* draft_logits, const void* target_logits, sv_dtype_t dtype,
                                     const int32_t* draft_tokens, const float* uniforms, int32_t batch,
                                     int32_t gamma, int32_t vocab, float temperature, int32_t* accepted_len,
                                     int32_t* next_token, int32_t reset, hipStream_t stream) {
    // the arguments first, against a stand-in workspace of the static size
    // (only its size and alignment are checked)
    sv::Call a{draft_logits, target_logits, dtype, draft_tokens, uniforms, batch, gamma, vocab, temperature,
               0.0f, 0.0f, accepted_len, next_token, reinterpret_cast<void*>(uintptr_t{256}),
               SV_STATIC_WORKSPACE_BYTES, stream, nullptr, nullptr, nullptr, nullptr, nullptr};
    sv::Plan pl;
    const sv_status_t valid = sv::validate(a, true, &pl);
    if (valid != SV_OK) return valid;
    sv_status_t st = SV_OK;
    a.ws = sv::static_workspace(stream, &st);
    if (a.ws == nullptr) return st;
    if (reset != 0) {
        sv::launch_fill(a.ws, pl.bytes, stream);
        if (hipGetLastError() != hipSuccess) return SV_ERR_HIP;
    }
    return sv::run(a, true);
}

sv_status_t spec_verify_exact_early_exit(const void* draft_logits, const void* target_logits, sv_dtype_t dtype,
                                         const int32_t* draft_tokens, const float* uniforms, int32_t batch,
                                         int32_t gamma, int32_t vocab, float temperature, int32_t* accepted_len,
                                         int32_t* next_token, void* workspace, size_t workspace_bytes,
                                         hipStream_t stream) {
    sv::Call a{draft_logits, target_logits, dtype, draft_tokens, uniforms, batch, gamma, vocab, temperature,
               0.0f, 0.0f, accepted_len, next_token, workspace, workspace_bytes, stream,
               nullptr, nullptr, nullptr, nullptr, nullptr, true};
    return sv::run(a, true);
}

sv_status_t spec_verify_sigmoid(const void* draft_logits, const void* target_logits, sv_dtype_t dtype,
                                const int32_t* draft_tokens, const float* uniforms, int32_t batch, int32_t gamma,
                                int32_t vocab, float temperature, float alpha, float beta, int32_t* accepted_len,
                                int32_t* next_token, void* workspace, size_t workspace_bytes, hipStream_t stream) {
    sv::Call a{draft_logits, target_logits, dtype, draft_tokens, uniforms, batch, gamma, vocab, temperature,
               alpha, beta, accepted_len, next_token, workspace, workspace_bytes, stream,
               nullptr, nullptr, nullptr, nullptr, nullptr};
    return sv::run(a, false);
}

sv_status_t spec_verify_exact_probe(const void* draft_logits, const void* target_logits, sv_dtype_t dtype,
                                    const int32_t* draft_tokens, const float* uniforms, int32_t batch, int32_t gamma,
                                    int32_t vocab, float temperature, int32_t* accepted_len, int32_t* next_token,
                                    void* workspace, size_t workspace_bytes, hipStream_t stream, double* tau_out,
                                    float* weight_out, double* mass_out, double* lognorm_out) {
    sv::Call a{draft_logits, target_logits, dtype, draft_tokens, uniforms, batch, gamma, vocab, temperature,
               0.0f, 0.0f, accepted_len, next_token, workspace, workspace_bytes, stream,
               tau_out, weight_out, mass_out, lognorm_out, nullptr};
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
               tau_out, weight_out, mass_out, nullptr, nullptr};
    return sv::run(a, false);
}

sv_status_t spec_verify_exact_ragged(const void* draft_logits, const void* target_logits, sv_dtype_t dtype,
                                     const int32_t* draft_tokens, const float* uniforms, const int32_t* gammas,
                                     int32_t batch, int32_t gamma_max, int32_t vocab, float temperature,
                                     int32_t* accepted_len, int32_t* next_token, void* workspace,
                                     size_t workspace_bytes, hipStream_t stream) {
    if (gammas == nullptr) return SV_ERR_NULL;
    sv::Call a{draft_logits, target_logits, dtype, draft_tokens, uniforms, batch, gamma_max, vocab, temperature,
               0.0f, 0.0f, accepted_len, next_token, workspace, workspace_bytes, stream,
               nullptr, nullptr, nullptr, nullptr, gammas};
    return sv::run(a, true);
}

sv_status_t spec_verify_sigmoid_ragged(const void* draft_logits, const void* target_logits, sv_dtype_t dtype,
                                       const int32_t* draft_tokens, const float* uniforms, const int32_t* gammas,
                                       int32_t batch, int32_t gamma_max, int32_t vocab, float temperature,
                                       float alpha, float beta, int32_t* accepted_len, int32_t* next_token,
                                       void* workspace, size_t workspace_bytes, hipStream_t stream) {
    if (gammas == nullptr) return SV_ERR_NULL;
    sv::Call a{draft_logits, target_logits, dtype, draft_tokens, uniforms, batch, gamma_max, vocab, temperature,
               alpha, beta, accepted_len, next_token, workspace, workspace_bytes, stream,
               nullptr, nullptr, nullptr, nullptr, gammas};
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
        case SV_ERR_ALLOC: return "host allocation failed";
        case SV_ERR_TIMEOUT: return "a wait between workgroups timed out; re-initialise the workspace";
    }
    return "unknown status";
}

}  // extern "C"
