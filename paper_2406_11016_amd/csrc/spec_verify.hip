// Fused speculative-sampling verification for gfx950 (MI355X): kernels and C ABI.
//
// Method: arXiv 2406.11016, Sec. 3.1 (eqs. (1)-(3)) and Sec. 3.2.2 (eqs. (4)-(5)).
//
// Exact mode, three launches on the caller's stream:
//   row_stats_kernel  grid = B * (2*gamma+1) * nchunk1 workgroups.  Each
//                     streams one chunk of one logit row exactly once with
//                     128-bit loads and writes that chunk's contribution to
//                     the row's softmax normaliser (eq. (4)).  This kernel
//                     moves every logit byte and bounds the step.
//   mass_kernel       grid = B * nchunk2.  Every workgroup of batch element b
//                     merges b's chunk normalisers in a fixed order, evaluates
//                     tau_c (eq. (1)) at the drafted tokens and runs the
//                     first-rejection scan, so all of them agree on L without
//                     communicating; each then sums the weights a(x) of the
//                     final distribution (residual of eqs. (2)-(3), or target
//                     row gamma) over its chunk of the selected row(s).
//   draw_kernel       grid = B.  Fixed-order prefix over b's chunk masses,
//                     then a workgroup scan inside the chunk the uniform falls
//                     in: the inverse-CDF draw of the next token.
// Sigmoid mode: mass_kernel and draw_kernel only; the element-wise
// approximation of eq. (5) needs no row normaliser, so only the logits at the
// drafted tokens and the row(s) the next token is drawn from are read.
#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <cmath>

#include "spec_verify.h"
#include "sv_device.hpp"

namespace sv {

enum : int { kResidual = 0, kTargetRow = 1 };

constexpr int kScanVec = 4;              // contiguous vectors per thread in the in-chunk scan
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

constexpr int kPassUnroll = 4;  // vectors per thread per round in the weight pass

// Sum of the weights over one chunk (rp/rq point at the chunk start, n
// elements); optionally stores every weight.  Valid in every thread.
template <class D, int KIND, class W>
__device__ __forceinline__ double chunk_weight_sum_k(const typename D::T* rp, const typename D::T* rq, int n,
                                                     const W& w, float* wout, double* scratch) {
    constexpr int E = D::E;
    constexpr bool two_rows = (KIND == kResidual);
    const int nvec = (n + E - 1) / E;
    const bool fast = pair_aligned<D>(rp, rq, two_rows);
    double acc = 0.0;
    for (int v0 = 0; v0 < nvec; v0 += kPassUnroll * kThreads) {
        float zp[kPassUnroll][E], zq[kPassUnroll][E];
        load_pair_u<D, kPassUnroll>(rp, rq, two_rows, fast, v0 + (int)threadIdx.x, kThreads, n, zp, zq);
#pragma unroll
        for (int u = 0; u < kPassUnroll; ++u) {
            const int v = v0 + u * kThreads + (int)threadIdx.x;
            if (v >= nvec) continue;
#pragma unroll
            for (int e = 0; e < E; ++e) {
                const float a = w.template eval<KIND>(zp[u][e], zq[u][e]);
                if (wout != nullptr && v * E + e < n) wout[v * E + e] = a;
                acc += (double)a;
            }
        }
    }
    return block_sum(acc, scratch);
}

template <class D, class W>
__device__ double chunk_weight_sum(const typename D::T* rp, const typename D::T* rq, int n, const W& w,
                                   float* wout, double* scratch) {
    return (w.kind == kTargetRow) ? chunk_weight_sum_k<D, kTargetRow>(rp, rq, n, w, wout, scratch)
                                  : chunk_weight_sum_k<D, kResidual>(rp, rq, n, w, wout, scratch);
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

// Index (relative to the chunk start) of the first element whose running
// weight sum exceeds t, or of the last positive weight if rounding leaves the
// chunk total at or below t.  Valid in every thread.  Thread i owns the
// contiguous vectors [i * kScanVec, (i + 1) * kScanVec), so one workgroup scan
// of the per-thread sums follows element order.  Needs n <= kScanVec * kThreads * E.
template <class D, int KIND, class W>
__device__ __forceinline__ int chunk_find_k(const typename D::T* rp, const typename D::T* rq, int n, const W& w,
                                            double t, double* scratch, double* incl_s /* [kThreads] */,
                                            int* iscratch) {
    constexpr int E = D::E;
    constexpr bool two_rows = (KIND == kResidual);
    constexpr int U = kScanVec;
    __shared__ int result;
    const int tid = threadIdx.x;
    const bool fast = pair_aligned<D>(rp, rq, two_rows);
    float a[U][E];
    double sum = 0.0;
    {
        float zp[U][E], zq[U][E];
        load_pair_u<D, U>(rp, rq, two_rows, fast, tid * U, 1, n, zp, zq);
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int e = 0; e < E; ++e) {
                a[u][e] = w.template eval<KIND>(zp[u][e], zq[u][e]);
                sum += (double)a[u][e];
            }
    }
    if (tid == 0) result = -1;
    double tot;
    const double incl = block_inclusive_scan(sum, scratch, &tot);
    incl_s[tid] = incl;
    const int first = block_first(incl > t, iscratch);
    if (first < kThreads) {
        if (tid == first) {
            double cum = (first == 0) ? 0.0 : incl_s[first - 1];
            int idx = -1, lastp = -1;
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int e = 0; e < E; ++e) {
                    if (a[u][e] > 0.0f) lastp = u * E + e;
                    cum += (double)a[u][e];
                    if (idx < 0 && cum > t && a[u][e] > 0.0f) idx = u * E + e;
                }
            if (idx < 0) idx = lastp;
            result = (idx >= 0) ? tid * U * E + idx : -1;
        }
    } else {
        // t lies at or beyond the chunk total (rounding only): the last positive weight
        int lastp = -1;
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int e = 0; e < E; ++e)
                if (a[u][e] > 0.0f) lastp = tid * U * E + u * E + e;
        const int lv = wave_max_int(lastp);
        if ((tid % kWave) == 0) iscratch[tid / kWave] = lv;
        __syncthreads();
        if (tid == 0) {
            int best = -1;
            for (int i = 0; i < kWaves; ++i) best = max(best, iscratch[i]);
            result = best;
        }
    }
    __syncthreads();
    return result;
}

template <class D, class W>
__device__ int chunk_find(const typename D::T* rp, const typename D::T* rq, int n, const W& w, double t,
                          double* scratch, double* incl_s, int* iscratch) {
    return (w.kind == kTargetRow) ? chunk_find_k<D, kTargetRow>(rp, rq, n, w, t, scratch, incl_s, iscratch)
                                  : chunk_find_k<D, kResidual>(rp, rq, n, w, t, scratch, incl_s, iscratch);
}

// ---------------------------------------------------------------------------
// exact mode, pass 1: per-chunk row normalisers
// ---------------------------------------------------------------------------
template <class D>
__global__ __launch_bounds__(kThreads) void row_stats_kernel(const typename D::T* __restrict__ draft,
                                                             const typename D::T* __restrict__ target, int gamma,
                                                             int V, int chunk, int nchunk, float c,
                                                             RowPartial* __restrict__ partial) {
    using T = typename D::T;
    constexpr int E = D::E;
    __shared__ float sk[kWaves];
    __shared__ double ss[kWaves];

    const int R = 2 * gamma + 1;
    const int tile = blockIdx.x;
    const int k = tile % nchunk;
    const int rowid = tile / nchunk;  // b * R + r
    const int b = rowid / R;
    const int r = rowid - b * R;
    const T* row = (r <= gamma) ? target + ((size_t)b * (gamma + 1) + r) * (size_t)V
                                : draft + ((size_t)b * gamma + (r - gamma - 1)) * (size_t)V;
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
    const Lse blk = block_lse(st, sk, ss);
    if (threadIdx.x == 0) partial[tile] = RowPartial{blk.s, blk.k, 0.0f};
}

// ---------------------------------------------------------------------------
// pass 2 (both modes): the decision and the final-distribution chunk masses
// pass 3 (both modes): the inverse-CDF draw
//
// Workgroups never wait on each other inside a kernel: on this multi-XCD part
// every device-scope release/acquire is an L2 writeback/invalidate, which
// costs far more than a kernel boundary.  Every pass-2 workgroup of a batch
// element therefore recomputes the (cheap) decision itself, and the draw is
// a separate launch.
// ---------------------------------------------------------------------------
struct SelectParams {
    const void* draft;
    const void* target;
    const int32_t* tokens;
    const float* uniforms;
    int B, gamma, V;
    int nchunk1;               // exact: chunks per row in `partial`
    int chunk2, nchunk2;       // chunking of the final-distribution pass
    float c;                   // exact: log2(e) / T
    float s, s0;               // sigmoid: u = fma(z, s, s0)
    double temperature, alpha, beta;
    const RowPartial* partial;
    double* chunk_mass;        // [B, nchunk2]
    struct Selection* sel;     // [B]
    int32_t* accepted_len;
    int32_t* next_token;
    double* tau_out;           // optional probes
    float* weight_out;
    double* mass_out;
    double* lognorm_out;
};

// The decision for one batch element, as pass 3 needs it.
struct Selection {
    int L;      // accepted length, in [0, gamma]
    int bad;    // 1: sentinel
    ExactWeights ew;
    SigmoidWeights sw;
};

constexpr int kMergeCap = 1024;  // row-normaliser partials staged in LDS at once

__device__ __forceinline__ double min1(double r) { return (r >= 1.0) ? 1.0 : r; }  // keeps NaN

template <class D, bool kExact>
__global__ __launch_bounds__(kThreads) void mass_kernel(SelectParams P) {
    using T = typename D::T;
    __shared__ float rowK[kExact ? kMaxRows : 1];
    __shared__ double rowS[kExact ? kMaxRows : 1];
    __shared__ float pk[kExact ? kMergeCap : 1];
    __shared__ double ps[kExact ? kMergeCap : 1];
    __shared__ double tau_s[kMaxGamma];
    __shared__ int stop_s[kMaxGamma];
    __shared__ double scratch[kWaves];
    __shared__ int sel_L, sel_bad, tok_bad;

    const int gamma = P.gamma, V = P.V, R = 2 * gamma + 1;
    const int b = blockIdx.x / P.nchunk2;
    const int k2 = blockIdx.x - b * P.nchunk2;
    const T* draft = static_cast<const T*>(P.draft) + (size_t)b * gamma * V;
    const T* target = static_cast<const T*>(P.target) + (size_t)b * (gamma + 1) * V;
    const int tid = threadIdx.x;

    // independent loads first: tokens and uniforms, then the drafted-token
    // logits (their latency overlaps the normaliser merge below)
    int x = 0;
    double r = 0.0;
    bool tok_ok = true;
    float zp = 0.0f, zq = 0.0f;
    if (tid == 0) tok_bad = 0;
    if (tid < gamma) {
        x = P.tokens[(size_t)b * gamma + tid];
        r = (double)P.uniforms[(size_t)b * (gamma + 1) + tid];
        tok_ok = (x >= 0 && x < V);
        const int xs = tok_ok ? x : 0;
        zp = to_f32(target[(size_t)tid * V + xs]);
        zq = to_f32(draft[(size_t)tid * V + xs]);
    }

    // row normalisers of b: partials staged in LDS by groups of rows, each row
    // merged sequentially in chunk order (identical in every workgroup of b,
    // and identical for draft and target rows with equal values)
    if (kExact) {
        const int nc1 = P.nchunk1;
        const RowPartial* pb = P.partial + (size_t)b * R * nc1;
        const int G = max(1, kMergeCap / nc1);
        for (int r0 = 0; r0 < R; r0 += G) {
            const int r1 = min(R, r0 + G);
            const int np = (r1 - r0) * nc1;
            __syncthreads();
            for (int i = tid; i < np; i += kThreads) {
                const RowPartial q = pb[(size_t)r0 * nc1 + i];
                pk[i] = q.k;
                ps[i] = q.s;
            }
            __syncthreads();
            if (tid < r1 - r0) {
                Lse st{-INFINITY, 0.0};
                for (int k = 0; k < nc1; ++k) st = lse_merge(st, Lse{pk[tid * nc1 + k], ps[tid * nc1 + k]});
                rowK[r0 + tid] = st.k;
                rowS[r0 + tid] = st.s;
            }
        }
    }
    __syncthreads();

    // eq. (1) at the drafted tokens
    if (tid < gamma) {
        if (!tok_ok) tok_bad = 1;
        double tau;
        bool row_ok;
        if (kExact) {
            const double lam_p = (double)rowK[tid] + log2(rowS[tid]);
            const double lam_q = (double)rowK[gamma + 1 + tid] + log2(rowS[gamma + 1 + tid]);
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
        tau_s[tid] = tau;
        stop_s[tid] = !row_ok ? 2 : ((r <= tau) ? 0 : 1);
    }
    __syncthreads();
    if (tid == 0) {
        int L = gamma, bad = tok_bad;
        for (int c = 0; c < gamma; ++c) {
            if (stop_s[c] != 0) {
                L = c;
                if (stop_s[c] == 2) bad = 1;
                break;
            }
        }
        if (kExact && !bad && L == gamma) {
            const double lam = (double)rowK[gamma] + log2(rowS[gamma]);
            if (!isfinite(lam)) bad = 1;
        }
        sel_L = L;
        sel_bad = bad;
    }
    __syncthreads();
    const int L = sel_L;
    const bool bad = sel_bad != 0;
    const bool two_rows = L < gamma;

    ExactWeights ew{};
    SigmoidWeights sw{};
    if (kExact && !bad) {
        const int rpi = min(L, gamma), rqi = gamma + 1 + min(L, gamma - 1);
        const double lp = log2(rowS[rpi]), lq = log2(rowS[rqi]);
        const double dl = ((double)rowK[rpi] + lp) - ((double)rowK[rqi] + lq);
        ew.kind = two_rows ? kResidual : kTargetRow;
        ew.c = P.c;
        ew.kp = rowK[rpi];
        ew.lp_hi = (float)lp;
        ew.lp_lo = (float)(lp - (double)ew.lp_hi);
        ew.kq = rowK[rqi];
        ew.lq_hi = (float)lq;
        ew.lq_lo = (float)(lq - (double)ew.lq_hi);
        ew.d_hi = (float)dl;
        ew.d_lo = (float)(dl - (double)ew.d_hi);
    }
    if (!kExact) {
        sw.kind = two_rows ? kResidual : kTargetRow;
        sw.s = P.s;
        sw.s0 = P.s0;
    }

    if (k2 == 0) {
        if (tid == 0) {
            Selection sel;
            sel.L = L;
            sel.bad = bad ? 1 : 0;
            sel.ew = ew;
            sel.sw = sw;
            P.sel[b] = sel;
        }
        if (P.tau_out != nullptr && tid < gamma) P.tau_out[(size_t)b * gamma + tid] = tau_s[tid];
        if (kExact && P.lognorm_out != nullptr)
            for (int i = tid; i < R; i += kThreads)
                P.lognorm_out[(size_t)b * R + i] = ((double)rowK[i] + log2(rowS[i])) * 0.693147180559945309417;
    }

    // this workgroup's chunk of the final distribution
    const T* rp = target + (size_t)min(L, gamma) * V;
    const T* rq = draft + (size_t)min(L, gamma - 1) * V;
    const int begin = k2 * P.chunk2;
    const int n = min(V, begin + P.chunk2) - begin;
    float* wrow = (P.weight_out != nullptr) ? P.weight_out + (size_t)b * V + begin : nullptr;
    double m = 0.0;
    if (!bad) {
        if (kExact)
            m = chunk_weight_sum<D>(rp + begin, rq + begin, n, ew, wrow, scratch);
        else
            m = chunk_weight_sum<D>(rp + begin, rq + begin, n, sw, wrow, scratch);
    }
    if (tid == 0) P.chunk_mass[(size_t)b * P.nchunk2 + k2] = m;
}

constexpr int kMaxChunks2 = 1024;

template <class D, bool kExact>
__global__ __launch_bounds__(kThreads) void draw_kernel(SelectParams P) {
    using T = typename D::T;
    __shared__ double cm[kMaxChunks2];
    __shared__ double scratch[kWaves];
    __shared__ double incl_s[kThreads];
    __shared__ int iscratch[kWaves];
    __shared__ int fin_chunk;
    __shared__ double fin_total, fin_t;

    const int gamma = P.gamma, V = P.V;
    const int b = blockIdx.x;
    const int tid = threadIdx.x;
    const Selection sel = P.sel[b];
    for (int k = tid; k < P.nchunk2; k += kThreads) cm[k] = P.chunk_mass[(size_t)b * P.nchunk2 + k];
    const double u = (double)P.uniforms[(size_t)b * (gamma + 1) + gamma];
    if (sel.bad) {
        if (tid == 0) {
            P.accepted_len[b] = -1;
            P.next_token[b] = -1;
            if (P.mass_out != nullptr) P.mass_out[b] = __builtin_nan("");
        }
        return;
    }
    const int L = sel.L;
    const T* target = static_cast<const T*>(P.target) + (size_t)b * (gamma + 1) * V;
    const T* draft = static_cast<const T*>(P.draft) + (size_t)b * gamma * V;
    const T* rp = target + (size_t)min(L, gamma) * V;
    const T* rq = draft + (size_t)min(L, gamma - 1) * V;
    ExactWeights ew = sel.ew;
    SigmoidWeights sw = sel.sw;
    bool two_rows = L < gamma;
    float* wrow = (P.weight_out != nullptr) ? P.weight_out + (size_t)b * V : nullptr;

    __syncthreads();
    if (tid == 0) {
        double tot = 0.0;
        for (int k = 0; k < P.nchunk2; ++k) tot += cm[k];
        fin_total = tot;
    }
    __syncthreads();
    if (two_rows && fin_total == 0.0) {
        // no residual mass (possible in sigmoid mode): draw from target row L
        two_rows = false;
        ew.kind = kTargetRow;
        sw.kind = kTargetRow;
        for (int k = 0; k < P.nchunk2; ++k) {
            const int bk = k * P.chunk2;
            const int nk = min(V, bk + P.chunk2) - bk;
            const double mk = kExact ? chunk_weight_sum<D>(rp + bk, rq + bk, nk, ew, wrow ? wrow + bk : nullptr, scratch)
                                     : chunk_weight_sum<D>(rp + bk, rq + bk, nk, sw, wrow ? wrow + bk : nullptr, scratch);
            if (tid == 0) cm[k] = mk;
        }
        __syncthreads();
        if (tid == 0) {
            double tot = 0.0;
            for (int k = 0; k < P.nchunk2; ++k) tot += cm[k];
            fin_total = tot;
        }
        __syncthreads();
    }
    const double total = fin_total;
    if (!(isfinite(total) && total > 0.0)) {
        if (tid == 0) {
            P.accepted_len[b] = -1;
            P.next_token[b] = -1;
            if (P.mass_out != nullptr) P.mass_out[b] = total;
        }
        return;
    }
    if (tid == 0) {
        const double t = u * total;
        double cum = 0.0;
        int j = -1, lastpos = 0;
        for (int k = 0; k < P.nchunk2; ++k) {
            if (cm[k] > 0.0) lastpos = k;
            if (cum + cm[k] > t) {
                j = k;
                break;
            }
            cum += cm[k];
        }
        if (j < 0) j = lastpos;  // rounding only
        fin_chunk = j;
        fin_t = t - cum;
    }
    __syncthreads();
    const int j = fin_chunk;
    const int bj = j * P.chunk2;
    const int nj = min(V, bj + P.chunk2) - bj;
    const int idx = kExact ? chunk_find<D>(rp + bj, rq + bj, nj, ew, fin_t, scratch, incl_s, iscratch)
                           : chunk_find<D>(rp + bj, rq + bj, nj, sw, fin_t, scratch, incl_s, iscratch);
    if (tid == 0) {
        P.accepted_len[b] = (idx >= 0) ? L : -1;
        P.next_token[b] = (idx >= 0) ? bj + idx : -1;
        if (P.mass_out != nullptr) P.mass_out[b] = total;
    }
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
    size_t off_partial, off_mass, off_sel, bytes;
};

static inline long long ceil_div(long long a, long long b) { return (a + b - 1) / b; }
static inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

static bool valid_dtype(sv_dtype_t dt) { return dt == SV_F32 || dt == SV_F16 || dt == SV_BF16; }

static bool make_plan(int32_t B, int32_t gamma, int32_t V, sv_dtype_t dt, Plan* p) {
    if (B < 1 || gamma < 1 || gamma > kMaxGamma || V < 1 || !valid_dtype(dt)) return false;
    const int E = (dt == SV_F32) ? 4 : 8;
    const int s = (dt == SV_F32) ? 4 : 2;
    const long long R = 2LL * gamma + 1;
    // every row offset is computed in size_t; chunk indices are int
    if ((long long)B * (gamma + 1) * (long long)V > (1LL << 40)) return false;
    const long long min_elems = (long long)kThreads * E;
    const long long max_cells = std::max<long long>(1, ceil_div(V, min_elems));

    long long nc = ceil_div(kWantStatsTiles, B * R);
    nc = std::max(nc, ceil_div(V, kStatsTileBytes / s));
    nc = std::min(nc, max_cells);
    long long chunk = ceil_div(ceil_div(V, nc), E) * E;
    p->chunk1 = (int)chunk;
    p->nchunk1 = (int)ceil_div(V, chunk);
    if ((long long)B * R * p->nchunk1 > 0x7fffffffLL) return false;

    const long long max_scan = (long long)kScanVec * kThreads * E;  // in-chunk scan capacity
    long long nc2 = ceil_div(kWantSampleTiles, B);
    nc2 = std::max(nc2, ceil_div(V, kSampleTileBytes / s));
    nc2 = std::min(nc2, max_cells);
    nc2 = std::max(nc2, ceil_div(V, max_scan));
    long long chunk2 = ceil_div(ceil_div(V, nc2), E) * E;
    p->chunk2 = (int)chunk2;
    p->nchunk2 = (int)ceil_div(V, chunk2);
    if ((long long)B * p->nchunk2 > 0x7fffffffLL) return false;
    p->E = E;

    if (p->nchunk2 > kMaxChunks2) return false;
    size_t off = 0;
    p->off_sel = off;
    off = align256(off + sizeof(Selection) * (size_t)B);
    p->off_mass = off;
    off = align256(off + sizeof(double) * (size_t)B * p->nchunk2);
    p->off_partial = off;
    off = align256(off + sizeof(RowPartial) * (size_t)B * R * p->nchunk1);
    p->bytes = off;
    return true;
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
    using T = typename D::T;
    const T* draft = static_cast<const T*>(a.draft);
    const T* target = static_cast<const T*>(a.target);
    char* ws = static_cast<char*>(a.ws);
    RowPartial* partial = reinterpret_cast<RowPartial*>(ws + pl.off_partial);

    SelectParams P{};
    P.draft = a.draft;
    P.target = a.target;
    P.tokens = a.tokens;
    P.uniforms = a.uniforms;
    P.B = a.B;
    P.gamma = a.gamma;
    P.V = a.V;
    P.nchunk1 = pl.nchunk1;
    P.chunk2 = pl.chunk2;
    P.nchunk2 = pl.nchunk2;
    P.temperature = (double)a.temperature;
    P.alpha = (double)a.alpha;
    P.beta = (double)a.beta;
    P.c = (float)(1.4426950408889634074 / (double)a.temperature);
    P.s = (float)(1.0 / ((double)a.temperature * ((double)a.beta - (double)a.alpha)));
    P.s0 = (float)(-(double)a.alpha / ((double)a.beta - (double)a.alpha));
    P.partial = partial;
    P.chunk_mass = reinterpret_cast<double*>(ws + pl.off_mass);
    P.sel = reinterpret_cast<Selection*>(ws + pl.off_sel);
    P.accepted_len = a.accepted_len;
    P.next_token = a.next_token;
    P.tau_out = a.tau_out;
    P.weight_out = a.weight_out;
    P.mass_out = a.mass_out;
    P.lognorm_out = a.lognorm_out;

    if (exact) {
        const int tiles = a.B * (2 * a.gamma + 1) * pl.nchunk1;
        hipLaunchKernelGGL(row_stats_kernel<D>, dim3(tiles), dim3(kThreads), 0, a.stream, draft, target, a.gamma,
                           a.V, pl.chunk1, pl.nchunk1, P.c, partial);
        hipLaunchKernelGGL((mass_kernel<D, true>), dim3(a.B * pl.nchunk2), dim3(kThreads), 0, a.stream, P);
        hipLaunchKernelGGL((draw_kernel<D, true>), dim3(a.B), dim3(kThreads), 0, a.stream, P);
    } else {
        hipLaunchKernelGGL((mass_kernel<D, false>), dim3(a.B * pl.nchunk2), dim3(kThreads), 0, a.stream, P);
        hipLaunchKernelGGL((draw_kernel<D, false>), dim3(a.B), dim3(kThreads), 0, a.stream, P);
    }
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
