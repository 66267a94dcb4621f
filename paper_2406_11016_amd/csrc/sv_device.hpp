// Device primitives of the verification kernels (gfx950, wave64).
//
// Storage-type traits and 128-bit row loaders, the one-pass row normaliser
// (running power-of-two reference plus fp64 sum), and deterministic wave64 /
// workgroup reductions and scans.  Every reduction here has a fixed
// combination order, so a row's result depends only on its values and the
// chunk geometry -- never on the row's address, the launch order or timing.
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "plan.hpp"

namespace sv {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
// 16 bytes at a 4-byte aligned address: still one global_load_dwordx4, so
// rows whose start is only 4-byte aligned (fp32 rows of odd length, 16-bit
// rows of even length) stream as fast as 16-byte aligned ones
typedef unsigned int u32x4_a4 __attribute__((ext_vector_type(4), aligned(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

// ---------------------------------------------------------------------------
// storage types: E elements per 16-byte vector
// ---------------------------------------------------------------------------
struct F32 {
    using T = float;
    static constexpr int E = 4;
};
struct F16 {
    using T = _Float16;
    static constexpr int E = 8;
};
struct BF16 {
    using T = uint16_t;  // raw bfloat16 bits
    static constexpr int E = 8;
};

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(_Float16 v) { return (float)v; }
__device__ __forceinline__ float to_f32(uint16_t v) { return __uint_as_float((uint32_t)v << 16); }

template <class D>
__device__ __forceinline__ void unpack(const u32x4 r, float (&x)[D::E]);

template <>
__device__ __forceinline__ void unpack<F32>(const u32x4 r, float (&x)[4]) {
    x[0] = __uint_as_float(r.x);
    x[1] = __uint_as_float(r.y);
    x[2] = __uint_as_float(r.z);
    x[3] = __uint_as_float(r.w);
}

template <>
__device__ __forceinline__ void unpack<BF16>(const u32x4 r, float (&x)[8]) {
    // bf16 is the upper half of a binary32: shift the low half up, mask the high half.
    x[0] = __uint_as_float(r.x << 16);
    x[1] = __uint_as_float(r.x & 0xffff0000u);
    x[2] = __uint_as_float(r.y << 16);
    x[3] = __uint_as_float(r.y & 0xffff0000u);
    x[4] = __uint_as_float(r.z << 16);
    x[5] = __uint_as_float(r.z & 0xffff0000u);
    x[6] = __uint_as_float(r.w << 16);
    x[7] = __uint_as_float(r.w & 0xffff0000u);
}

template <>
__device__ __forceinline__ void unpack<F16>(const u32x4 r, float (&x)[8]) {
    const f16x8 h = __builtin_bit_cast(f16x8, r);
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] = (float)h[e];
}

// Whether 16-byte vector loads may start at p (any 4-byte aligned address).
__device__ __forceinline__ bool vec_loadable(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

// A 16-byte vector whose every element is -inf in storage type D.
template <class D>
__device__ __forceinline__ u32x4 neg_inf_vec();
template <>
__device__ __forceinline__ u32x4 neg_inf_vec<F32>() { return u32x4{0xff800000u, 0xff800000u, 0xff800000u, 0xff800000u}; }
template <>
__device__ __forceinline__ u32x4 neg_inf_vec<F16>() { return u32x4{0xfc00fc00u, 0xfc00fc00u, 0xfc00fc00u, 0xfc00fc00u}; }
template <>
__device__ __forceinline__ u32x4 neg_inf_vec<BF16>() { return u32x4{0xff80ff80u, 0xff80ff80u, 0xff80ff80u, 0xff80ff80u}; }

// Vector v (elements v E .. v E + E - 1) of a chunk starting at a 4-byte
// aligned address and holding nfull (>= 1) whole vectors, or the -inf vector
// when v >= nfull.  The load is unconditional (its index is clamped into
// range) so that a block of such loads is issued back to back.  The element
// assignment does not depend on the chunk's address, so equal rows give
// equal bits wherever they are.
template <class D, bool NT>
__device__ __forceinline__ u32x4 load_vec_or_pad(const typename D::T* base, int v, int nfull) {
    const u32x4_a4* p = reinterpret_cast<const u32x4_a4*>(base + (size_t)min(v, nfull - 1) * D::E);
    const u32x4 r = NT ? __builtin_nontemporal_load(p) : *p;
    return (v < nfull) ? r : neg_inf_vec<D>();
}

// Elements i..i+E-1 of a chunk of n (>= 1) elements with element-wise loads
// (any alignment); indices at or beyond n read as -inf.  Loads are
// unconditional (clamped indices), so they issue back to back.
template <class D>
__device__ __forceinline__ void load_elems_or_pad(const typename D::T* base, int i, int n, float (&x)[D::E]) {
#pragma unroll
    for (int e = 0; e < D::E; ++e) {
        const float val = to_f32(base[min(i + e, n - 1)]);
        x[e] = (i + e < n) ? val : -INFINITY;
    }
}

// ---------------------------------------------------------------------------
// wave64 / workgroup reductions (every lane ends with the same bits)
//
// Within each 16-lane row a butterfly of DPP lane permutations (swap
// neighbours, swap pairs, mirror halves, mirror the row) leaves every lane
// with the row's value; the four row values are then combined in a fixed
// order from lanes 0, 16, 32 and 48.  DPP moves run at VALU latency, unlike
// LDS-routed lane shuffles.
// ---------------------------------------------------------------------------
constexpr int kDppSwap1 = 0xB1;        // quad_perm [1, 0, 3, 2]
constexpr int kDppSwap2 = 0x4E;        // quad_perm [2, 3, 0, 1]
constexpr int kDppHalfMirror = 0x141;  // lane i <- 7 - i within each half row
constexpr int kDppMirror = 0x140;      // lane i <- 15 - i within each row
constexpr int kDppRowShr = 0x110;      // + n: lane i <- i - n within each row
constexpr int kDppRowBcast15 = 0x142;  // lane 15 of each row -> the next row
constexpr int kDppRowBcast31 = 0x143;  // lane 31 -> rows 2 and 3

template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}

template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
    const long long x = __double_as_longlong(v);
    const int lo = __builtin_amdgcn_update_dpp(0, (int)x, CTRL, 0xF, 0xF, false);
    const int hi = __builtin_amdgcn_update_dpp(0, (int)(x >> 32), CTRL, 0xF, 0xF, false);
    return __longlong_as_double(((long long)hi << 32) | (long long)(unsigned int)lo);
}

// A DPP move of a double into the rows ROWS; lanes with no source in range,
// or outside ROWS, read 0.
template <int CTRL, int ROWS>
__device__ __forceinline__ double dpp_f64_or0(double v) {
    const long long x = __double_as_longlong(v);
    const int lo = __builtin_amdgcn_update_dpp(0, (int)x, CTRL, ROWS, 0xF, false);
    const int hi = __builtin_amdgcn_update_dpp(0, (int)(x >> 32), CTRL, ROWS, 0xF, false);
    return __longlong_as_double(((long long)hi << 32) | (long long)(unsigned int)lo);
}

__device__ __forceinline__ float lane_f32(float v, int lane) {
    return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), lane));
}

__device__ __forceinline__ double lane_f64(double v, int lane) {
    const long long x = __double_as_longlong(v);
    const int lo = __builtin_amdgcn_readlane((int)x, lane);
    const int hi = __builtin_amdgcn_readlane((int)(x >> 32), lane);
    return __longlong_as_double(((long long)hi << 32) | (long long)(unsigned int)lo);
}

__device__ __forceinline__ unsigned long long lane_u64(unsigned long long v, int lane) {
    const int lo = __builtin_amdgcn_readlane((int)v, lane);
    const int hi = __builtin_amdgcn_readlane((int)(v >> 32), lane);
    return ((unsigned long long)(unsigned int)hi << 32) | (unsigned long long)(unsigned int)lo;
}

__device__ __forceinline__ float wave_max(float v) {
    v = fmaxf(v, dpp_f32<kDppSwap1>(v));
    v = fmaxf(v, dpp_f32<kDppSwap2>(v));
    v = fmaxf(v, dpp_f32<kDppHalfMirror>(v));
    v = fmaxf(v, dpp_f32<kDppMirror>(v));
    return fmaxf(fmaxf(lane_f32(v, 0), lane_f32(v, 16)), fmaxf(lane_f32(v, 32), lane_f32(v, 48)));
}

__device__ __forceinline__ double wave_sum(double v) {
    v += dpp_f64<kDppSwap1>(v);
    v += dpp_f64<kDppSwap2>(v);
    v += dpp_f64<kDppHalfMirror>(v);
    v += dpp_f64<kDppMirror>(v);
    return (lane_f64(v, 0) + lane_f64(v, 16)) + (lane_f64(v, 32) + lane_f64(v, 48));
}

// Inclusive prefix sums over the wave in lane order (fixed order, fp64):
// shifts by 1, 2, 4 and 8 within each 16-lane row, then row 0's total into
// row 1 and row 2's into row 3, then the total of rows 0-1 into rows 2-3.
__device__ __forceinline__ double wave_inclusive_scan(double v) {
    v += dpp_f64_or0<kDppRowShr + 1, 0xF>(v);
    v += dpp_f64_or0<kDppRowShr + 2, 0xF>(v);
    v += dpp_f64_or0<kDppRowShr + 4, 0xF>(v);
    v += dpp_f64_or0<kDppRowShr + 8, 0xF>(v);
    v += dpp_f64_or0<kDppRowBcast15, 0xA>(v);
    v += dpp_f64_or0<kDppRowBcast31, 0xC>(v);
    return v;
}

// Maximum / sum over aligned groups of G (1, 2, 4, 8 or 16) lanes, left in
// every lane of the group; the same butterfly as wave_max / wave_sum, cut
// after log2(G) steps.  G must be uniform over the wave.
__device__ __forceinline__ float group_max(float v, int G) {
    if (G >= 2) v = fmaxf(v, dpp_f32<kDppSwap1>(v));
    if (G >= 4) v = fmaxf(v, dpp_f32<kDppSwap2>(v));
    if (G >= 8) v = fmaxf(v, dpp_f32<kDppHalfMirror>(v));
    if (G >= 16) v = fmaxf(v, dpp_f32<kDppMirror>(v));
    return v;
}

__device__ __forceinline__ double group_sum(double v, int G) {
    if (G >= 2) v += dpp_f64<kDppSwap1>(v);
    if (G >= 4) v += dpp_f64<kDppSwap2>(v);
    if (G >= 8) v += dpp_f64<kDppHalfMirror>(v);
    if (G >= 16) v += dpp_f64<kDppMirror>(v);
    return v;
}

__device__ __forceinline__ int wave_max_int(int v) {
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o, kWave));
    return v;
}

// Sum over the workgroup in a fixed order; the result is valid in every thread.
__device__ __forceinline__ double block_sum(double v, double* scratch /* [kWaves] in LDS */) {
    const int wave = threadIdx.x / kWave;
    const int lane = threadIdx.x % kWave;
    v = wave_sum(v);
    __syncthreads();
    if (lane == 0) scratch[wave] = v;
    __syncthreads();
    double s = scratch[0];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) s += scratch[w];
    return s;
}

// Inclusive scan over the workgroup in thread order (fixed order, fp64).
// Returns the inclusive prefix; `*total` receives the workgroup total.
__device__ __forceinline__ double block_inclusive_scan(double v, double* scratch /* [kWaves] */,
                                                       double* total) {
    const int wave = threadIdx.x / kWave;
    const int lane = threadIdx.x % kWave;
    v = wave_inclusive_scan(v);
    __syncthreads();
    if (lane == kWave - 1) scratch[wave] = v;
    __syncthreads();
    double off = 0.0;
    for (int w = 0; w < wave; ++w) off += scratch[w];
    double t = 0.0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) t += scratch[w];
    *total = t;
    return off + v;
}

// ---------------------------------------------------------------------------
// row normaliser: log sum_x exp(w(x)) = ln2 * (k + log2 s)
//
// With y = z * c (c = log2(e) / T) the running reference k is an integer
// (a ceiling of the running maximum of y), so rescaling the running sum when
// the maximum grows is an exact power-of-two scaling.  Each term
// 2^(fma(z, c, -k)) is evaluated from one correctly rounded argument, and the
// sum is kept in fp64.
// ---------------------------------------------------------------------------
struct Lse {
    float k;   // integral reference, or -inf while nothing finite was seen
    double s;  // sum of 2^(y - k)
};

// Exponent difference for ldexp: -inf and NaN map to a large negative value.
__device__ __forceinline__ int exp_delta(float d) { return (int)fmaxf(d, -2048.0f); }

__device__ __forceinline__ Lse lse_merge(Lse a, Lse b) {
    const float k = fmaxf(a.k, b.k);
    return Lse{k, ldexp(a.s, exp_delta(a.k - k)) + ldexp(b.s, exp_delta(b.k - k))};
}

// Absorb a block of U vectors with one update of the reference: the block's
// maximum first, then its terms summed pairwise in fp32 and added to the fp64
// running sum once.
template <int U, int E>
__device__ __forceinline__ void lse_absorb_block(Lse& st, const float (&x)[U][E], float c) {
    float m = x[0][0];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
        for (int e = 0; e < E; ++e) m = fmaxf(m, x[u][e]);
    const float kv = ceilf(m * c);
    if (kv > st.k) {
        st.s = ldexp(st.s, exp_delta(st.k - kv));
        st.k = kv;
    }
    const float nk = (st.k == -INFINITY) ? 0.0f : -st.k;
    float t[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        float v[E];
#pragma unroll
        for (int e = 0; e < E; ++e) v[e] = __builtin_amdgcn_exp2f(fmaf(x[u][e], c, nk));
#pragma unroll
        for (int w = E / 2; w >= 1; w /= 2)
#pragma unroll
            for (int e = 0; e < w; ++e) v[e] += v[e + w];
        t[u] = v[0];
    }
#pragma unroll
    for (int w = U / 2; w >= 1; w /= 2)
#pragma unroll
        for (int u = 0; u < w; ++u) t[u] += t[u + w];
    st.s += (double)t[0];
}

__device__ __forceinline__ Lse wave_lse(Lse st) {
    const float kw = wave_max(st.k);
    return Lse{kw, wave_sum(ldexp(st.s, exp_delta(st.k - kw)))};
}

// Valid in thread 0 only.
__device__ __forceinline__ Lse block_lse(Lse st, float* sk /* [kWaves] */, double* ss /* [kWaves] */) {
    const int wave = threadIdx.x / kWave;
    const int lane = threadIdx.x % kWave;
    const Lse w = wave_lse(st);
    if (lane == 0) {
        sk[wave] = w.k;
        ss[wave] = w.s;
    }
    __syncthreads();
    Lse out{-INFINITY, 0.0};
    if (threadIdx.x == 0) {
        out = Lse{sk[0], ss[0]};
#pragma unroll
        for (int i = 1; i < kWaves; ++i) out = lse_merge(out, Lse{sk[i], ss[i]});
    }
    return out;
}

// block_lse with the result in every thread (same bits as block_lse's thread 0).
__device__ __forceinline__ Lse block_lse_all(Lse st, float* sk /* [kWaves] */, double* ss /* [kWaves] */) {
    const int wave = threadIdx.x / kWave;
    const int lane = threadIdx.x % kWave;
    const Lse w = wave_lse(st);
    if (lane == 0) {
        sk[wave] = w.k;
        ss[wave] = w.s;
    }
    __syncthreads();
    Lse out{sk[0], ss[0]};
#pragma unroll
    for (int i = 1; i < kWaves; ++i) out = lse_merge(out, Lse{sk[i], ss[i]});
    return out;
}

}  // namespace sv
