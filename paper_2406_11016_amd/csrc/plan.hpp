// Host-side planning of the verification launch: tile sizes, workspace
// layout, the order of the roles in the grid, and argument validation.
//
// Plain C++17 with no device code, so the same code is compiled into the
// HIP library and, on the CPU, into a sanitizer-instrumented checker of its
// arithmetic (tests/native/plan_check.cpp).  div_of is constexpr, so the
// kernels call it too.  role_at is the host model of verify_kernel's role
// split: the kernel spells the same branches out inline, each calling its
// role directly, because routing every role through one returned value
// merges their register live ranges and makes the kernel spill.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <algorithm>
#include <cmath>

#include "spec_verify.h"

namespace sv {

constexpr int kThreads = 256;            // threads per workgroup (4 wave64s)
constexpr int kWave = 64;
constexpr int kWaves = kThreads / kWave;
constexpr int kMaxGamma = SV_MAX_GAMMA;
constexpr int kMaxRows = 2 * kMaxGamma + 1;
constexpr int kUnroll = 8;               // 16-byte loads in flight per thread in the stats stream

constexpr int kWantStatsTiles = 1024;    // enough workgroups to fill 256 CUs (4 per CU) once
constexpr int kWantSampleTiles = 1024;
constexpr int kStatsTileBytes = 32768;   // at most 32 KiB of one row per stats workgroup
constexpr long long kSelfDecideWords = 16384;     // pair copies polled by self-deciding mass workgroups
constexpr long long kLagStreamBytes = 56000000;  // stream between an element's stats and its mass tiles
constexpr int kGammaTileBytes = 16384;   // target rows gamma, streamed last: short tiles end the stream sharply
constexpr int kSampleTileBytes = 32768;
constexpr int kMaxStatsSub = 1028;       // stats chunks of one batch element's 2 gamma decision rows
constexpr int kMaxSub = 1024;            // sub-chunk masses of one batch element (nchunk2 * kWaves)
constexpr int kMaxSpins = 1 << 17;       // default bound on every wait (about 0.1 s), so every wave exits
constexpr int kDecisionWords = 5;        // L and the sentinel flag, then 8 floats of weight constants

// Workspace header (the first 256 bytes): the 32-bit word at byte 4 is the
// sticky error flag (a wait timed out); the 32-bit word at byte 8, when
// nonzero, replaces kMaxSpins as the bound on each wait (a test hook: a
// zero-filled workspace uses the default).
constexpr size_t kHeaderBytes = 256;
constexpr size_t kErrorFlagOffset = 4;
constexpr size_t kSpinLimitOffset = 8;

inline long long ceil_div(long long a, long long b) { return (a + b - 1) / b; }

// XCDs of the GPU: workgroup i of a launch runs on XCD i mod kXcds (see g_tile).
constexpr int kXcds = 8;
inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

inline bool valid_dtype(sv_dtype_t dt) { return dt == SV_F32 || dt == SV_F16 || dt == SV_BF16; }
inline int bytes_per_logit(sv_dtype_t dt) { return dt == SV_F32 ? 4 : 2; }

// ---------------------------------------------------------------------------
// n / d for 0 <= n < 2^31 as one 32 x 32 -> 64-bit multiply and a shift:
// with L = ceil(log2 d) and m = floor(2^(31+L) / d) + 1 (< 2^32), the error of
// n m / 2^(31+L) over n / d is below 2^-L <= 1/d, so the floor is exact.
// ---------------------------------------------------------------------------
struct Div {
    unsigned int m, sh;
};

constexpr unsigned int div_of(Div d, unsigned int n) {
    return (unsigned int)(((unsigned long long)n * d.m) >> d.sh);
}

inline Div make_div(unsigned int d) {
    unsigned int L = 0;
    while ((1ull << L) < d) ++L;
    const unsigned long long m = ((1ull << (31 + L)) / d) + 1;
    return Div{(unsigned int)m, 31 + L};
}

// ---------------------------------------------------------------------------
// Tile sizes and workspace layout; they depend only on (B, gamma, V, dtype).
// ---------------------------------------------------------------------------
struct Plan {
    int E;                   // elements per 16-byte vector
    int chunk1, nchunk1;     // decision rows: chunk length and chunks per row
    int chunk1s, nchunk1s;   // the same for the row-staged early exit (twice as long)
    int chunk2, nchunk2;     // final-distribution tiles
    int chunkg, nchunkg;     // target row gamma: short tiles, one (K, S) pair per quarter
    long long pstride;       // stats words per batch element
    long long qstride;       // words of one mass workgroup's copy of the decision rows' pairs (0: no copies)
    long long n_stats, n_mass;
    int gwords;              // row-staged early exit: gate words per stage
    long long gstride;       //                        and gate + state words per batch element
    size_t off_dslot, off_pslot, off_mslot, off_gslot, off_qslot, bytes;
};

inline bool pipelined_waits(long long B, long long gamma, long long V, sv_dtype_t dt);

inline bool make_plan(int32_t B, int32_t gamma, int32_t V, sv_dtype_t dt, Plan* p) {
    if (B < 1 || gamma < 1 || gamma > kMaxGamma || V < 1 || !valid_dtype(dt)) return false;
    const int E = (dt == SV_F32) ? 4 : 8;
    const int s = bytes_per_logit(dt);
    const long long R = 2LL * gamma;  // the decision rows
    const long long R1 = R + 1;       // all rows of an element
    if ((long long)B * (gamma + 1) * (long long)V > (1LL << 40)) return false;
    const long long min_elems = (long long)kThreads * E;
    const long long max_cells = std::max<long long>(1, ceil_div(V, min_elems));

    // decision-row chunks: enough workgroups to fill the GPU, at most 32 KiB
    // each (smaller tiles end the stream sooner after their dispatch, but past
    // ~10K workgroups per launch the dispatcher, not HBM, sets the pace); the
    // chunk count is sized over all 2 gamma + 1 rows of an element
    long long nc = ceil_div(kWantStatsTiles, B * R1);
    nc = std::max(nc, ceil_div(V, kStatsTileBytes / s));
    nc = std::min(nc, max_cells);
    nc = std::min(nc, std::max<long long>(1, kMaxStatsSub / R1));
    const long long chunk = ceil_div(ceil_div(V, nc), E) * E;
    p->chunk1 = (int)chunk;
    p->nchunk1 = (int)ceil_div(V, chunk);
    if (R1 * p->nchunk1 > kMaxStatsSub) return false;
    // the row-staged early exit streams chunks twice as long: when most of
    // its rows are skipped it is bound by how fast workgroups are dispatched,
    // not by HBM, so fewer of them pay
    const long long chunks = ceil_div(ceil_div(V, std::max(1LL, ceil_div(p->nchunk1, 2))), E) * E;
    p->chunk1s = (int)chunks;
    p->nchunk1s = (int)ceil_div(V, chunks);

    // target row gamma in short tiles whose quarters fit the bonus draw's scan
    // (at most one vector per thread of a workgroup); the row's quarter masses
    // must fit kMaxSub
    const long long ncg = std::max(ceil_div(V, kGammaTileBytes / s), ceil_div(V, (long long)kWaves * kThreads * E));
    const long long chunkg = ceil_div(ceil_div(V, ncg), E) * E;
    p->chunkg = (int)chunkg;
    p->nchunkg = (int)ceil_div(V, chunkg);
    if ((long long)p->nchunkg * kWaves > kMaxSub || ceil_div(chunkg / E, kWaves) > kThreads) return false;

    // final-distribution tiles: a sub-chunk (a quarter tile) must fit one
    // vector per thread, and b's sub-chunk masses must fit kMaxSub
    const long long max_tile_vecs = (long long)kWaves * kThreads;
    long long nc2 = ceil_div(kWantSampleTiles, B);
    nc2 = std::max(nc2, ceil_div(V, kSampleTileBytes / s));
    nc2 = std::min(nc2, max_cells);
    nc2 = std::min(nc2, (long long)kMaxSub / kWaves);
    nc2 = std::max(nc2, ceil_div(V, max_tile_vecs * E));
    const long long chunk2 = ceil_div(ceil_div(V, nc2), E) * E;
    p->chunk2 = (int)chunk2;
    p->nchunk2 = (int)ceil_div(V, chunk2);
    if ((long long)p->nchunk2 * kWaves > kMaxSub || chunk2 / E > max_tile_vecs) return false;
    p->E = E;

    p->n_stats = (long long)B * (R * p->nchunk1 + p->nchunkg);
    p->n_mass = (long long)B * p->nchunk2;
    // plus a decider, a draw and a bonus workgroup per batch element
    if (p->n_stats + p->n_mass + 3LL * B > 0x7fffffffLL) return false;

    size_t off = kHeaderBytes;
    p->off_dslot = off;
    off = align256(off + sizeof(unsigned long long) * (size_t)B * (p->nchunk2 + 2) * kDecisionWords);
    p->off_pslot = off;
    p->pstride = 2 * (R * p->nchunk1 + (long long)kWaves * p->nchunkg);
    off = align256(off + sizeof(unsigned long long) * (size_t)B * p->pstride);
    p->off_mslot = off;
    off = align256(off + sizeof(unsigned long long) * (size_t)p->n_mass * kWaves);
    p->gwords = std::max(2 * p->nchunk1, p->nchunkg);
    p->gstride = (long long)(gamma + 1) * p->gwords + gamma;
    p->off_gslot = off;
    off = align256(off + sizeof(unsigned long long) * (size_t)B * p->gstride);
    // short streams with few pairs to copy: each mass workgroup decides for
    // itself from its own copy of the decision rows' (K, S) pairs
    p->qstride = (pipelined_waits(B, gamma, V, dt) && (long long)B * p->nchunk2 * 2 * R * p->nchunk1 <= kSelfDecideWords)
                     ? 2 * R * p->nchunk1
                     : 0;
    p->off_qslot = off;
    off = align256(off + sizeof(unsigned long long) * (size_t)B * p->nchunk2 * p->qstride);
    p->bytes = off;
    return true;
}

// ---------------------------------------------------------------------------
// Role order of the single-pass launch (verify_kernel).  Units u = 0 .. B-1:
// unit u holds the S stats tiles of b = u's decision rows, then b's decider,
// followed (for u >= lagM) by the Mt mass tiles and the draw of b = u - lagM;
// then the G tiles of every target row gamma; then the mass tiles and draws
// of the last lagM elements; then one bonus workgroup per element.  Segments
// have uniform unit sizes, so a workgroup finds its role with at most one
// division.
// ---------------------------------------------------------------------------
struct Layout {
    Div d0, d1, d2, dc1, dcg;          // division by size0, size1, size2, nchunk1, nchunkg
    unsigned int end0, end1;           // ends of unit segments 0 (stats + decider) and 1 (all four)
    unsigned int endg, end2;           // ends of segment G (target rows gamma) and 2 (mass + draw)
    unsigned int size0, size1, size2;  // workgroups per unit in segments 0, 1, 2
    int lagM;                          // unit lag of the mass and draw roles
    int b2;                            // batch element of the first unit of segment 2
    int S;                             // stats tiles per unit (0 in sigmoid mode)
    int Mt;                            // mass tiles per batch element
};

// The lag in units: about kLagStreamBytes of stream (~9 us at 6.5 TB/s, the
// time a decision takes to publish under load) behind the element's stats,
// and all of them after the stream when the whole stream is shorter than
// that (or absent: the sigmoid mode streams no rows).
inline long long lag_units(long long B, long long unit_bytes) {
    if (unit_bytes <= 0) return B;
    return std::min(B, std::max(1LL, ceil_div(kLagStreamBytes, unit_bytes)));
}

inline Layout make_layout(long long B, long long S, long long Mt, long long G, int nchunk1, int nchunkg,
                          long long lagM) {
    Layout y{};
    y.size0 = (unsigned int)(S + 1);
    y.size1 = (unsigned int)(S + Mt + 2);
    y.size2 = (unsigned int)(Mt + 1);
    y.end0 = (unsigned int)(lagM * (S + 1));
    y.end1 = (unsigned int)(y.end0 + (B - lagM) * (S + Mt + 2));
    y.endg = (unsigned int)(y.end1 + G);
    y.end2 = (unsigned int)(y.endg + lagM * (Mt + 1));
    y.lagM = (int)lagM;
    y.b2 = (int)(B - lagM);
    y.S = (int)S;
    y.Mt = (int)Mt;
    y.d0 = make_div(y.size0);
    y.d1 = make_div(y.size1);
    y.d2 = make_div(y.size2);
    y.dc1 = make_div((unsigned int)std::max(1, nchunk1));
    y.dcg = make_div((unsigned int)std::max(1, nchunkg));
    return y;
}

enum RoleKind : int { kRoleStats = 0, kRoleDecider = 1, kRoleMass = 2, kRoleDraw = 3, kRoleRowG = 4, kRoleBonus = 5 };

struct Role {
    int kind;
    int b;      // batch element
    int slot;   // stats: decision-row slot (target rows 0 .. gamma-1, then draft rows 0 .. gamma-1)
    int k;      // stats: chunk of the slot; row gamma: tile; mass: tile
};

// Target row gamma's tiles (segment G of the single pass).  Workgroup i of a
// launch runs on XCD i mod kXcds (the dispatcher deals workgroups to the XCDs
// in turn), and each XCD has its own L2, so a workgroup re-reads data that
// another workgroup of its XCD loaded from that L2 (about a quarter of the
// latency of HBM).  The elements are taken in groups of kXcds: in a full
// group, tile j of the group's element e sits at position
// kXcds j + (e + d) mod kXcds of the group, d = (end2 - end1) mod kXcds, so
// that every tile of element b runs on the XCD of b's bonus workgroup (id
// end2 + b), whose draw re-reads one of their quarters.  The elements of a
// last partial group keep their tiles contiguous.
struct GTile {
    int b;  // batch element
    int k;  // tile of its target row gamma
};

// Tile t of segment G: dcg divides by nchunkg, and end1 / end2 are the
// layout's.  Scalar arguments and forced inlining keep the kernel's launch
// arguments in registers (a call would spill around it).
__attribute__((always_inline)) constexpr GTile g_tile(Div dcg, unsigned int end1, unsigned int end2, int B, int nchunkg,
                                                      int t) {
    static_assert(kXcds == 8, "the masks below take kXcds = 8");
    const int bfull = B & ~7;
    if (t < bfull * nchunkg) {
        const int g = (int)div_of(dcg, (unsigned int)t >> 3);
        const int p = t - g * 8 * nchunkg;
        const int d = (int)((end2 - end1) & 7u);
        return GTile{8 * g + (((p & 7) - d) & 7), p >> 3};
    }
    const int t2 = t - bfull * nchunkg;
    const int bb = (int)div_of(dcg, (unsigned int)t2);
    return GTile{bfull + bb, t2 - bb * nchunkg};
}

// The role of workgroup `id` of the single-pass launch (id < end2 + B).
constexpr Role role_at(const Layout& y, int nchunk1, int nchunkg, unsigned int id) {
    unsigned int r = 0;
    int bs = 0, bm = 0;
    if (id < y.end0) {
        const unsigned int k = div_of(y.d0, id);
        r = id - k * y.size0;
        bs = (int)k;
    } else if (id < y.end1) {
        const unsigned int loc = id - y.end0;
        const unsigned int k = div_of(y.d1, loc);
        r = loc - k * y.size1;
        bs = y.lagM + (int)k;
        bm = (int)k;
    } else if (id < y.endg) {
        const GTile g = g_tile(y.dcg, y.end1, y.end2, y.b2 + y.lagM, nchunkg, (int)(id - y.end1));
        return Role{kRoleRowG, g.b, 0, g.k};
    } else if (id < y.end2) {
        const unsigned int loc = id - y.endg;
        const unsigned int k = div_of(y.d2, loc);
        r = loc - k * y.size2 + (unsigned int)y.S + 1u;
        bm = y.b2 + (int)k;
    } else {
        return Role{kRoleBonus, (int)(id - y.end2), 0, 0};
    }
    const unsigned int S = (unsigned int)y.S;
    if (r < S) {
        const int slot = (int)div_of(y.dc1, r);
        return Role{kRoleStats, bs, slot, (int)r - slot * nchunk1};
    }
    if (r == S) return Role{kRoleDecider, bs, 0, 0};
    r -= S + 1u;
    if (r < (unsigned int)y.Mt) return Role{kRoleMass, bm, 0, (int)r};
    return Role{kRoleDraw, bm, 0, 0};
}

// The single-pass layout of a call: in the exact mode units of the 2 gamma
// decision rows' stats tiles; target row gamma (exact: stats tiles, sigmoid:
// row tiles) after the units; the lag from kLagStreamBytes of decision-row
// stream.  The grid has end2 + B workgroups (the bonus workgroups last).
inline Layout single_pass_layout(long long B, long long gamma, long long V, sv_dtype_t dt, bool exact, const Plan& pl) {
    const long long unit_bytes = exact ? 2LL * gamma * V * bytes_per_logit(dt) : 0;
    return make_layout(B, exact ? 2LL * gamma * pl.nchunk1 : 0, pl.nchunk2, B * pl.nchunkg, pl.nchunk1, pl.nchunkg,
                       lag_units(B, unit_bytes));
}

// Whether the single pass (exact mode, not ragged) waits with two polls in
// flight: where the decision rows' stream is shorter than the mass lag, the
// step after the stream is a chain of waits (decision, masses, draw) that
// the quicker detection shortens.  On long streams the second poll measured
// slower, so they keep one.
inline bool pipelined_waits(long long B, long long gamma, long long V, sv_dtype_t dt) {
    return 2LL * gamma * V * bytes_per_logit(dt) * B < kLagStreamBytes;
}

// Copies of each decision record, one per reader: every mass workgroup, the
// draw and the bonus workgroup (exact mode; the mass workgroups' copies stay
// unwritten where they decide for themselves, see qstride); only the bonus
// workgroup (sigmoid mode, whose mass and draw workgroups decide for
// themselves).
inline int decision_copies(bool exact, const Plan& pl) { return exact ? pl.nchunk2 + 2 : 1; }

// ---------------------------------------------------------------------------
// Role order of the row-staged early exit (staged_kernel): gamma B units of
// 2 nchunk1 tiles and a row-decider slot (unit c B + b), B row deciders of
// position gamma - 1, B nchunkg tiles of the target rows gamma, B units of
// Mt mass tiles and a draw; the B bonus workgroups follow end2.
// ---------------------------------------------------------------------------
inline Layout make_staged_layout(long long B, long long gamma, int nchunk1, int nchunkg, long long Mt) {
    Layout y{};
    y.size0 = (unsigned int)(2LL * nchunk1 + 1);
    y.size2 = (unsigned int)(Mt + 1);
    y.end0 = (unsigned int)(gamma * B * y.size0);
    y.end1 = (unsigned int)(y.end0 + B);
    y.endg = (unsigned int)(y.end1 + B * nchunkg);
    y.end2 = (unsigned int)(y.endg + B * y.size2);
    y.Mt = (int)Mt;
    y.d0 = make_div(y.size0);
    y.d1 = make_div((unsigned int)B);
    y.d2 = make_div(y.size2);
    y.dcg = make_div((unsigned int)std::max(1, nchunkg));
    return y;
}

enum StagedRoleKind : int { kStagedTile = 0, kStagedRowDecider = 1, kStagedRowG = 2, kStagedMass = 3,
                            kStagedDraw = 4, kStagedBonus = 5 };

struct StagedRole {
    int kind;
    int b;
    int c;  // tile: stage (draft position); row decider: its position
    int k;  // tile: index in the stage's 2 nchunk1 tiles; row gamma: tile; mass: tile
};

// The role of workgroup `id` of the staged launch (id < end2 + B): the host
// model of staged_kernel's split.
constexpr StagedRole staged_role_at(const Layout& y, int B, int gamma, int nchunkg, unsigned int id) {
    if (id < y.end0) {
        const unsigned int u = div_of(y.d0, id);  // unit c B + b
        const unsigned int r = id - u * y.size0;
        const unsigned int c = div_of(y.d1, u);
        const int b = (int)(u - c * (unsigned int)B);
        if (r + 1u < y.size0) return StagedRole{kStagedTile, b, (int)c, (int)r};
        return StagedRole{kStagedRowDecider, b, (int)c - 1, 0};  // c == 0: none (the slot is idle)
    }
    if (id < y.end1) return StagedRole{kStagedRowDecider, (int)(id - y.end0), gamma - 1, 0};
    if (id < y.endg) {
        const int t = (int)(id - y.end1);
        const int b = (int)div_of(y.dcg, (unsigned int)t);
        return StagedRole{kStagedRowG, b, gamma, t - b * nchunkg};
    }
    if (id < y.end2) {
        const unsigned int loc = id - y.endg;
        const unsigned int b = div_of(y.d2, loc);
        const unsigned int r = loc - b * y.size2;
        if (r < (unsigned int)y.Mt) return StagedRole{kStagedMass, (int)b, 0, (int)r};
        return StagedRole{kStagedDraw, (int)b, 0, 0};
    }
    return StagedRole{kStagedBonus, (int)(id - y.end2), 0, 0};
}

// Stages between a row decider and the tiles it gates: about kLagStreamBytes
// of stream (the time a decision takes to publish under load), so that a
// gated tile rarely waits, and at least 2 (row decider c sits among the units
// of stage c + 1).
inline int gate_stages(long long B, long long V, long long s) {
    return (int)std::max(2LL, ceil_div(kLagStreamBytes, 2 * B * V * s));
}

// Workgroups of the staged launch, or -1 when the staged order cannot skip
// any row (gate >= gamma: the single pass serves) or exceeds 2^31 workgroups.
inline long long staged_workgroups(long long B, long long gamma, long long V, sv_dtype_t dt, const Plan& pl) {
    const long long n = B * (gamma * (2LL * pl.nchunk1s + 1) + 1 + pl.nchunkg + pl.nchunk2 + 2);
    if (gate_stages(B, V, bytes_per_logit(dt)) >= gamma || n > 0x7fffffffLL) return -1;
    return n;
}

// The decoding loop's automatic choice of the early exit for the next step:
// after a step of `gamma` drafts whose accepted lengths sum to `accepted_sum`
// over B elements, the early exit pays when the mean accepted length is below
// gamma / 2 (it measured 1.16-1.59x the single pass at mean accepted 1.23 ..
// 0.02 of gamma 8, and 0.77x at 7.41).
inline bool early_exit_pays(long long accepted_sum, long long B, int gamma) {
    return B > 0 && 2 * accepted_sum < (long long)gamma * B;
}

// ---------------------------------------------------------------------------
// Arguments of one call and their validation (before anything is launched).
// ---------------------------------------------------------------------------
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
    const int32_t* gammas;  // ragged variant, else nullptr
    bool staged = false;    // exact mode: the row-staged early exit
};

inline sv_status_t validate(const Call& a, bool exact, Plan* pl) {
    if (a.draft == nullptr || a.target == nullptr || a.tokens == nullptr || a.uniforms == nullptr ||
        a.accepted_len == nullptr || a.next_token == nullptr || a.ws == nullptr)
        return SV_ERR_NULL;
    if (!valid_dtype(a.dt)) return SV_ERR_DTYPE;
    if (!make_plan(a.B, a.gamma, a.V, a.dt, pl)) return SV_ERR_SHAPE;
    if (!(std::isfinite(a.temperature) && a.temperature > 0.0f)) return SV_ERR_PARAM;
    const double c = 1.4426950408889634074 / (double)a.temperature;
    if (!(std::isfinite((float)c) && (float)c > 0.0f)) return SV_ERR_PARAM;
    if (!exact) {
        if (!(std::isfinite(a.alpha) && std::isfinite(a.beta) && a.alpha < a.beta)) return SV_ERR_PARAM;
        const double s = 1.0 / ((double)a.temperature * ((double)a.beta - (double)a.alpha));
        if (!(std::isfinite((float)s) && (float)s > 0.0f)) return SV_ERR_PARAM;
    }
    if (a.ws_bytes < pl->bytes || (reinterpret_cast<uintptr_t>(a.ws) & 15u) != 0) return SV_ERR_WORKSPACE;
    return SV_OK;
}

}  // namespace sv
