// Host-side checks of the launch planning in plan.hpp, built on the CPU with
// -fsanitize=address,undefined (tests/test_plan_native.py builds and runs it).
//
//   1. The multiply-shift division is exact for every divisor and dividend the
//      layouts use (brute force over small ranges, every multiple boundary).
//   2. make_plan over a grid of shapes up to the largest vocabularies the
//      header allows: tile counts within the LDS arrays the kernels size for
//      them, chunks covering each row exactly, the target row gamma always in
//      short tiles the bonus draw can scan, workspace regions aligned and
//      disjoint, and the size limits rejected.
//   3. Both launch layouts simulated workgroup by workgroup (role_at,
//      staged_role_at): every role of every element appears exactly once, and
//      every workgroup that waits comes after the workgroups it waits on (the
//      ordering the kernels' deadlock-freedom rests on); target row gamma's
//      tiles of an element share its bonus workgroup's XCD (id mod 8).
//   4. Argument validation: the cases of the C ABI's error contract.
//
// Prints one line per section and exits nonzero on the first failure.
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <cmath>
#include <limits>
#include <vector>

#include "plan.hpp"

using namespace sv;

static long long g_checks = 0;

#define CHECK(cond, ...)                                                       \
    do {                                                                       \
        ++g_checks;                                                            \
        if (!(cond)) {                                                         \
            fprintf(stderr, "FAILED %s:%d: %s: ", __FILE__, __LINE__, #cond);  \
            fprintf(stderr, __VA_ARGS__);                                      \
            fprintf(stderr, "\n");                                             \
            exit(1);                                                           \
        }                                                                      \
    } while (0)

// --- 1. division -------------------------------------------------------------

static void check_div(unsigned int d, unsigned int nmax_brute) {
    const Div q = make_div(d);
    for (unsigned int n = 0; n < nmax_brute; ++n) CHECK(div_of(q, n) == n / d, "d=%u n=%u", d, n);
    // every multiple boundary below 2^31 for small d is too many; sample them
    const unsigned long long step = std::max<unsigned long long>(1, (0x7fffffffULL / d) / 4096);
    for (unsigned long long k = 1; k * d <= 0x7fffffffULL; k += step)
        for (long long off = -1; off <= 1; ++off) {
            const long long n = (long long)(k * d) + off;
            if (n < 0 || n > 0x7fffffffLL) continue;
            CHECK(div_of(q, (unsigned int)n) == (unsigned int)n / d, "d=%u n=%lld", d, n);
        }
    CHECK(div_of(q, 0x7fffffffu) == 0x7fffffffu / d, "d=%u n=2^31-1", d);
}

static void section_div() {
    for (unsigned int d = 1; d <= 4096; ++d) check_div(d, d <= 64 ? 1u << 16 : 4 * d + 3);
    const unsigned int big[] = {4097, 5441, 65535, 65536, 65537, 1u << 20, (1u << 20) + 1, 123456789u,
                                0x3fffffffu, 0x7fffffffu};
    for (unsigned int d : big) check_div(d, 4096);
    printf("division: ok\n");
}

// --- 2. plans -----------------------------------------------------------------

static const sv_dtype_t kDtypes[] = {SV_F32, SV_F16, SV_BF16};

static long long vmax(sv_dtype_t dt) { return dt == SV_F32 ? (1LL << 20) : (1LL << 21); }

static void check_plan(int B, int gamma, int V, sv_dtype_t dt, const Plan& p) {
    const int E = (dt == SV_F32) ? 4 : 8;
    CHECK(p.E == E, "E");
    // decision rows: chunks cover the row exactly, in whole vectors
    CHECK(p.chunk1 % E == 0 && p.chunk1 > 0, "chunk1 %d", p.chunk1);
    CHECK((long long)p.nchunk1 * p.chunk1 >= V && (long long)(p.nchunk1 - 1) * p.chunk1 < V, "nchunk1");
    CHECK((2LL * gamma + 1) * p.nchunk1 <= kMaxStatsSub, "stats pairs %d x %d exceed the LDS arrays", gamma, p.nchunk1);
    // the early exit's chunks: whole vectors, covering V, at most the single
    // pass's count (so its pairs and gate words fit the same regions)
    CHECK(p.chunk1s % E == 0 && p.chunk1s >= p.chunk1, "chunk1s %d", p.chunk1s);
    CHECK((long long)p.nchunk1s * p.chunk1s >= V && (long long)(p.nchunk1s - 1) * p.chunk1s < V, "nchunk1s");
    CHECK(p.nchunk1s >= 1 && p.nchunk1s <= p.nchunk1 && p.nchunk1s >= (p.nchunk1 + 1) / 2 - 1, "nchunk1s %d of %d",
          p.nchunk1s, p.nchunk1);
    // the stats stream: each wave's quarter of a chunk
    // target row gamma: quarters fit the bonus draw (one vector per thread of a
    // workgroup, or 4 vectors per lane of one wave), masses fit kMaxSub
    CHECK(p.chunkg % E == 0 && (long long)p.nchunkg * p.chunkg >= V && (long long)(p.nchunkg - 1) * p.chunkg < V,
          "nchunkg");
    CHECK((long long)p.nchunkg * kWaves <= kMaxSub, "row gamma quarters %d", p.nchunkg * kWaves);
    CHECK(ceil_div(p.chunkg / E, kWaves) <= kThreads, "row gamma quarter vectors");
    // final-distribution tiles
    CHECK(p.chunk2 % E == 0 && (long long)p.nchunk2 * p.chunk2 >= V && (long long)(p.nchunk2 - 1) * p.chunk2 < V,
          "nchunk2");
    CHECK((long long)p.nchunk2 * kWaves <= kMaxSub, "mass words");
    CHECK(ceil_div(p.chunk2 / E, kWaves) <= kThreads, "sub-chunk vectors");
    // workspace: header, then aligned, disjoint regions in order
    CHECK(p.off_dslot == kHeaderBytes, "dslot offset");
    CHECK(p.off_dslot % 256 == 0 && p.off_pslot % 256 == 0 && p.off_mslot % 256 == 0 && p.off_gslot % 256 == 0 &&
              p.bytes % 256 == 0, "alignment");
    const size_t w = sizeof(unsigned long long);
    CHECK(p.off_pslot >= p.off_dslot + w * (size_t)B * (p.nchunk2 + 2) * kDecisionWords, "dslot size");
    CHECK(p.pstride == 2 * (2LL * gamma * p.nchunk1 + (long long)kWaves * p.nchunkg), "pstride");
    CHECK(p.off_mslot >= p.off_pslot + w * (size_t)B * (size_t)p.pstride, "pslot size");
    CHECK(p.off_gslot >= p.off_mslot + w * (size_t)B * p.nchunk2 * kWaves, "mslot size");
    CHECK(p.off_qslot % 256 == 0 && p.off_qslot >= p.off_gslot + w * (size_t)B * (size_t)p.gstride, "gslot size");
    // the self-deciding mass workgroups' pair copies: only for short streams
    // with few words to copy, one copy of every decision-row pair per tile
    CHECK(p.qstride == 0 || (pipelined_waits(B, gamma, V, dt) && p.qstride == 4LL * gamma * p.nchunk1 &&
                             (long long)B * p.nchunk2 * p.qstride <= kSelfDecideWords),
          "qstride %lld", p.qstride);
    CHECK(p.bytes >= p.off_qslot + w * (size_t)B * p.nchunk2 * (size_t)p.qstride, "qslot size");
    CHECK(p.gwords >= 2 * p.nchunk1 && p.gwords >= p.nchunkg, "gwords");
    // the kernels index the stats words with int
    CHECK(p.pstride < 0x7fffffffLL && p.gstride < 0x7fffffffLL && p.qstride < 0x7fffffffLL, "strides");
}

static std::vector<int> batch_grid() { return {1, 2, 3, 5, 7, 16, 17, 32, 63, 64, 65, 128, 257, 1000, 4096}; }
static std::vector<int> gamma_grid() { return {1, 2, 3, 4, 5, 8, 10, 16, 17, 20, 31, 32, 33, 64, 65, 100, 127, 128}; }
static std::vector<int> vocab_grid() {
    return {1, 2, 7, 8, 9, 63, 64, 65, 255, 256, 1023, 1024, 1025, 2047, 2048, 2049, 4096, 4097, 8191, 8192, 8193,
            32000, 50272, 51865, 128256, 131072, 131073, 300007, 600011, (1 << 20) - 1, 1 << 20, (1 << 20) + 1,
            (1 << 21) - 1, 1 << 21, (1 << 21) + 1};
}

static void section_plans() {
    long long valid = 0;
    for (sv_dtype_t dt : kDtypes)
        for (int B : batch_grid())
            for (int gamma : gamma_grid())
                for (int V : vocab_grid()) {
                    Plan p{};
                    const bool ok = make_plan(B, gamma, V, dt, &p);
                    const bool in_range = V <= vmax(dt) && (long long)B * (gamma + 1) * (long long)V <= (1LL << 40);
                    if (ok) {
                        ++valid;
                        check_plan(B, gamma, V, dt, p);
                        const long long grid = p.n_stats + p.n_mass + 3LL * B;
                        CHECK(grid <= 0x7fffffffLL, "grid");
                    } else {
                        // the only rejections on this grid: vocabularies past the
                        // limit and tensors past 2^40 logits (no grid here comes
                        // near 2^31 workgroups)
                        CHECK(!in_range, "rejected B=%d gamma=%d V=%d dt=%d", B, gamma, V, (int)dt);
                    }
                    if (V > vmax(dt)) CHECK(!ok, "accepted V=%d past the limit for dt=%d", V, (int)dt);
                }
    // invalid arguments
    Plan p{};
    CHECK(!make_plan(0, 5, 100, SV_F32, &p) && !make_plan(1, 0, 100, SV_F32, &p) &&
              !make_plan(1, 129, 100, SV_F32, &p) && !make_plan(1, 5, 0, SV_F32, &p) &&
              !make_plan(1, 5, 100, (sv_dtype_t)3, &p) && !make_plan(-1, 5, 100, SV_F32, &p),
          "invalid sizes accepted");
    printf("plans: ok (%lld valid shapes)\n", valid);
}

// --- 3. layouts ----------------------------------------------------------------

struct Seen {
    std::vector<long long> stats, rowg, mass, decider, draw, bonus;
};

static void simulate_single_pass(int B, int gamma, int V, sv_dtype_t dt, bool exact) {
    Plan p{};
    CHECK(make_plan(B, gamma, V, dt, &p), "plan");
    const Layout y = single_pass_layout(B, gamma, V, dt, exact, p);
    const long long n = (long long)y.end2 + B;
    CHECK(n <= 0x7fffffffLL, "grid");
    const int S = exact ? 2 * gamma * p.nchunk1 : 0;
    CHECK(y.S == S && y.Mt == p.nchunk2, "unit sizes");
    CHECK(y.lagM >= 1 && y.lagM <= B, "lag %d", y.lagM);
    CHECK(y.end0 <= y.end1 && y.end1 <= y.endg && y.endg <= y.end2, "segment order");
    Seen s;
    s.stats.assign((size_t)B * (S > 0 ? S : 1), -1);
    s.rowg.assign((size_t)B * p.nchunkg, -1);
    s.mass.assign((size_t)B * p.nchunk2, -1);
    s.decider.assign(B, -1);
    s.draw.assign(B, -1);
    s.bonus.assign(B, -1);
    auto mark = [&](std::vector<long long>& v, long long i, long long id, const char* what) {
        CHECK(i >= 0 && i < (long long)v.size(), "%s index %lld out of range (id %lld)", what, i, id);
        CHECK(v[i] < 0, "%s %lld assigned twice (ids %lld and %lld)", what, i, v[i], id);
        v[i] = id;
    };
    for (long long id = 0; id < n; ++id) {
        const Role r = role_at(y, p.nchunk1, p.nchunkg, (unsigned int)id);
        CHECK(r.b >= 0 && r.b < B, "element %d (id %lld)", r.b, id);
        switch (r.kind) {
            case kRoleStats:
                CHECK(exact && r.slot >= 0 && r.slot < 2 * gamma && r.k >= 0 && r.k < p.nchunk1, "stats slot");
                mark(s.stats, (long long)r.b * S + (long long)r.slot * p.nchunk1 + r.k, id, "stats");
                break;
            case kRoleRowG: mark(s.rowg, (long long)r.b * p.nchunkg + r.k, id, "row gamma tile"); break;
            case kRoleMass: mark(s.mass, (long long)r.b * p.nchunk2 + r.k, id, "mass tile"); break;
            case kRoleDecider: mark(s.decider, r.b, id, "decider"); break;
            case kRoleDraw: mark(s.draw, r.b, id, "draw"); break;
            case kRoleBonus: mark(s.bonus, r.b, id, "bonus"); break;
            default: CHECK(false, "role %d", r.kind);
        }
    }
    // every role once, and each waiting role after what it waits on
    for (int b = 0; b < B; ++b) {
        CHECK(s.decider[b] >= 0 && s.draw[b] >= 0 && s.bonus[b] >= 0, "element %d misses a role", b);
        for (int i = 0; i < S; ++i) {
            const long long t = s.stats[(size_t)b * S + i];
            CHECK(t >= 0 && t < s.decider[b], "stats %d of element %d at %lld, decider at %lld", i, b, t, s.decider[b]);
        }
        for (int k = 0; k < p.nchunkg; ++k) {
            const long long t = s.rowg[(size_t)b * p.nchunkg + k];
            CHECK(t >= 0 && t < s.bonus[b], "row gamma tile %d of element %d", k, b);
            // in a full group of kXcds elements, on the XCD of the element's bonus workgroup
            if (b < (B & ~(kXcds - 1)))
                CHECK(t % kXcds == s.bonus[b] % kXcds, "row gamma tile %d of element %d: XCD %lld, bonus %lld", k, b,
                      t % kXcds, s.bonus[b] % kXcds);
        }
        for (int k = 0; k < p.nchunk2; ++k) {
            const long long t = s.mass[(size_t)b * p.nchunk2 + k];
            CHECK(t > s.decider[b] && t < s.draw[b], "mass tile %d of element %d between decider and draw", k, b);
        }
        CHECK(s.draw[b] > s.decider[b] && s.bonus[b] > s.decider[b], "element %d", b);
    }
}

static void simulate_staged(int B, int gamma, int V, sv_dtype_t dt) {
    Plan p{};
    CHECK(make_plan(B, gamma, V, dt, &p), "plan");
    const long long n_staged = staged_workgroups(B, gamma, V, dt, p);
    if (n_staged < 0) return;  // the single pass serves
    const int gate = gate_stages(B, V, bytes_per_logit(dt));
    CHECK(gate >= 2 && gate < gamma, "gate %d", gate);
    const Layout y = make_staged_layout(B, gamma, p.nchunk1s, p.nchunkg, p.nchunk2);
    const long long n = (long long)y.end2 + B;
    CHECK(n == n_staged, "staged grid %lld vs %lld", n, n_staged);
    const int T = 2 * p.nchunk1s;
    std::vector<long long> tile((size_t)B * gamma * T, -1), rowdec((size_t)B * gamma, -1), rowg((size_t)B * p.nchunkg, -1),
        mass((size_t)B * p.nchunk2, -1), draw(B, -1), bonus(B, -1);
    long long idle = 0;
    auto mark = [&](std::vector<long long>& v, long long i, long long id, const char* what) {
        CHECK(i >= 0 && i < (long long)v.size(), "%s index %lld out of range (id %lld)", what, i, id);
        CHECK(v[i] < 0, "%s %lld assigned twice", what, i);
        v[i] = id;
    };
    for (long long id = 0; id < n; ++id) {
        const StagedRole r = staged_role_at(y, B, gamma, p.nchunkg, (unsigned int)id);
        CHECK(r.b >= 0 && r.b < B, "element");
        switch (r.kind) {
            case kStagedTile:
                CHECK(r.c >= 0 && r.c < gamma && r.k >= 0 && r.k < T, "tile");
                mark(tile, ((long long)r.b * gamma + r.c) * T + r.k, id, "tile");
                break;
            case kStagedRowDecider:
                if (r.c < 0) {
                    ++idle;
                    break;
                }
                mark(rowdec, (long long)r.b * gamma + r.c, id, "row decider");
                break;
            case kStagedRowG: mark(rowg, (long long)r.b * p.nchunkg + r.k, id, "row gamma"); break;
            case kStagedMass: mark(mass, (long long)r.b * p.nchunk2 + r.k, id, "mass"); break;
            case kStagedDraw: mark(draw, r.b, id, "draw"); break;
            case kStagedBonus: mark(bonus, r.b, id, "bonus"); break;
            default: CHECK(false, "staged role %d", r.kind);
        }
    }
    CHECK(idle == B, "idle slots %lld (the units of stage 0 hold no row decider)", idle);
    for (int b = 0; b < B; ++b) {
        for (int c = 0; c < gamma; ++c) {
            const long long d = rowdec[(size_t)b * gamma + c];
            CHECK(d >= 0, "row decider (%d, %d) missing", b, c);
            for (int k = 0; k < T; ++k) {
                const long long t = tile[((size_t)b * gamma + c) * T + k];
                CHECK(t >= 0 && t < d, "tile (%d, %d, %d) after its row decider", b, c, k);
                // a gated tile waits on row decider (b, c - gate)
                if (c >= gate) CHECK(rowdec[(size_t)b * gamma + c - gate] < t, "gate of tile (%d, %d)", b, c);
            }
            if (c > 0) CHECK(rowdec[(size_t)b * gamma + c - 1] < d, "row decider chain (%d, %d)", b, c);
        }
        for (int k = 0; k < p.nchunkg; ++k) {
            const long long t = rowg[(size_t)b * p.nchunkg + k];
            CHECK(t >= 0 && t < bonus[b], "row gamma (%d, %d)", b, k);
            if (gamma >= gate) CHECK(rowdec[(size_t)b * gamma + gamma - gate] < t, "gate of row gamma");
        }
        const long long last = rowdec[(size_t)b * gamma + gamma - 1];
        for (int k = 0; k < p.nchunk2; ++k) {
            const long long t = mass[(size_t)b * p.nchunk2 + k];
            CHECK(t > last && t < draw[b], "mass (%d, %d)", b, k);
        }
        CHECK(bonus[b] > last, "bonus after every row decider of %d", b);
    }
}

static void section_layouts() {
    long long cases = 0;
    const int Bs[] = {1, 2, 3, 16, 64, 65, 128};
    const int gammas[] = {1, 2, 3, 5, 8, 10, 17, 33};
    const int Vs[] = {1, 7, 65, 4097, 32000, 51865, 128256};
    for (sv_dtype_t dt : kDtypes)
        for (int B : Bs)
            for (int gamma : gammas)
                for (int V : Vs) {
                    Plan p{};
                    if (!make_plan(B, gamma, V, dt, &p)) continue;
                    if (p.n_stats + p.n_mass + 3LL * B > 2000000) continue;  // keep the run short
                    simulate_single_pass(B, gamma, V, dt, true);
                    simulate_single_pass(B, gamma, V, dt, false);
                    simulate_staged(B, gamma, V, dt);
                    ++cases;
                }
    // the early exit's choice on the named exact workloads: only the largest
    // batch gates any decision row; the others run the single pass
    {
        Plan p{};
        CHECK(make_plan(1, 5, 51865, SV_F32, &p) && staged_workgroups(1, 5, 51865, SV_F32, p) < 0, "B=1 fp32");
        CHECK(make_plan(1, 10, 32000, SV_F16, &p) && staged_workgroups(1, 10, 32000, SV_F16, p) < 0, "B=1 fp16");
        CHECK(make_plan(16, 5, 51865, SV_F32, &p) && staged_workgroups(16, 5, 51865, SV_F32, p) < 0, "B=16");
        CHECK(make_plan(64, 8, 128256, SV_BF16, &p) && staged_workgroups(64, 8, 128256, SV_BF16, p) > 0, "B=64");
        CHECK(gate_stages(64, 128256, 2) == 2, "gate at the headline shape");
        for (int V : {1, 2, 7, 65, 300007})
            for (sv_dtype_t dt : kDtypes)
                CHECK(make_plan(3, 3, V, dt, &p) && staged_workgroups(3, 3, V, dt, p) < 0, "B=3 V=%d", V);
    }
    // the gated staged shapes the tests run, and the limits of gamma
    simulate_staged(64, 8, 128256, SV_BF16);
    simulate_staged(128, 8, 128256, SV_BF16);
    simulate_staged(64, 128, 4097, SV_F32);
    simulate_single_pass(2, 128, 2049, SV_F16, true);
    simulate_single_pass(1, 1, 1 << 21, SV_BF16, true);
    simulate_single_pass(1, 3, 1 << 20, SV_F32, true);
    printf("layouts: ok (%lld shapes in both modes)\n", cases);
}

// --- 4. validation -------------------------------------------------------------

static Call base_call() {
    Call a{};
    a.draft = (const void*)0x1000;
    a.target = (const void*)0x2000;
    a.dt = SV_F32;
    a.tokens = (const int32_t*)0x3000;
    a.uniforms = (const float*)0x4000;
    a.B = 2;
    a.gamma = 3;
    a.V = 100;
    a.temperature = 1.0f;
    a.alpha = -1.0e4f;
    a.beta = 1.0e4f;
    a.accepted_len = (int32_t*)0x5000;
    a.next_token = (int32_t*)0x6000;
    a.ws = (void*)0x7000;
    a.ws_bytes = 1 << 20;
    a.stream = nullptr;
    return a;
}

static sv_status_t val(const Call& a, bool exact) {
    Plan p{};
    return validate(a, exact, &p);
}

// Which single passes wait with two polls in flight: the short streams of
// the small workloads, not the long stream of the large one.
static void section_pipelined_waits() {
    CHECK(pipelined_waits(1, 5, 51865, SV_F32) && pipelined_waits(1, 10, 32000, SV_F16) &&
              pipelined_waits(16, 5, 51865, SV_F32),
          "short streams");
    CHECK(!pipelined_waits(64, 8, 128256, SV_BF16) && !pipelined_waits(56, 3, 128256, SV_BF16), "long streams");
    for (long long B : {1LL, 7LL, 64LL})
        for (long long g : {1LL, 8LL, 128LL})
            for (long long V : {1LL, 4097LL, 1LL << 20})
                CHECK(pipelined_waits(B, g, V, SV_F32) == (2 * g * V * 4 * B < kLagStreamBytes), "rule");
    // which short streams' mass workgroups decide for themselves (pair
    // copies): the named B = 1 fp16 workload and the reduced test shapes do,
    // the named B = 1 and B = 16 fp32 workloads wait for the decider's record
    Plan p{};
    CHECK(make_plan(1, 10, 32000, SV_F16, &p) && p.qstride == 4LL * 10 * p.nchunk1, "B=1 fp16 copies");
    CHECK(make_plan(1, 5, 9001, SV_F32, &p) && p.qstride > 0, "reduced B=1 fp32 copies");
    CHECK(make_plan(1, 5, 51865, SV_F32, &p) && p.qstride == 0, "B=1 fp32 record");
    CHECK(make_plan(16, 5, 51865, SV_F32, &p) && p.qstride == 0, "B=16 fp32 record");
    CHECK(make_plan(64, 8, 128256, SV_BF16, &p) && p.qstride == 0, "long stream: no copies");
    printf("pipelined waits: ok\n");
}

// The decoding loop's automatic early exit: below half of gamma accepted on
// average (hand-worked cases, the same as the Python loop's tests).
static void section_loop_early_exit() {
    CHECK(early_exit_pays(11, 4, 8), "mean 2.75 < 4");
    CHECK(!early_exit_pays(16, 4, 8), "mean 4 is not below 4");
    CHECK(!early_exit_pays(24, 4, 8), "mean 6");
    CHECK(early_exit_pays(0, 64, 1), "nothing accepted at gamma 1");
    CHECK(!early_exit_pays(32, 64, 1), "half accepted at gamma 1");
    CHECK(early_exit_pays(31, 64, 1), "just under half");
    CHECK(!early_exit_pays(0, 0, 8), "empty batch");
    printf("loop early exit: ok\n");
}

static void section_validation() {
    const float inf = std::numeric_limits<float>::infinity();
    const float nan = std::numeric_limits<float>::quiet_NaN();
    for (bool exact : {true, false}) {
        CHECK(val(base_call(), exact) == SV_OK, "valid call");
        Call a = base_call(); a.draft = nullptr; CHECK(val(a, exact) == SV_ERR_NULL, "draft");
        a = base_call(); a.target = nullptr; CHECK(val(a, exact) == SV_ERR_NULL, "target");
        a = base_call(); a.tokens = nullptr; CHECK(val(a, exact) == SV_ERR_NULL, "tokens");
        a = base_call(); a.uniforms = nullptr; CHECK(val(a, exact) == SV_ERR_NULL, "uniforms");
        a = base_call(); a.accepted_len = nullptr; CHECK(val(a, exact) == SV_ERR_NULL, "accepted_len");
        a = base_call(); a.next_token = nullptr; CHECK(val(a, exact) == SV_ERR_NULL, "next_token");
        a = base_call(); a.ws = nullptr; CHECK(val(a, exact) == SV_ERR_NULL, "ws");
        a = base_call(); a.dt = (sv_dtype_t)7; CHECK(val(a, exact) == SV_ERR_DTYPE, "dtype");
        a = base_call(); a.dt = (sv_dtype_t)-1; CHECK(val(a, exact) == SV_ERR_DTYPE, "dtype");
        for (int B : {0, -1, -2147483647 - 1}) { a = base_call(); a.B = B; CHECK(val(a, exact) == SV_ERR_SHAPE, "B=%d", B); }
        for (int g : {0, -1, 129, 2147483647}) { a = base_call(); a.gamma = g; CHECK(val(a, exact) == SV_ERR_SHAPE, "gamma=%d", g); }
        for (int V : {0, -5, (1 << 21) + 1, 2147483647}) { a = base_call(); a.V = V; a.dt = SV_BF16; CHECK(val(a, exact) == SV_ERR_SHAPE, "V=%d", V); }
        a = base_call(); a.V = (1 << 20) + 1; CHECK(val(a, exact) == SV_ERR_SHAPE, "fp32 V past 2^20");
        a = base_call(); a.B = 2147483647; a.gamma = 128; a.V = 1 << 20; CHECK(val(a, exact) == SV_ERR_SHAPE, "huge");
        for (float T : {0.0f, -1.0f, nan, inf, -inf, 1e-40f}) {
            a = base_call(); a.temperature = T; CHECK(val(a, exact) == SV_ERR_PARAM, "T=%g", (double)T);
        }
        a = base_call(); a.ws_bytes = 0; CHECK(val(a, exact) == SV_ERR_WORKSPACE, "ws bytes");
        Plan p{};
        CHECK(make_plan(2, 3, 100, SV_F32, &p), "plan");
        a = base_call(); a.ws_bytes = p.bytes - 1; CHECK(val(a, exact) == SV_ERR_WORKSPACE, "ws one short");
        a = base_call(); a.ws_bytes = p.bytes; CHECK(val(a, exact) == SV_OK, "ws exact");
        a = base_call(); a.ws = (void*)0x7008; CHECK(val(a, exact) == SV_ERR_WORKSPACE, "ws misaligned");
    }
    // sigmoid constants
    for (auto ab : {std::pair<float, float>{1.0f, 1.0f}, {2.0f, 1.0f}, {std::numeric_limits<float>::quiet_NaN(), 1.0f},
                    {-std::numeric_limits<float>::infinity(), 1.0f}, {0.0f, std::numeric_limits<float>::infinity()},
                    {0.0f, 1e-45f}}) {
        Call a = base_call();
        a.alpha = ab.first;
        a.beta = ab.second;
        CHECK(val(a, false) == SV_ERR_PARAM, "alpha=%g beta=%g", (double)ab.first, (double)ab.second);
        CHECK(val(a, true) == SV_OK, "exact mode ignores alpha/beta");
    }
    {
        Call a = base_call();
        a.temperature = 2e-38f;  // log2(e) / T fits fp32, 1 / (T (beta - alpha)) does not
        a.alpha = 0.0f;
        a.beta = 0.01f;
        CHECK(val(a, true) == SV_OK, "exact mode at a tiny temperature");
        CHECK(val(a, false) == SV_ERR_PARAM, "sigmoid scale overflow");
    }
    printf("validation: ok\n");
}

int main() {
    section_div();
    section_plans();
    section_layouts();
    section_pipelined_waits();
    section_loop_early_exit();
    section_validation();
    printf("all checks passed (%lld)\n", g_checks);
    return 0;
}
