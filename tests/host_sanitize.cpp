// Host-side checks of libmsda under AddressSanitizer and UndefinedBehaviorSanitizer, on the CPU.
//
// Built by tests/test_host_sanitize.py with the sanitizers on the host code only. Everything called
// here runs on the host and makes no GPU call: the argument checks, the workspace sizing (the
// owner-computes plan: tile sizes, bins, work items and byte counts per level), the error paths of
// every entry point that reject a call before anything is enqueued, the chunk table of the band
// arrangement of the forward and backward kernels, and the status strings.
// Random problems come from a fixed-seed generator; the program prints one line per group of
// checks and exits non-zero if a check fails (a sanitizer report aborts it).
#include <cstdint>
#include <cstdio>
#include <vector>

#include "msda.h"
#include "msda_internal.h"

namespace {

uint64_t g_state = 0x9E3779B97F4A7C15ull;

// splitmix64
uint64_t next_u64() {
    uint64_t z = (g_state += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

int64_t uniform(int64_t lo, int64_t hi) { return lo + (int64_t)(next_u64() % (uint64_t)(hi - lo + 1)); }

struct Problem {
    std::vector<int64_t> shapes, starts;
    int64_t N, S, M, D, Lq, L, P;
    int dtype;
};

Problem random_problem() {
    Problem p;
    p.L = uniform(1, MSDA_MAX_LEVELS);
    p.S = 0;
    for (int64_t l = 0; l < p.L; ++l) {
        const int64_t H = uniform(1, 80), W = uniform(1, 80);
        p.shapes.push_back(H);
        p.shapes.push_back(W);
        p.starts.push_back(p.S);
        p.S += H * W;
    }
    p.N = uniform(0, 4);
    p.M = uniform(1, 12);
    p.D = uniform(1, 300);
    p.Lq = uniform(0, 3000);
    p.P = uniform(1, 9);
    p.dtype = uniform(0, 1) ? MSDA_F16 : MSDA_F32;
    return p;
}

int g_failures = 0;

void expect(bool ok, const char* what, int64_t i) {
    if (!ok) {
        ++g_failures;
        std::printf("FAILED: %s (problem %lld): %s\n", what, (long long)i, msda_last_error());
    }
}

}  // namespace

int main() {
    // 1. valid problems: the checks accept them and every workspace mode sizes them
    const int kProblems = 400;
    int sized = 0;
    for (int i = 0; i < kProblems; ++i) {
        const Problem p = random_problem();
        const msda_status_t st = msda_check_args(p.shapes.data(), p.starts.data(), p.N, p.S, p.M, p.D, p.Lq, p.L,
                                                 p.P, p.dtype);
        expect(st == MSDA_SUCCESS, "valid problem accepted", i);
        for (int mode : {MSDA_WORKSPACE_PREFERRED, MSDA_WORKSPACE_OWNER, MSDA_WORKSPACE_DETERMINISTIC}) {
            size_t plain = 1, fused = 1;
            const msda_status_t a = msda_backward_workspace_size(p.shapes.data(), p.starts.data(), p.N, p.S, p.M,
                                                                 p.D, p.Lq, p.L, p.P, p.dtype, mode, &plain);
            const msda_status_t b = msda_backward_fused_workspace_size(p.shapes.data(), p.starts.data(), p.N, p.S,
                                                                       p.M, p.D, p.Lq, p.L, p.P, p.dtype, mode,
                                                                       &fused);
            expect(a == MSDA_SUCCESS || a == MSDA_ERROR_NOT_SUPPORTED, "workspace size", i);
            expect(b == MSDA_SUCCESS || b == MSDA_ERROR_NOT_SUPPORTED, "fused workspace size", i);
            if (a == MSDA_SUCCESS && b == MSDA_SUCCESS) {
                expect(fused >= plain, "fused workspace holds the plain one", i);
                ++sized;
            }
        }
    }
    std::printf("valid problems: %d, workspace sizes: %d\n", kProblems, sized);

    // 2. invalid problems: each is rejected with a status, never accepted
    int rejected = 0;
    for (int i = 0; i < kProblems; ++i) {
        Problem p = random_problem();
        switch (i % 7) {
            case 0: p.S += 1; break;                                      // S differs from sum H*W
            case 1: if (p.L > 1) p.starts[p.L - 1] += 1; else p.S = -1; break;  // wrong start
            case 2: p.M = 0; break;
            case 3: p.D = -uniform(0, 5); break;
            case 4: p.P = 0; break;
            case 5: p.shapes[0] = 0; break;                               // empty level
            default: p.dtype = 7; break;                                  // unknown dtype
        }
        const msda_status_t st = msda_check_args(p.shapes.data(), p.starts.data(), p.N, p.S, p.M, p.D, p.Lq, p.L,
                                                 p.P, p.dtype);
        expect(st != MSDA_SUCCESS, "invalid problem rejected", i);
        size_t bytes = 0;
        const msda_status_t w = msda_backward_workspace_size(p.shapes.data(), p.starts.data(), p.N, p.S, p.M, p.D,
                                                             p.Lq, p.L, p.P, p.dtype, MSDA_WORKSPACE_OWNER, &bytes);
        expect(w != MSDA_SUCCESS, "invalid problem not sized", i);
        rejected += st != MSDA_SUCCESS;
    }
    std::printf("invalid problems rejected: %d of %d\n", rejected, kProblems);
    // more levels than the build supports, and null tables
    {
        std::vector<int64_t> shapes(2 * (MSDA_MAX_LEVELS + 1), 2), starts(MSDA_MAX_LEVELS + 1);
        for (int l = 0; l <= MSDA_MAX_LEVELS; ++l) starts[l] = 4 * l;
        expect(msda_check_args(shapes.data(), starts.data(), 1, 4 * (MSDA_MAX_LEVELS + 1), 1, 1, 1,
                               MSDA_MAX_LEVELS + 1, 1, MSDA_F32) == MSDA_ERROR_NOT_SUPPORTED,
               "too many levels", 0);
        expect(msda_check_args(nullptr, starts.data(), 1, 4, 1, 1, 1, 1, 1, MSDA_F32) == MSDA_ERROR_INVALID_VALUE,
               "null level table", 0);
        expect(msda_backward_workspace_size(shapes.data(), starts.data(), 1, 4, 1, 1, 1, 1, 1, MSDA_F32,
                                            MSDA_WORKSPACE_OWNER, nullptr) == MSDA_ERROR_INVALID_VALUE,
               "null size pointer", 0);
    }

    // 3. entry points with null buffers (nonzero extent) are rejected before anything is enqueued
    {
        const int64_t shapes[4] = {4, 5, 2, 3}, starts[2] = {0, 20};
        const int64_t N = 2, S = 26, M = 3, D = 8, Lq = 7, L = 2, P = 2;
        expect(msda_forward(nullptr, shapes, starts, nullptr, nullptr, nullptr, N, S, M, D, Lq, L, P, MSDA_F32,
                            nullptr) == MSDA_ERROR_INVALID_VALUE, "forward nulls", 0);
        expect(msda_backward(nullptr, shapes, starts, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                             0, N, S, M, D, Lq, L, P, MSDA_F32, nullptr) == MSDA_ERROR_INVALID_VALUE,
               "backward nulls", 0);
        expect(msda_backward_atomic(nullptr, shapes, starts, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, N,
                                    S, M, D, Lq, L, P, MSDA_F32, nullptr) == MSDA_ERROR_INVALID_VALUE,
               "atomic backward nulls", 0);
        expect(msda_backward_deterministic(nullptr, shapes, starts, nullptr, nullptr, nullptr, nullptr, nullptr,
                                           nullptr, nullptr, 0, N, S, M, D, Lq, L, P, MSDA_F32,
                                           nullptr) == MSDA_ERROR_INVALID_VALUE,
               "deterministic backward nulls", 0);
        expect(msda_forward_fused(nullptr, shapes, starts, nullptr, nullptr, nullptr, nullptr, N, S, M, D, Lq, L, P,
                                  MSDA_F32, nullptr) == MSDA_ERROR_INVALID_VALUE, "fused forward nulls", 0);
        expect(msda_backward_fused(nullptr, shapes, starts, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                                   nullptr, nullptr, nullptr, 0, N, S, M, D, Lq, L, P, MSDA_F32,
                                   nullptr) == MSDA_ERROR_INVALID_VALUE,
               "fused backward nulls", 0);
        // a bad level table is reported before the pointers are looked at
        const int64_t bad_starts[2] = {0, 21};
        expect(msda_forward(nullptr, shapes, bad_starts, nullptr, nullptr, nullptr, N, S, M, D, Lq, L, P, MSDA_F32,
                            nullptr) == MSDA_ERROR_INVALID_VALUE, "forward bad table", 0);
    }

    // 4. the band arrangement's chunk table: every query chunk of a level-major pixel order lies in exactly
    //    one (level, band) range, the band of its first query's row floor(8 (h + 1/2) / H), counted in its
    //    band; checked by brute force over random level tables and chunk sizes
    int tables = 0;
    for (int i = 0; i < kProblems; ++i) {
        const Problem pr = random_problem();
        msda::Params p = {};
        p.L = (int)pr.L;
        for (int64_t l = 0; l < pr.L; ++l) {
            p.H[l] = (int)pr.shapes[2 * l];
            p.W[l] = (int)pr.shapes[2 * l + 1];
            p.start[l] = (int)pr.starts[l];
        }
        p.q_per_block = 1 << uniform(0, 8);
        msda::set_bands(p);
        const int64_t qpb = p.q_per_block, chunks = (pr.S + qpb - 1) / qpb;
        std::vector<int> band(chunks, -1);
        int counted[8] = {0}, cap = 0;
        bool ok = true;
        for (int l = 0; l < p.L && ok; ++l)
            for (int x = 0; x < 8 && ok; ++x)
                for (int c = p.band_c[l][x]; c < p.band_c[l][x + 1] && ok; ++c) {
                    const int64_t q = c * qpb, rel = q - p.start[l];
                    ok = c >= 0 && c < chunks && band[c] < 0 && rel >= 0 && rel < (int64_t)p.H[l] * p.W[l] &&
                         (8 * (rel / p.W[l]) + 4) / p.H[l] == x;
                    if (ok) {
                        band[c] = x;
                        ++counted[x];
                    }
                }
        for (int64_t c = 0; c < chunks && ok; ++c) ok = band[c] >= 0;
        for (int x = 0; x < 8 && ok; ++x) {
            ok = counted[x] == p.band_count[x];
            if (counted[x] > cap) cap = counted[x];
        }
        expect(ok && cap == p.band_cap, "band table partitions the query chunks", i);
        tables += ok;
    }
    std::printf("band tables checked: %d of %d\n", tables, kProblems);

    // 5. status strings and the version
    for (int s = -1; s <= 4; ++s) expect(msda_status_string(s) != nullptr, "status string", s);
    expect(msda_version() > 0, "version", 0);

    std::printf("failures: %d\n", g_failures);
    return g_failures == 0 ? 0 : 1;
}
