// Randomised exercise of the host-side schedule builders (ta_build_schedule,
// ta_build_blocksparse_schedule) under AddressSanitizer and UBSan: valid shapes
// must build into exactly info.words words, a one-word-short buffer must be
// rejected, and malformed inputs must be rejected without any out-of-range
// access.  Compiled with g++ for the host only (tests/test_host_sanitizers.py).

#include <cstdio>
#include <cstdlib>
#include <cstdint>
#include <random>
#include <vector>
#include "triattn.h"

#ifndef ITERS
#define ITERS 3000
#endif

static std::mt19937_64 rng(12345);
static int ri(int lo, int hi) { return std::uniform_int_distribution<int>(lo, hi)(rng); }

int main()
{
    long ok = 0, rejected = 0;
    for (int it = 0; it < ITERS; ++it) {
        const int batch = ri(0, 5);
        std::vector<int32_t> cu(batch + 1, 0);
        for (int b = 0; b < batch; ++b) {
            int n = ri(0, 3) == 0 ? ri(0, 3) : ri(1, it % 50 == 0 ? 200000 : 3000);
            cu[b + 1] = cu[b] + n;
        }
        const int kind = ri(0, 1) ? TA_KIND_TRIANGLE : TA_KIND_CAUSAL;
        const int tile = ri(0, 1) ? 64 : 128;
        const int sink = ri(0, 3) == 0 ? 0 : ri(0, 300);
        const int window = ri(1, 3000);
        const int last = ri(0, 3) == 0 ? 0 : ri(0, 400);
        const int splits = ri(0, 4) == 0 ? ri(1, 600) : 0;
        ta_schedule_info info{};
        ta_status st = ta_build_schedule(kind, cu.data(), batch, sink, window, last, tile, splits,
                                         nullptr, 0, &info);
        if (st != TA_OK) { ++rejected; continue; }
        int32_t *out = new int32_t[info.words];
        st = ta_build_schedule(kind, cu.data(), batch, sink, window, last, tile, splits, out,
                               info.words, &info);
        if (st != TA_OK) { printf("second call failed: %s\n", ta_last_error()); return 1; }
        (void)ta_workspace_bytes(&info, 32, 128);
        delete[] out;
        // a too-small buffer must be rejected, not overrun
        if (info.words > 1) {
            int32_t *small = new int32_t[info.words - 1];
            st = ta_build_schedule(kind, cu.data(), batch, sink, window, last, tile, splits, small,
                                   info.words - 1, &info);
            if (st == TA_OK) { printf("short buffer accepted\n"); return 1; }
            delete[] small;
        }
        // block-sparse lists over the same sequences
        std::vector<int32_t> ptr(1, 0), idx;
        for (int b = 0; b < batch; ++b) {
            const int n = cu[b + 1] - cu[b];
            const int nq = (n + tile - 1) / tile;
            for (int t = 0; t < nq; ++t) {
                for (int k = 0; k <= t; ++k)
                    if (k == t || ri(0, 9) == 0)
                        idx.push_back(k);
                ptr.push_back((int32_t)idx.size());
            }
        }
        const int bound = ri(0, 2) == 0 ? ri(1, 40) : 0;
        st = ta_build_blocksparse_schedule(cu.data(), batch, tile, ptr.data(),
                                           idx.empty() ? nullptr : idx.data(), bound, nullptr, 0,
                                           &info);
        if (st != TA_OK) { ++rejected; continue; }
        out = new int32_t[info.words];
        st = ta_build_blocksparse_schedule(cu.data(), batch, tile, ptr.data(),
                                           idx.empty() ? nullptr : idx.data(), bound, out,
                                           info.words, &info);
        if (st != TA_OK) { printf("blocksparse second call failed: %s\n", ta_last_error()); return 1; }
        delete[] out;
        ++ok;
    }
    // malformed inputs: must be rejected without any out-of-range access
    long bad_rej = 0, bad_ok = 0;
    for (int it = 0; it < ITERS; ++it) {
        const int batch = ri(1, 4);
        std::vector<int32_t> cu(batch + 1, 0);
        for (int b = 0; b < batch; ++b)
            cu[b + 1] = cu[b] + ri(1, 2000);
        const int tile = ri(0, 1) ? 64 : 128;
        std::vector<int32_t> ptr(1, 0), idx;
        for (int b = 0; b < batch; ++b) {
            const int nq = (cu[b + 1] - cu[b] + tile - 1) / tile;
            for (int t = 0; t < nq; ++t) {
                for (int k = 0; k <= t; ++k)
                    if (k == t || ri(0, 5) == 0)
                        idx.push_back(k);
                ptr.push_back((int32_t)idx.size());
            }
        }
        const int mode = ri(0, 5);
        if (mode == 0 && batch > 1) std::swap(cu[1], cu[2]);             // decreasing
        if (mode == 1 && !idx.empty()) idx[ri(0, (int)idx.size() - 1)] = ri(-5, 100000);  // bad index
        if (mode == 2 && idx.size() > 1) { size_t a = ri(0, (int)idx.size() - 2); std::swap(idx[a], idx[a + 1]); }
        if (mode == 3 && ptr.size() > 2) { size_t a = ri(1, (int)ptr.size() - 2); ptr[a] = ptr[a + 1] + 1 <= (int)idx.size() ? ptr[a + 1] + 1 : ptr[a]; }
        if (mode == 4) cu[0] = ri(1, 5);
        ta_schedule_info info{};
        ta_status st = ta_build_blocksparse_schedule(cu.data(), batch, tile, ptr.data(),
                                                     idx.empty() ? nullptr : idx.data(), 0,
                                                     nullptr, 0, &info);
        if (st != TA_OK) { ++bad_rej; continue; }
        int32_t *out = new int32_t[info.words];
        st = ta_build_blocksparse_schedule(cu.data(), batch, tile, ptr.data(),
                                           idx.empty() ? nullptr : idx.data(), 0, out, info.words,
                                           &info);
        delete[] out;
        ++bad_ok;
        st = ta_build_schedule(TA_KIND_TRIANGLE, cu.data(), batch, ri(-2, 50), ri(-2, 500),
                               ri(-2, 100), ri(0, 1) ? 64 : 96, ri(-2, 5), nullptr, 0, &info);
        (void)st;
    }
    printf("malformed: rejected %ld accepted %ld\n", bad_rej, bad_ok);
    printf("ok %ld rejected %ld\n", ok, rejected);
    return 0;
}
