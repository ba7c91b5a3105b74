// Host-only fuzz driver for the launch planner (igemm_plan.cpp, no HIP):
// random and extreme extents, leading dimensions, alignments, kernels, k-slice
// counts and convolution descriptors, validated the way the entry points
// validate them. Built and run under the undefined-behaviour and address
// sanitizers by tests/test_host_sanitizers.py.
#include <cstdio>
#include <cstdint>
#include <random>
#include "igemm_internal.h"
using namespace igemm;
int main() {
    std::mt19937_64 rng(1);
    const int64_t big[] = {0, 1, 2, 7, 63, 64, 65, 255, 256, 1000, 4096, 32768, 32769, 70000,
                           (1LL << 31) - 1, 1LL << 31, 1LL << 40, 1LL << 62, -1, -5};
    auto pick = [&](bool ext) -> int64_t {
        if (ext || rng() % 5 == 0) return big[rng() % (sizeof(big) / sizeof(big[0]))];
        return (int64_t)(rng() % 5000);
    };
    int ok = 0, bad = 0;
    for (int it = 0; it < 100000; ++it) {
        const int es = 1 + (int)(rng() % 2);
        int64_t m = pick(false), n = pick(false), k = pick(false);
        int64_t lda = k + (int64_t)(rng() % 3), ldb = n + (int64_t)(rng() % 3), ldc = n;
        const void *A = (const void *)(uintptr_t)(0x10000 + rng() % 17);
        igemm_plan p;
        int kernel = (int)(rng() % (K_COUNT + 1)) - 1;
        int split = (int)(rng() % 6) - 1;
        int st = validate(es, m, n, k, A, lda, A, ldb, A, ldc);
        if (st == IGEMM_OK) st = make_plan(es, m, n, k, A, lda, A, ldb, ldc, 256, kernel, split, true, &p);
        (st == IGEMM_OK ? ok : bad)++;
        igemm_conv2d_desc d;
        d.n = pick(false) % 5; d.h = pick(false); d.w = pick(false); d.c = pick(false);
        d.k = pick(false); d.r = pick(false) % 9; d.s = pick(false) % 9;
        d.stride_h = pick(false) % 5; d.stride_w = pick(false) % 5; d.pad_h = pick(false) % 7;
        d.pad_w = pick(false) % 7; d.dil_h = pick(false) % 4; d.dil_w = pick(false) % 4;
        if (rng() % 10 == 0) { d.n = pick(true); d.h = pick(true); d.pad_w = pick(true); d.dil_h = pick(true); d.c = pick(true); }
        ConvGeom g; int gather;
        st = make_conv_plan(es, &d, A, A, A, 256, -1, -1, &p, &g, &gather);
        (st == IGEMM_OK ? ok : bad)++;
        st = validate(es, m, n, k, A, lda, A, ldb, A, ldc);
        if (st == IGEMM_OK && m > 0 && n > 0 && k > 0)
            st = make_srs_plan(es, m, n, k, A, lda, A, ldb, ldc, 256, -1, &p);
        (st == IGEMM_OK ? ok : bad)++;
        (void)conv_out_dim(pick(true), pick(true), pick(true), pick(true), pick(true));
    }
    std::printf("ok %d bad %d\n", ok, bad);
    return 0;
}
