// Batcher's odd-even merge sorting network for a compile-time power-of-two size NP,
// generated at compile time so that every comparator's two positions are constants after
// unrolling (the data stays in registers; no dynamic register indexing).
// Usable from host code (for tests) and device code.
#pragma once

#if defined(__HIPCC__)
#define ELB_HD __host__ __device__
#else
#define ELB_HD
#endif

namespace elb {

template <int NP>
struct OddEvenMergeNet {
    static_assert(NP >= 2 && (NP & (NP - 1)) == 0, "power of two");
    static constexpr int kMax = NP * 12;  // >= comparators for NP <= 64 (543 at NP = 64)
    int a[kMax];
    int b[kMax];
    int n;
    constexpr OddEvenMergeNet() : a(), b(), n(0) {
        for (int p = 1; p < NP; p += p)
            for (int k = p; k > 0; k /= 2)
                for (int j = k % p; j + k < NP; j += k + k)
                    for (int i = 0; i < k && i + j + k < NP; ++i)
                        if ((i + j) / (p + p) == (i + j + k) / (p + p)) {
                            a[n] = i + j;
                            b[n] = i + j + k;
                            ++n;
                        }
    }
};

}  // namespace elb
