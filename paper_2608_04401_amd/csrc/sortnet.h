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
    int lvl[kMax];  // merge level p of the comparator: it lies inside one aligned 2p-block
    int n;
    constexpr OddEvenMergeNet() : a(), b(), lvl(), n(0) {
        for (int p = 1; p < NP; p += p)
            for (int k = p; k > 0; k /= 2)
                for (int j = k % p; j + k < NP; j += k + k)
                    for (int i = 0; i < k && i + j + k < NP; ++i)
                        if ((i + j) / (p + p) == (i + j + k) / (p + p)) {
                            a[n] = i + j;
                            b[n] = i + j + k;
                            lvl[n] = p;
                            ++n;
                        }
    }
};

// The same network split into P + 1 groups for data that arrives in P parts (positions
// [q B, q B + B), B = NP / P): group q < P holds, in network order, the comparators of
// levels below B inside part q -- the sorting network of that part alone, runnable as soon
// as the part is present -- and group P the remaining levels (the merges across parts).
// Comparators of different parts at levels below B are independent, so running the groups
// in order sorts exactly as the whole network does.
template <int NP, int P>
struct PhasedNet {
    static_assert(P >= 1 && NP % P == 0 && ((NP / P) & (NP / P - 1)) == 0, "parts");
    static constexpr int B = NP / P;
    static constexpr int kMax = OddEvenMergeNet<NP>::kMax;
    int idx[P + 1][kMax];  // comparator indices into OddEvenMergeNet<NP>
    int cnt[P + 1];
    constexpr PhasedNet() : idx(), cnt() {
        constexpr OddEvenMergeNet<NP> net{};
        for (int g = 0; g <= P; ++g) cnt[g] = 0;
        for (int c = 0; c < net.n; ++c) {
            const int g = (net.lvl[c] < B) ? net.a[c] / B : P;
            idx[g][cnt[g]++] = c;
        }
    }
};

}  // namespace elb
