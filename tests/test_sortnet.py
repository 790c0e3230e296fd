"""The routing kernel's compile-time sorting network (csrc/sortnet.h), checked on the host:
compiled with g++ into a small program that applies the network (descending compare-
exchanges) and verifies the output is sorted, exhaustively over all 0/1 inputs for
NP <= 16 (the 0-1 principle makes that a proof for those sizes) and on random inputs up to
NP = 64; likewise the phased order of the same comparators (each part sorted alone first,
then the merges across parts), which the routing kernel runs as its input arrives."""
import os
import subprocess
import tempfile

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

PROG = r'''
#include <cstdio>
#include <cstdlib>
#include <random>
#include "sortnet.h"
template <int NP> int check(bool exhaustive) {
    constexpr elb::OddEvenMergeNet<NP> net{};
    std::mt19937 rng(NP);
    long cases = exhaustive ? (1L << NP) : 200000;
    for (long c = 0; c < cases; ++c) {
        float v[NP];
        for (int i = 0; i < NP; ++i)
            v[i] = exhaustive ? (float)((c >> i) & 1) : (float)(rng() % 50);
        for (int q = 0; q < net.n; ++q) {
            float a = v[net.a[q]], b = v[net.b[q]];
            v[net.a[q]] = a > b ? a : b;
            v[net.b[q]] = a > b ? b : a;
        }
        for (int i = 1; i < NP; ++i) if (v[i - 1] < v[i]) { printf("FAIL %d\n", NP); return 1; }
    }
    printf("NP=%d comparators=%d ok\n", NP, net.n);
    return 0;
}
// the phased order: each part's group sorts that part alone (checked right after it runs),
// and all groups in order sort the whole input
template <int NP, int P> int check_phased(bool exhaustive) {
    constexpr elb::OddEvenMergeNet<NP> net{};
    constexpr elb::PhasedNet<NP, P> ph{};
    constexpr int B = NP / P;
    int total = 0;
    for (int g = 0; g <= P; ++g) total += ph.cnt[g];
    if (total != net.n) { printf("FAIL phased count %d/%d\n", NP, P); return 1; }
    std::mt19937 rng(NP * 7 + P);
    long cases = exhaustive ? (1L << NP) : 200000;
    for (long c = 0; c < cases; ++c) {
        float v[NP];
        for (int i = 0; i < NP; ++i)
            v[i] = exhaustive ? (float)((c >> i) & 1) : (float)(rng() % 50);
        for (int g = 0; g <= P; ++g) {
            for (int q = 0; q < ph.cnt[g]; ++q) {
                const int x = ph.idx[g][q];
                float a = v[net.a[x]], b = v[net.b[x]];
                v[net.a[x]] = a > b ? a : b;
                v[net.b[x]] = a > b ? b : a;
            }
            if (g < P)
                for (int i = g * B + 1; i < g * B + B; ++i)
                    if (v[i - 1] < v[i]) { printf("FAIL phased part %d/%d\n", NP, P); return 1; }
        }
        for (int i = 1; i < NP; ++i)
            if (v[i - 1] < v[i]) { printf("FAIL phased %d/%d\n", NP, P); return 1; }
    }
    printf("NP=%d P=%d phased ok\n", NP, P);
    return 0;
}
int main() {
    return check<2>(true) | check<4>(true) | check<8>(true) | check<16>(true) |
           check<32>(false) | check<64>(false) | check_phased<16, 4>(true) |
           check_phased<16, 2>(true) | check_phased<32, 4>(false) | check_phased<64, 4>(false);
}
'''


def test_sorting_network_sorts():
    with tempfile.TemporaryDirectory() as d:
        src = os.path.join(d, "t.cpp")
        exe = os.path.join(d, "t")
        open(src, "w").write(PROG)
        subprocess.check_call(["g++", "-O2", "-std=c++17", "-I",
                               os.path.join(ROOT, "paper_2608_04401_amd", "csrc"), src, "-o", exe])
        out = subprocess.run([exe], stdout=subprocess.PIPE, text=True, check=True).stdout
    assert "NP=64 comparators=543 ok" in out
    assert "NP=64 P=4 phased ok" in out and "NP=16 P=4 phased ok" in out
    assert "FAIL" not in out
