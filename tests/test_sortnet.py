"""The routing kernel's compile-time sorting network (csrc/sortnet.h), checked on the host:
compiled with g++ into a small program that applies the network (descending compare-
exchanges) and verifies the output is sorted, exhaustively over all 0/1 inputs for
NP <= 16 (the 0-1 principle makes that a proof for those sizes) and on random inputs up to
NP = 64."""
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
int main() {
    return check<2>(true) | check<4>(true) | check<8>(true) | check<16>(true) |
           check<32>(false) | check<64>(false);
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
    assert "FAIL" not in out
