"""The combine kernel's summation of a long segment's pieces, checked on the CPU.

The kernel sums whole aligned runs of 16 pieces as fixed trees (two runs at
once joined into a run of 32 on rows that allow it) and pushes each run into a
pairwise counter at its level, then adds the last pieces one by one with the
counter's low levels known at compile time.  That must give, bit for bit, the
pairwise (binary-counter) sum of the pieces one by one.  The helpers are taken
from the kernel source as written, compiled for the host with g++, and compared
with a plain counter written here, for every piece count up to 300 and a spread
of larger ones (beyond 2^12 pieces the counter's top accumulator is used).
"""
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "paper_2512_23236_amd", "csrc", "tbe_backward.hip")

HEADER = r"""
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <random>
#include <vector>
struct float4 { float x, y, z, w; };
inline float4 make_float4(float a, float b, float c, float d) { return float4{a, b, c, d}; }
constexpr int kPairLevels = 12;
"""

MAIN = r"""
// pairwise sum of p in order, pushing one piece at a time
static float counter_sum(const std::vector<float> &p) {
    float st[kPairLevels];
    float top = 0.f;
    bool top_used = false;
    uint32_t n = 0;
    for (float x : p) {
        int l = 0;
        for (; l < kPairLevels && ((n >> l) & 1u); ++l) x = st[l] + x;
        if (l < kPairLevels) st[l] = x;
        else { top = top_used ? top + x : x; top_used = true; }
        ++n;
    }
    float sum = top;
    bool have = top_used;
    for (int l = kPairLevels - 1; l >= 0; --l)
        if ((n >> l) & 1u) { sum = have ? sum + st[l] : st[l]; have = true; }
    return sum;
}

// the kernel's order: runs of 2 kB (pairs) while they fit, single runs of kB,
// then the last pieces
static float kernel_sum(const std::vector<float> &p, bool pairs) {
    constexpr int kB = 1 << kRunLevel;
    const uint32_t snp = static_cast<uint32_t>(p.size());
    RunSum rs;
    rs.top = make_float4(0.f, 0.f, 0.f, 0.f);
    rs.top_used = false;
    rs.n = 0;
    const uint32_t full = snp / kB * kB;
    float4 xs[kB];
    uint32_t p0 = 0;
    if (pairs) {
        for (; p0 + 2 * kB <= full; p0 += 2 * kB) {
            for (int r = 0; r < kB; ++r) xs[r] = make_float4(p[p0 + r], 0.f, 0.f, 0.f);
            const float4 a = run_tree(xs);
            for (int r = 0; r < kB; ++r) xs[r] = make_float4(p[p0 + kB + r], 0.f, 0.f, 0.f);
            const float4 b = run_tree(xs);
            run_push<kRunLevel + 1>(rs, add4(a, b));
        }
    }
    for (; p0 < full; p0 += kB) {
        for (int r = 0; r < kB; ++r) xs[r] = make_float4(p[p0 + r], 0.f, 0.f, 0.f);
        run_push<kRunLevel>(rs, run_tree(xs));
    }
    bool have;
    const float4 hi = run_total(rs, have);
    const uint32_t rem = snp - full;
    for (int r = 0; r < kB - 1; ++r) xs[r] = make_float4(static_cast<uint32_t>(r) < rem ? p[full + r] : 0.f, 0.f, 0.f, 0.f);
    return tail_total(xs, rem, hi, have).x;
}

int main() {
    std::mt19937 g(7);
    std::uniform_real_distribution<float> u(-1.f, 1.f);
    std::vector<int> counts;
    for (int n = 1; n <= 300; ++n) counts.push_back(n);
    for (int n : {511, 512, 513, 1000, 1023, 1024, 1025, 4095, 4096, 4097, 4111, 4127, 8192, 8207, 9000, 12345})
        counts.push_back(n);
    int bad = 0;
    for (int n : counts) {
        std::vector<float> p(n);
        for (auto &x : p) x = u(g) * static_cast<float>(1u << (g() % 24));  // wide magnitudes: order matters
        const float ref = counter_sum(p);
        for (int pairs = 0; pairs < 2; ++pairs) {
            const float got = kernel_sum(p, pairs != 0);
            if (std::memcmp(&ref, &got, sizeof(float)) != 0) {
                if (bad < 5) std::printf("n=%d pairs=%d counter=%a kernel=%a\n", n, pairs, ref, got);
                ++bad;
            }
        }
    }
    std::printf("checked %zu counts, %d mismatches\n", counts.size(), bad);
    return bad != 0;
}
"""


def _helpers() -> str:
    src = open(SRC).read()
    a = src.index("constexpr int kRunLevel")
    b = src.index("// Sums the pieces of every long segment")
    code = src[a:b]
    return code.replace("__device__ __attribute__((always_inline)) inline", "inline").replace("__device__ inline",
                                                                                               "inline")


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_run_trees_equal_the_pairwise_counter():
    with tempfile.TemporaryDirectory() as d:
        cpp = os.path.join(d, "order.cpp")
        exe = os.path.join(d, "order")
        with open(cpp, "w") as f:
            f.write(HEADER + _helpers() + MAIN)
        subprocess.run(["g++", "-O1", "-std=c++17", "-ffp-contract=off", cpp, "-o", exe], check=True,
                       capture_output=True, text=True)
        r = subprocess.run([exe], capture_output=True, text=True)
        assert r.returncode == 0, r.stdout + r.stderr
        assert "0 mismatches" in r.stdout
