"""Host logic: the split of a launch group's N-sized passes over workgroups
(csrc/edkm_partition.h), compiled with g++ and checked on the workload mixes.

Every N-pass workgroup holds a whole CU's LDS, so a grid larger than the CU
count runs a second wave; the split must stay within the budget while covering
every weight exactly once, in proportion to matrix size."""
import os
import shutil
import subprocess

import pytest

from paper_2309_00964_amd import inputs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HDR = os.path.join(ROOT, "paper_2309_00964_amd", "csrc", "edkm_partition.h")
MIN_CHUNK = 16384

DRIVER = r'''
#include "edkm_partition.h"
#include <cstdio>
int main() {
    int count, budget;
    while (std::scanf("%d %d", &count, &budget) == 2) {
        uint64_t n[64], chunk[64];
        uint32_t cnt[64], beg[64];
        for (int i = 0; i < count; ++i) std::scanf("%llu", (unsigned long long*)&n[i]);
        unsigned grid = edkm::split_passes(n, count, budget, %MIN%ull, chunk, cnt, beg);
        std::printf("%u", grid);
        for (int i = 0; i < count; ++i)
            std::printf(" %llu %u %u", (unsigned long long)chunk[i], cnt[i], beg[i]);
        std::printf("\n");
    }
}
'''


@pytest.fixture(scope="module")
def split(tmp_path_factory):
    if shutil.which("g++") is None:
        pytest.skip("g++ not available")
    d = tmp_path_factory.mktemp("split")
    src = d / "driver.cpp"
    src.write_text(DRIVER.replace("%MIN%", str(MIN_CHUNK)))
    exe = d / "driver"
    subprocess.check_call(["g++", "-O1", "-std=c++17", "-I", os.path.dirname(HDR), "-o", str(exe),
                           str(src)])

    def run(sizes, budget):
        line = "%d %d %s\n" % (len(sizes), budget, " ".join(str(s) for s in sizes))
        out = subprocess.run([str(exe)], input=line, capture_output=True, text=True,
                             check=True).stdout.split()
        vals = [int(x) for x in out]
        grid, rest = vals[0], vals[1:]
        return grid, [tuple(rest[3 * i:3 * i + 3]) for i in range(len(sizes))]
    return run


LAYER = [r * c for _, r, c in inputs.LLAMA7B_LAYER]
STACK = [r * c for _, r, c in inputs.WORKLOADS[5]["mats"]]
GROUP = 28   # EDKM_LAUNCH_GROUP: the stack runs as 8 launch groups of 28 matrices
MIXES = [LAYER, STACK[:8], STACK[8:16], STACK[16:24], [65536], [4096 * 4096], [11008 * 4096],
         [1], [7, 9, 1], [65536 + 37, 300007, 8], [16384 * 3 + 1, 10 ** 9], [2 ** 32 - 1] * 8,
         [1] * 8, [16384] * 8, STACK[:GROUP], STACK[GROUP * 7:], [1] * GROUP,
         [4096 * 4096] * (GROUP - 1) + [7]]


@pytest.mark.parametrize("budget", [512, 256, 255, 80, 32, 8, 1])
@pytest.mark.parametrize("mix", range(len(MIXES)))
def test_split_covers_every_weight_within_budget(split, mix, budget):
    sizes = MIXES[mix]
    grid, parts = split(sizes, budget)
    begin = 0
    for n, (chunk, cnt, beg) in zip(sizes, parts):
        assert chunk % 8 == 0 and chunk >= 8
        assert cnt >= 1 and beg == begin
        assert (cnt - 1) * chunk < n <= cnt * chunk          # every weight once, no empty slice
        assert cnt <= max(1, -(-n // MIN_CHUNK))               # no slice below the minimum chunk
        begin += cnt
    assert grid == begin
    assert grid <= max(budget, len(sizes))
    if budget >= len(sizes) and sum(-(-n // MIN_CHUNK) for n in sizes) >= budget:
        assert grid >= budget - len(sizes)     # the budget is used (chunk rounding may drop a few)


@pytest.mark.parametrize("mix", [0, 1, 2, 3])
def test_split_is_proportional(split, mix):
    """Each matrix's per-workgroup share is within one workgroup of proportional."""
    sizes = MIXES[mix]
    grid, parts = split(sizes, 256)
    assert grid == 256 or grid == 255
    total = sum(sizes)
    for n, (_, cnt, _) in zip(sizes, parts):
        assert abs(cnt - 256 * n / total) <= 1.0


@pytest.mark.parametrize("mix", [14, 15])
@pytest.mark.parametrize("budget", [256, 512])
def test_full_launch_group_is_proportional(split, mix, budget):
    """A launch group of 28 matrices (four layers of the stack) under the
    one-per-CU budget of the training passes and the two-per-CU budget of the
    palettization export."""
    sizes = MIXES[mix]
    assert len(sizes) == GROUP
    grid, parts = split(sizes, budget)
    assert budget - GROUP <= grid <= budget
    total = sum(sizes)
    for n, (_, cnt, _) in zip(sizes, parts):
        assert abs(cnt - budget * n / total) <= 1.0


def test_first_stack_group_fits_one_wave(split):
    """Layer 0 plus the next layer's first projection: independent rounding of
    each share gives 5 x 20 + 3 x 53 = 259 workgroups, a second wave on 256 CUs."""
    grid, _ = split(STACK[:8], 256)
    assert grid <= 256
