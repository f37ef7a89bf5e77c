"""The hot-set kernels' batch schedule (csrc/scd_kernels.h: hot_sched and its helpers), compiled for
the host with g++ and checked over every window, consumer count and batch capacity the kernels use:
the batches of a launch tile its positions exactly once and in order, every consumer takes the same
number of steps per batch, no batch exceeds the capacity, and the adaptive consumer count keeps at
least two coordinates per consumer step.  Host only; no GPU."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_1702_07005_amd", "csrc")

HARNESS = r"""
#include "scd_kernels.h"
#include <cstdio>
using namespace scd;
int main() {
    const unsigned caps[] = {8, 9, 10, 12, 13, 16, 21, 32, 40, 64};
    const unsigned ns[] = {1, 2, 7, 31, 32, 33, 100, 999, 1000, 4096, 50001};
    for (unsigned cap : caps)
        for (unsigned NC = 1; NC <= (unsigned)kHotMaxConsumers; ++NC)
            for (unsigned W = NC; W <= (unsigned)kHotMaxWindow; ++W) {
                if ((W + NC - 1) / NC > (unsigned)kHotMaxGroups || (W + NC - 1) / NC > cap) continue;
                for (unsigned n : ns) {
                    const HotSched s = hot_sched(W, NC, cap, n);
                    unsigned pos = 0, total_w = 0;
                    for (unsigned c = 0; c < NC; ++c) total_w += hot_groups(s, c);
                    if (total_w != W || s.S < 1 || s.NP != (unsigned)kHotWaves - NC || s.NP % NC) {
                        printf("BAD shares W=%u NC=%u cap=%u\n", W, NC, cap); return 1;
                    }
                    for (unsigned b = 0; b < s.nb; ++b) {
                        const unsigned c = hot_consumer_of(s, b), B = hot_batch_size(s, b);
                        if (c != b % NC || hot_batch_start(s, b) != pos || B > cap ||
                            B != s.S * hot_groups(s, c) || hot_groups(s, c) > (unsigned)kHotMaxGroups) {
                            printf("BAD batch W=%u NC=%u cap=%u n=%u b=%u\n", W, NC, cap, n, b); return 1;
                        }
                        pos += B;
                    }
                    // every position covered, and no batch starts past the end
                    if (pos < n || (s.nb > 0 && hot_batch_start(s, s.nb - 1) >= n)) {
                        printf("BAD tiling W=%u NC=%u cap=%u n=%u nb=%u pos=%u\n", W, NC, cap, n, s.nb, pos); return 1;
                    }
                }
            }
    for (unsigned W = 2; W <= (unsigned)kHotMaxWindow; ++W) {
        const unsigned NC = hot_adaptive_consumers(W);
        if (NC < 1 || NC > (unsigned)kHotMaxConsumers || (NC > 1 && W / NC < 2)) {
            printf("BAD adaptive W=%u NC=%u\n", W, NC); return 1;
        }
        printf("adaptive %u %u\n", W, NC);
    }
    printf("OK\n");
    return 0;
}
"""


@pytest.mark.skipif(shutil.which("g++") is None or not os.path.isdir("/opt/rocm/include"),
                    reason="needs g++ and the ROCm headers")
def test_hot_schedule_tiles_every_launch(tmp_path):
    src = tmp_path / "sched.cpp"
    src.write_text(HARNESS)
    exe = tmp_path / "sched"
    subprocess.run(["g++", "-std=c++17", "-O1", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", "-I", CSRC,
                    str(src), "-o", str(exe)], check=True, capture_output=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True)
    assert out.returncode == 0 and out.stdout.strip().endswith("OK"), out.stdout[-2000:]
    nc = {int(w): int(n) for w, n in (l.split()[1:] for l in out.stdout.splitlines() if l.startswith("adaptive"))}
    # at 16 in flight: four consumers of 4; at 11: four consumers of 3, 3, 3 and 2
    assert nc[16] == 4 and nc[11] == 4 and nc[5] == 2 and nc[3] == 1
