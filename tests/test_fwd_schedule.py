"""CPU check of the forward kernel's LDS-DMA load/wait schedule.

The forward kernel stages K and V blocks in LDS with loads that write LDS
directly; each wavefront waits only for its own loads (vmcnt) and a barrier
then publishes a tile to the workgroup. `fwd_ring_model.cpp` replays the
kernel's issue order for every wavefront (prologue staging rows, K/V ring
tiles, the v' rows of iteration 0, the conditional loads near the end of a
window) for head_dim 64 and 128, one or two wavefronts per query and 1..40 key
blocks, using the schedule functions the kernel itself includes, and checks
that every LDS read follows a wait that covers the data and a barrier.
"""

import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2507_02754_amd", "csrc")


@pytest.fixture(scope="module")
def model(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path_factory.mktemp("ring") / "fwd_ring_model")
    subprocess.run([gxx, "-std=c++17", "-O1", "-Wall", "-Werror", f"-I{CSRC}",
                    os.path.join(ROOT, "tests", "fwd_ring_model.cpp"), "-o", exe], check=True)

    def run(rule):
        out = subprocess.run([exe, rule], check=True, capture_output=True, text=True).stdout
        m = re.search(r"violations: (\d+) cases: (\d+)", out)
        assert m, out[-2000:]
        return int(m.group(1)), int(m.group(2)), out

    return run


def test_kernel_schedule_covers_every_lds_read(model):
    violations, cases, out = model("kernel")
    assert cases == 2 * 2 * 40
    assert violations == 0, out[:4000]


def test_model_detects_the_uncovered_tail_reads(model):
    """The model has teeth: with a fixed 3-tile wait in every iteration it
    finds the reads of the last K block and of the last two V blocks that no
    wait covers (at head_dim 128, w2 <= 32 and 17 blocks: K16 in iteration 14,
    V15 and V16 in the last two iterations)."""
    violations, _, out = model("steady")
    assert violations > 0
    for what in ("iteration 14 K16", "iteration 15 V15", "iteration 16 V16"):
        assert re.search(rf"D=128 G=1 nb=17: {what}: wavefront \d's load of \w+ is not covered", out), what


def test_kernel_uses_the_modelled_schedule():
    """The forward kernel takes its waits and conditional loads from the same
    schedule functions the model evaluates."""
    src = open(os.path.join(CSRC, "fwd_mfma.hip")).read()
    assert '#include "fwd_schedule.h"' in src
    for call in ("fwd_schedule::inflight_tiles(blk, nb)", "fwd_schedule::loads_k(blk, nb)",
                 "fwd_schedule::loads_v(blk, nb)", "fwd_schedule::epilogue_waits(nb)"):
        assert call in src, call
    # no fixed-count ring wait is left in the block loop
    loop = src[src.index("auto iteration = [&]"):src.index("// ---- epilogue")]
    assert "wait_tiles(IC<3>{});\n    lds_barrier" not in loop
