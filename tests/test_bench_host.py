"""Host-side checks of bench.py (no GPU): the one-GPU contract, the
instruction mix behind the roofline, the storage sizes behind the byte counts,
the workload definitions and the source list the traffic profile is tied to."""
import re
import subprocess
import sys
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parent.parent


@pytest.fixture(scope="module")
def bench():
    sys.path.insert(0, str(ROOT))
    import bench as b
    return b


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, str(ROOT / "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_instruction_mix(bench):
    assert sum(bench.INNER_LOOP_MIX.values()) == 62
    assert bench.INSTR_PER_PARAM_SEED == 15.5
    assert bench.VALU_LANE_INSTR_PER_S == pytest.approx(157.3e12 / 4, rel=1e-3)


def test_storage_bytes(bench):
    from paper_2306_10015_amd import synth
    assert bench.storage_bytes(synth.WORKLOADS["opt125m"]) == 4.0
    assert bench.storage_bytes(synth.WORKLOADS["opt1.3b"]) == 2.0
    assert bench.storage_bytes(synth.WORKLOADS["opt6.7b-nf4"]) == 0.5625


def test_workloads_are_consistent():
    from paper_2306_10015_amd import synth
    for name, w in synth.WORKLOADS.items():
        assert w.K == w.machines * w.samples_per_machine, name
        assert len(synth.workload_seeds(w)) == w.K
    sizes = {"opt125m": 123_581_952, "opt1.3b": 1_311_117_312, "opt6.7b": 6_648_897_536}
    for name, n in sizes.items():
        assert synth.WORKLOADS[name].numel == n


def test_traffic_profile_hash_covers_the_kernel_sources(bench):
    """Every file kernels.hip includes from csrc is hashed with it."""
    csrc = ROOT / "paper_2306_10015_amd" / "csrc"
    seen, todo = set(), ["kernels.hip"]
    while todo:
        f = todo.pop()
        if f in seen:
            continue
        seen.add(f)
        todo += [m for m in re.findall(r'#include "([^"]+)"', (csrc / f).read_text()) if (csrc / m).exists()]
    listed = {Path(p).name for p in bench.KERNEL_SOURCES}
    assert seen <= listed
