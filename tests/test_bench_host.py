"""Host-side checks of bench.py (no GPU): the one-GPU contract, the
instruction mix behind the roofline, the storage sizes behind the byte counts,
the workload definitions and the sources a counter profile is tied to."""
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
    # 8 transcendentals per block of 4 Gaussians issue on their own unit
    assert bench.NONTRANS_PER_PARAM_SEED == 13.5
    assert bench.VALU_LANE_INSTR_PER_S == pytest.approx(157.3e12 / 4, rel=1e-3)
    assert bench.PARAM_SEED_PEAK == pytest.approx(2.9127e12, rel=1e-4)


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


def test_profile_hash_covers_each_units_include_closure():
    """A profile is stamped with the hash of its kernel's translation unit
    and every header it includes: each unit of the library, and nothing
    outside the repository."""
    from paper_2306_10015_amd import build, profile_summary
    csrc = ROOT / "paper_2306_10015_amd" / "csrc"
    for unit in build.KERNEL_UNITS:
        seen, todo = set(), [unit]
        while todo:
            f = todo.pop()
            if f in seen:
                continue
            seen.add(f)
            todo += [m for m in re.findall(r'#include "([^"]+)"', (csrc / f).read_text()) if (csrc / m).exists()]
        listed = {Path(p).name for p in profile_summary.unit_sources(unit)}
        assert listed == seen, unit
    # the dense engine does not compile from the NF4, checksum or conversion code
    dense = {Path(p).name for p in profile_summary.unit_sources("engine_dense.hip")}
    assert not dense & {"nf4_ops.hpp", "nf4.hpp", "checksum.hip", "nf4_convert.hip", "engine_nf4.hip"}


def test_stale_profiles_are_not_quoted(bench, tmp_path, monkeypatch):
    """bench.py quotes a profile's counters only while the hash of the
    kernel's sources is the one stored with it."""
    import json
    from paper_2306_10015_amd import profile_summary, synth
    w = synth.WORKLOADS["opt6.7b"]
    good = {"kernel_unit": "engine_dense.hip",
            "kernel_source_sha256": profile_summary.source_hash("engine_dense.hip"),
            "hbm_bytes_per_dispatch": 1.0}
    monkeypatch.setattr(bench, "PROFILE", str(tmp_path / "engine_kernel_{workload}.json"))
    (tmp_path / "engine_kernel_opt6.7b.json").write_text(json.dumps(good))
    assert bench.engine_profile(w, "fast")["hbm_bytes_per_dispatch"] == 1.0
    assert bench.engine_profile(w, "portable") is None
    stale = dict(good, kernel_source_sha256="0" * 64)
    (tmp_path / "engine_kernel_opt6.7b.json").write_text(json.dumps(stale))
    assert bench.engine_profile(w, "fast") is None
    other = dict(good, kernel_unit="engine_nf4.hip")
    (tmp_path / "engine_kernel_opt6.7b.json").write_text(json.dumps(other))
    assert bench.engine_profile(w, "fast") is None


def test_host_cores_reports_the_process_share(bench, monkeypatch):
    monkeypatch.setenv("OMP_NUM_THREADS", "3")
    threads, cores = bench.host_cores()
    assert threads == min(3, cores["affinity"])
    assert cores["nproc"] >= cores["affinity"] >= 1
    monkeypatch.delenv("OMP_NUM_THREADS")
    threads, cores = bench.host_cores()
    assert threads == cores["affinity"]
