"""Host-side tests of libmezo that need no GPU: the library loads and exports
every symbol include/mezo.h declares; the one-byte codec (Section 3) matches
the oracle bit for bit; argument checks return the documented codes before
anything touches a device."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from paper_2306_10015_amd import mezo

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    text = open(os.path.join(ROOT, "include", "mezo.h")).read()
    return sorted(set(re.findall(r"^MEZO_API\s+[\w\s\*]*?\b(\w+)\s*\(", text, re.M)))


def test_header_declares_the_boundary_calls():
    names = declared_symbols()
    for required in ("mezo_perturb", "mezo_update_multi", "mezo_replay", "quantize_projgrad"):
        assert required in names
    assert sorted(mezo.EXPORTS) == names


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(str(mezo.LIB_PATH))
    for name in declared_symbols():
        assert hasattr(lib, name), name


def test_no_cpu_fallback_in_the_binding():
    """The binding only marshals arguments: it never imports the oracle."""
    src = open(mezo.__file__).read()
    assert "oracle" not in src.replace("oracle.", "")  # no import or call
    assert "import oracle" not in src


def test_product_package_never_touches_the_oracle():
    pkg = os.path.join(ROOT, "paper_2306_10015_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".cpp", ".hip", ".hpp", ".h")):
                text = open(os.path.join(dirpath, f)).read()
                assert not re.search(r"^\s*(import|from)\s+oracle\b", text, re.M), f
                assert "mezo_oracle" not in text and "liboracle" not in text, f


def test_binding_fails_loudly_without_the_library(tmp_path):
    """A copy of the binding next to no libmezo.so refuses to import."""
    import shutil
    import subprocess
    import sys
    pkg = tmp_path / "pkg"
    pkg.mkdir()
    shutil.copy(mezo.__file__, pkg / "mezo.py")
    (pkg / "__init__.py").write_text("")
    r = subprocess.run([sys.executable, "-c", "import pkg.mezo"], cwd=tmp_path, capture_output=True,
                       text=True, timeout=300)
    assert r.returncode != 0
    assert "ImportError" in r.stderr and "not built" in r.stderr


# ---- codec parity with the oracle -----------------------------------------

CODECS = [(mezo.LINEAR, 1 / 127, 1.0), (mezo.LINEAR, 0.25, 1.0), (mezo.LINEAR, 3e-4, 1.0),
          (mezo.SIGNED_LOG, 1.0, mezo.LOG2_ALPHA), (mezo.SIGNED_LOG, 1.0, 3.0), (mezo.SIGNED_LOG, 1.0, 1.0),
          (mezo.SIGNED_LOG, 1.0, 0.3),
          (mezo.SIGNED_LOG, 1.0, 17.5)]


@pytest.mark.parametrize("kind,scale,alpha", CODECS)
def test_quantize_matches_oracle_bit_exact(kind, scale, alpha):
    rng = np.random.Generator(np.random.PCG64(31))
    g = np.concatenate([
        rng.normal(0, 1, 20000), rng.normal(0, 1e3, 20000), rng.uniform(-2, 2, 20000),
        (np.arange(-300, 301) * 0.5) * scale,            # exact ties of the linear code
        np.array([0.0, -0.0, np.inf, -np.inf, 3.4e38, -3.4e38, 1e-45]),
    ]).astype(np.float32)
    got = mezo.quantize_projgrad(g, mezo.codec(kind, scale, alpha))
    want = oracle.quantize(g, kind, scale, alpha)
    assert np.array_equal(got, want)


@pytest.mark.parametrize("kind,scale,alpha", CODECS)
def test_dequantize_matches_oracle_bit_exact(kind, scale, alpha):
    qmax = oracle.signed_log_qmax(alpha) if kind == mezo.SIGNED_LOG else 127
    q = np.arange(-qmax, qmax + 1, dtype=np.int8)
    got = mezo.dequantize(q, mezo.codec(kind, scale, alpha))
    want = oracle.dequantize(q, kind, scale, alpha)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


def test_codec_errors():
    with pytest.raises(mezo.MezoError) as e:
        mezo.quantize_projgrad([np.nan])
    assert e.value.code == mezo.ERANGE
    with pytest.raises(mezo.MezoError) as e:
        mezo.dequantize([-128])
    assert e.value.code == mezo.ERANGE
    for bad in (mezo.codec(mezo.LINEAR, 0.0), mezo.codec(mezo.LINEAR, float("inf")),
                mezo.codec(mezo.SIGNED_LOG, 1.0, 1e-3), mezo.codec(7, 1.0, 1.0)):
        with pytest.raises(mezo.MezoError) as e:
            mezo.quantize_projgrad([1.0], bad)
        assert e.value.code == mezo.ERANGE
    assert mezo.quantize_projgrad(np.zeros(0, dtype=np.float32)).size == 0
    # the natural log's codes stop at 88: larger received codes are refused
    nat = mezo.codec(mezo.SIGNED_LOG, 1.0, 1.0)
    with pytest.raises(mezo.MezoError) as e:
        mezo.dequantize([89], nat)
    assert e.value.code == mezo.ERANGE
    assert mezo.quantize_projgrad([3.4e38], nat)[0] == 88


# ---- argument checks (no device is touched) -------------------------------

def create(entries):
    arr = (mezo.Tensor * max(1, len(entries)))()
    for i, e in enumerate(entries):
        ptr, n, tid, dt = e[:4]
        arr[i] = mezo.Tensor(ptr, n, tid, dt, e[4] if len(e) > 4 else None, e[5] if len(e) > 5 else 0)
    h = ctypes.c_void_p()
    rc = mezo.lib.mezo_paramset_create(arr, len(entries), ctypes.byref(h))
    return rc, h


@pytest.mark.parametrize("entries,code", [
    ([], mezo.EINVAL),
    ([(0, 16, 0, mezo.F32)], mezo.EINVAL),                         # null data
    ([(0x1004, 16, 0, mezo.F32)], mezo.EINVAL),                    # not 16-byte aligned
    ([(0x1000, 0, 0, mezo.F32)], mezo.EINVAL),                     # empty tensor
    ([(0x1000, (1 << 34) + 1, 0, mezo.F32)], mezo.EINVAL),         # too many elements
    ([(0x1000, 16, 0, 5)], mezo.EDTYPE),
    ([(0x1000, 16, 3, mezo.F32), (0x2000, 16, 3, mezo.F32)], mezo.EINVAL),   # duplicate id
    ([(0x1000, 16, 0, mezo.F32), (0x1030, 16, 1, mezo.F32)], mezo.EOVERLAP),
    ([(0x1000, 16, 0, mezo.BF16), (0x1010, 16, 1, mezo.F32)], mezo.EOVERLAP),
    ([(0x1000, 16, 0, mezo.NF4)], mezo.EINVAL),                    # NF4 without absmax
    ([(0x1000, 16, 0, mezo.NF4, 0x2008)], mezo.EINVAL),            # absmax not 16-byte aligned
    ([(0x1000, 16, 0, mezo.F32, 0x2000)], mezo.EINVAL),            # absmax on a float tensor
    ([(0x1000, 16, 0, mezo.NF4, 0x1000)], mezo.EOVERLAP),          # codes and absmax overlap
    ([(0x1000, 260, 0, mezo.NF4, 0x2000), (0x2010, 4, 1, mezo.F32)], mezo.EOVERLAP),  # 5 absmax = 20 B
    ([(0x1000, 33, 0, mezo.NF4, 0x2000), (0x1010, 4, 1, mezo.F32)], mezo.EOVERLAP),   # 17 code bytes
    ([(0x1000, 16, 0, mezo.F32, None, 4)], mezo.EINVAL),           # shard offset not a multiple of 8
    ([(0x1000, 16, 0, mezo.F32, None, (1 << 34) - 8)], mezo.EINVAL),  # shard past the counter's range
    ([(0x1000, 16, 0, mezo.NF4, 0x2000, 64)], mezo.EINVAL),        # NF4 split by whole tensors only
])
def test_paramset_create_rejects(entries, code):
    rc, h = create(entries)
    assert rc == code
    assert not h.value


def test_paramset_create_accepts_shards():
    # the last 16 elements of the counter's range, and a shard at offset 8
    rc, h = create([(0x1000, 16, 0, mezo.F32, None, (1 << 34) - 16), (0x2000, 8, 1, mezo.BF16, None, 8)])
    assert rc == mezo.OK
    mezo.lib.mezo_paramset_destroy(h)


def test_paramset_create_accepts_adjacent_and_reports_numel():
    rc, h = create([(0x1000, 16, 0, mezo.F32), (0x1040, 24, 1, mezo.BF16)])
    assert rc == mezo.OK
    assert mezo.lib.mezo_paramset_numel(h) == 40
    mezo.lib.mezo_paramset_destroy(h)
    mezo.lib.mezo_paramset_destroy(None)


def test_nf4_tensors_accepted_when_adjacent():
    # 32 elements: 16 code bytes and one absmax; the next tensor may start right after
    rc, h = create([(0x1000, 32, 0, mezo.NF4, 0x3000), (0x1010, 4, 1, mezo.F32), (0x3010, 8, 2, mezo.BF16)])
    assert rc == mezo.OK
    assert mezo.lib.mezo_paramset_numel(h) == 44
    mezo.lib.mezo_paramset_destroy(h)


def test_nf4_conversion_argument_checks():
    lib = mezo.lib
    q, d = lib.mezo_nf4_quantize, lib.mezo_nf4_dequantize
    assert q(0x1000, 9, 64, 0x2000, 0x3000, None) == mezo.EDTYPE
    assert q(None, mezo.F32, 64, 0x2000, 0x3000, None) == mezo.EINVAL
    assert q(0x1000, mezo.F32, 0, 0x2000, 0x3000, None) == mezo.EINVAL
    assert q(0x1000, mezo.F32, (1 << 34) + 1, 0x2000, 0x3000, None) == mezo.EINVAL
    assert q(0x1008, mezo.F32, 64, 0x2000, 0x3000, None) == mezo.EINVAL
    assert q(0x1000, mezo.F32, 64, 0x1080, 0x3000, None) == mezo.EOVERLAP    # 256 B of values
    assert q(0x1000, mezo.BF16, 64, 0x1080, 0x1090, None) == mezo.EOVERLAP   # 32 code bytes
    assert d(0x2000, 0x3000, 64, 0x1000, 9, None) == mezo.EDTYPE
    assert d(0x2000, None, 64, 0x1000, mezo.F32, None) == mezo.EINVAL
    assert d(0x2000, 0x2010, 64, 0x1000, mezo.F32, None) == mezo.EOVERLAP


def test_tensor_struct_layout():
    assert ctypes.sizeof(mezo.Tensor) == 40
    assert mezo.Tensor.absmax.offset == 24
    assert mezo.Tensor.first.offset == 32


@pytest.fixture
def fake_ps():
    rc, h = create([(0x10000, 1024, 0, mezo.F32)])
    assert rc == mezo.OK
    yield h
    mezo.lib.mezo_paramset_destroy(h)


def seeds_of(*triples):
    return mezo.seeds_array(list(triples))


def test_update_argument_checks(fake_ps):
    lib = mezo.lib
    c = mezo.codec()
    s = seeds_of((0, 0, 0), (1, 0, 0))
    q = np.array([3, 4], dtype=np.int8)
    assert lib.mezo_update_multi(None, s.ctypes.data, q.ctypes.data, 2, c, 1e-3, None) == mezo.EINVAL
    assert lib.mezo_update_multi(fake_ps, None, q.ctypes.data, 2, c, 1e-3, None) == mezo.EINVAL
    assert lib.mezo_update_multi(fake_ps, s.ctypes.data, q.ctypes.data, 2, None, 1e-3, None) == mezo.EINVAL
    assert lib.mezo_update_multi(fake_ps, s.ctypes.data, q.ctypes.data, 2, c, float("nan"), None) == mezo.ERANGE
    bad_q = np.array([3, -128], dtype=np.int8)
    assert lib.mezo_update_multi(fake_ps, s.ctypes.data, bad_q.ctypes.data, 2, c, 1e-3, None) == mezo.ERANGE
    for order in [((1, 0, 0), (0, 0, 0)), ((0, 0, 0), (0, 0, 0)), ((0, 1, 0), (0, 0, 5)),
                  ((0, 0, 2), (0, 0, 1))]:
        so = seeds_of(*order)
        assert lib.mezo_update_multi(fake_ps, so.ctypes.data, q.ctypes.data, 2, c, 1e-3, None) == mezo.EORDER
    # no-ops return OK without touching a device
    assert lib.mezo_update_multi(fake_ps, s.ctypes.data, q.ctypes.data, 0, c, 1e-3, None) == mezo.OK
    assert lib.mezo_update_multi(fake_ps, s.ctypes.data, q.ctypes.data, 2, c, 0.0, None) == mezo.OK
    z = np.zeros(2, dtype=np.int8)
    assert lib.mezo_update_multi(fake_ps, s.ctypes.data, z.ctypes.data, 2, c, 1e-3, None) == mezo.OK


def test_perturb_and_replay_argument_checks(fake_ps):
    lib = mezo.lib
    assert lib.mezo_perturb(fake_ps, mezo.Seed(0, 0, 0), float("inf"), None) == mezo.ERANGE
    assert lib.mezo_perturb(None, mezo.Seed(0, 0, 0), 1.0, None) == mezo.EINVAL
    assert lib.mezo_perturb(fake_ps, mezo.Seed(0, 0, 0), 0.0, None) == mezo.OK
    c = mezo.codec()
    steps = (mezo.Step * 2)()
    s0 = seeds_of((0, 0, 0), (1, 0, 0))
    s1 = seeds_of((1, 1, 0), (0, 1, 0))          # unsorted
    q = np.array([1, 2], dtype=np.int8)
    steps[0] = mezo.Step(s0.ctypes.data, q.ctypes.data, 2, 1e-3)
    steps[1] = mezo.Step(s1.ctypes.data, q.ctypes.data, 2, 1e-3)
    assert lib.mezo_replay(fake_ps, steps, 2, c, None) == mezo.EORDER
    assert lib.mezo_replay(fake_ps, steps, 0, c, None) == mezo.OK
    assert lib.mezo_replay(fake_ps, None, 2, c, None) == mezo.EINVAL
    steps[1] = mezo.Step(s0.ctypes.data, q.ctypes.data, 2, float("nan"))
    assert lib.mezo_replay(fake_ps, steps, 2, c, None) == mezo.ERANGE
    # more than 2^32 - 1 terms in one call: rejected from the step counts
    # alone, before any seed or code is read
    steps[0] = mezo.Step(s0.ctypes.data, q.ctypes.data, 1 << 31, 1e-3)
    steps[1] = mezo.Step(s0.ctypes.data, q.ctypes.data, 1 << 31, 1e-3)
    assert lib.mezo_replay(fake_ps, steps, 2, c, None) == mezo.ERANGE


def test_perturb_multi_argument_checks(fake_ps):
    lib = mezo.lib
    s = seeds_of((0, 0, 0), (1, 0, 0))
    sc = np.array([1e-3, float("nan")], dtype=np.float32)
    assert lib.mezo_perturb_multi(fake_ps, s.ctypes.data, sc.ctypes.data, 2, None) == mezo.ERANGE
    sc = np.array([1e-3, float("inf")], dtype=np.float32)
    assert lib.mezo_perturb_multi(fake_ps, s.ctypes.data, sc.ctypes.data, 2, None) == mezo.ERANGE
    assert lib.mezo_perturb_multi(None, s.ctypes.data, sc.ctypes.data, 2, None) == mezo.EINVAL
    assert lib.mezo_perturb_multi(fake_ps, None, sc.ctypes.data, 2, None) == mezo.EINVAL
    assert lib.mezo_perturb_multi(fake_ps, s.ctypes.data, None, 2, None) == mezo.EINVAL
    # nothing to apply: OK without touching a device
    assert lib.mezo_perturb_multi(fake_ps, None, None, 0, None) == mezo.OK
    z = np.zeros(2, dtype=np.float32)
    assert lib.mezo_perturb_multi(fake_ps, s.ctypes.data, z.ctypes.data, 2, None) == mezo.OK


def test_debug_generate_range_check():
    lib = mezo.lib
    assert lib.mezo_debug_generate(mezo.Seed(0, 0, 0), 0, (1 << 34) - 4, 8, 0, 0x1000, None, None) == mezo.EINVAL
    assert lib.mezo_debug_generate(mezo.Seed(0, 0, 0), 0, 0, 16, 7, 0x1000, None, None) == mezo.EINVAL
    assert lib.mezo_debug_generate(mezo.Seed(0, 0, 0), 0, 0, 0, 0, 0x1000, None, None) == mezo.OK
    assert lib.mezo_debug_generate(mezo.Seed(0, 0, 0), 0, 0, 16, 1, None, None, None) == mezo.OK


def test_gaussian_mode_setter():
    rc, h = create([(0x1000, 16, 0, mezo.F32)])
    assert rc == mezo.OK
    assert mezo.lib.mezo_paramset_set_gaussian(h, mezo.GAUSS_PORTABLE) == mezo.OK
    assert mezo.lib.mezo_paramset_set_gaussian(h, mezo.GAUSS_FAST) == mezo.OK
    assert mezo.lib.mezo_paramset_set_gaussian(h, 2) == mezo.EINVAL
    assert mezo.lib.mezo_paramset_set_gaussian(None, 0) == mezo.EINVAL
    mezo.lib.mezo_paramset_destroy(h)


def test_strerror_covers_every_code():
    for code in (mezo.OK, mezo.EINVAL, mezo.EDTYPE, mezo.EOVERLAP, mezo.EORDER, mezo.ERANGE,
                 mezo.EHIP, mezo.ENOMEM):
        assert mezo.lib.mezo_strerror(code).decode() not in ("", "unknown error code")
    assert mezo.lib.mezo_strerror(-99).decode() == "unknown error code"


def test_one_hip_runtime_in_the_process():
    """libmezo binds to the HIP runtime torch loaded (torch's streams and
    pointers are only valid there); no second copy is mapped."""
    paths = set()
    with open("/proc/self/maps") as f:
        for line in f:
            p = line.split()[-1]
            if "libamdhip64" in p:
                paths.add(p)
    assert len(paths) == 1, paths


def test_from_calls_check_layout_and_overlap():
    lib = mezo.lib
    c = mezo.codec()
    s = seeds_of((0, 0, 0), (1, 0, 0))
    q = np.array([3, 4], dtype=np.int8)
    _, dst = create([(0x100000, 1024, 0, mezo.F32), (0x200000, 512, 1, mezo.BF16)])
    _, ok_src = create([(0x300000, 1024, 0, mezo.F32), (0x400000, 512, 1, mezo.BF16)])
    _, bad_n = create([(0x300000, 1000, 0, mezo.F32), (0x400000, 512, 1, mezo.BF16)])
    _, bad_id = create([(0x300000, 1024, 5, mezo.F32), (0x400000, 512, 1, mezo.BF16)])
    _, bad_cnt = create([(0x300000, 1024, 0, mezo.F32)])
    _, overlap = create([(0x100800, 1024, 0, mezo.F32), (0x400000, 512, 1, mezo.BF16)])
    _, twin = create([(0x100000, 1024, 0, mezo.F32), (0x400000, 512, 1, mezo.BF16)])
    try:
        for src, code in [(bad_n, mezo.EINVAL), (bad_id, mezo.EINVAL), (bad_cnt, mezo.EINVAL),
                          (overlap, mezo.EOVERLAP)]:
            assert lib.mezo_update_multi_from(dst, src, s.ctypes.data, q.ctypes.data, 2, c, 1e-3,
                                              None) == code
            assert lib.mezo_perturb_from(dst, src, mezo.Seed(0, 0, 0), 1e-3, None) == code
        # argument checks come first, as for the in-place calls
        assert lib.mezo_update_multi_from(dst, ok_src, s.ctypes.data, q.ctypes.data, 2, c,
                                          float("nan"), None) == mezo.ERANGE
        assert lib.mezo_perturb_from(dst, ok_src, mezo.Seed(0, 0, 0), float("inf"), None) == mezo.ERANGE
        assert lib.mezo_perturb_from(None, ok_src, mezo.Seed(0, 0, 0), 1.0, None) == mezo.EINVAL
        # a tensor that is its own source is allowed; valid calls get as far as
        # the device (none here)
        assert lib.mezo_perturb_from(dst, twin, mezo.Seed(0, 0, 0), 1.0, None) == mezo.EHIP
        assert lib.mezo_perturb_from(dst, ok_src, mezo.Seed(0, 0, 0), 0.0, None) == mezo.EHIP
    finally:
        for h in (dst, ok_src, bad_n, bad_id, bad_cnt, overlap, twin):
            lib.mezo_paramset_destroy(h)


def test_step_lr():
    assert mezo.step_lr(0.1, 4) == pytest.approx(0.025)
    assert mezo.step_lr(0.1, 4, sqrt_scaling=True) == pytest.approx(0.05)
    assert mezo.step_lr(1e-6, 1) == 1e-6
    with pytest.raises(ValueError):
        mezo.step_lr(0.1, 0)


@pytest.mark.parametrize("compiler,std", [("gcc", "-std=c99"), ("g++", "-std=c++17")])
def test_header_is_plain_c_and_cpp(tmp_path, compiler, std):
    """include/mezo.h needs no HIP or torch header and compiles as C99 and
    C++ with warnings as errors."""
    import shutil
    import subprocess
    if not shutil.which(compiler):
        pytest.skip(f"{compiler} not available")
    src = tmp_path / ("use.c" if compiler == "gcc" else "use.cpp")
    src.write_text('#include "mezo.h"\n'
                   'int use(mezo_paramset_t ps, void* s) {\n'
                   '    mezo_seed_t seed = {1u, 2u, 3u};\n'
                   '    return mezo_perturb(ps, seed, 1e-3f, s) + (int)sizeof(mezo_tensor_t);\n'
                   '}\n')
    r = subprocess.run([compiler, std, "-Wall", "-Wextra", "-pedantic", "-Werror", "-fsyntax-only",
                        "-I", os.path.join(ROOT, "include"), str(src)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def test_kernel_resource_remarks_parse():
    """The build reads VGPRs, scratch and occupancy per kernel from the
    compiler's resource-usage remarks (the spill check rests on it)."""
    from paper_2306_10015_amd import build as b
    tag = " [-Rpass-analysis=kernel-resource-usage]"
    remarks = [f"x.hip:1:1: remark: Function Name: _Z1kv{tag}",
               f"x.hip:1:1: remark:     VGPRs: 40{tag}",
               f"x.hip:1:1: remark:     ScratchSize [bytes/lane]: 8{tag}",
               f"x.hip:1:1: remark:     Occupancy [waves/SIMD]: 8{tag}",
               f"x.hip:1:1: remark: Function Name: _Z1jv{tag}",
               f"x.hip:1:1: remark:     VGPRs: 12{tag}",
               f"x.hip:1:1: remark:     ScratchSize [bytes/lane]: 0{tag}"]
    assert b.kernel_resources(remarks) == [
        {"kernel": "_Z1kv", "VGPRs": 40, "ScratchSize": 8, "Occupancy": 8},
        {"kernel": "_Z1jv", "VGPRs": 12, "ScratchSize": 0}]


def test_no_kernel_spills_to_scratch():
    """Every kernel of the last build keeps its values in registers (the
    build records each kernel's resources and refuses a spill)."""
    from paper_2306_10015_amd import build as b
    path = b.BUILD_DIR / "kernel_resources.txt"
    if not path.exists():
        pytest.skip("no in-tree build record (run python -m paper_2306_10015_amd.build)")
    rows = [l.split() for l in path.read_text().splitlines() if l.strip()]
    assert {r[0] for r in rows} == set(b.KERNEL_UNITS)
    for r in rows:
        fields = dict(kv.split("=") for kv in r[2:])
        assert fields["scratch"] == "0", r
        assert int(fields["vgprs"]) <= 128, r
