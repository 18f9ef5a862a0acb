"""CPU oracle for the seeded perturbation engine (arXiv 2306.10015).

TEST INFRASTRUCTURE ONLY. Only the tests, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package. The product path
(``paper_2306_10015_amd``) never imports it and shares no code with it.

This module is argument marshalling around ``mezo_oracle.c`` (plain C99, fp64),
whose header cites the passages of the paper each function follows:

* ``perturb`` — Algorithm 1, ``PerturbParameters(theta, eps, s)``;
* ``update`` — Algorithm 1, the apply loop after ``GetGradients``;
* ``replay`` — Appendix B, late-joiner catch-up;
* ``quantize`` / ``dequantize`` — Section 3, the one-byte projected gradient.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from pathlib import Path

import numpy as np

HERE = Path(__file__).resolve().parent
SRC = HERE / "mezo_oracle.c"
LIB = HERE / "liboracle.so"

F32, BF16 = 0, 1
LINEAR, SIGNED_LOG = 0, 1

#: Default signed-log slope: a base-2 log, so code 127 is just inside fp32.
LOG2_ALPHA = 1.0 / 0.6931471805599453

#: Memory layout of ``orc_seed_t``: (machine u64, step u32, sample u32), 16 B.
SEED_DTYPE = np.dtype([("machine", "<u8"), ("step", "<u4"), ("sample", "<u4")])


def build(force: bool = True) -> Path:
    """Compile ``liboracle.so`` with gcc (-O2, no fast-math, no contraction)."""
    if LIB.exists() and not force:
        return LIB
    tmp = LIB.with_suffix(".so.tmp")
    cmd = [
        "gcc", "-std=c99", "-O2", "-fPIC", "-shared", "-fopenmp",
        "-ffp-contract=off", "-fno-fast-math", "-Wall", "-Wextra",
        str(SRC), "-o", str(tmp), "-lm",
    ]
    subprocess.run(cmd, check=True, cwd=HERE)
    os.replace(tmp, LIB)
    return LIB


_lib = None


def lib() -> ctypes.CDLL:
    """Load the oracle library, compiling it first only if it is not built."""
    global _lib
    if _lib is None:
        if not LIB.exists():
            build(force=True)
        L = ctypes.CDLL(str(LIB))
        vp, u32, u64, i32, f32 = (ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint64,
                                   ctypes.c_int, ctypes.c_float)

        class Seed(ctypes.Structure):
            _fields_ = [("machine", ctypes.c_uint64), ("step", ctypes.c_uint32),
                        ("sample", ctypes.c_uint32)]

        L.Seed = Seed
        L.orc_philox4x32_10.argtypes = [vp, vp, vp]
        L.orc_philox4x32_10.restype = None
        L.orc_block_words.argtypes = [Seed, u32, u64, vp]
        L.orc_block_words.restype = None
        L.orc_box_muller.argtypes = [vp, vp]
        L.orc_box_muller.restype = None
        L.orc_z.argtypes = [Seed, u32, u64]
        L.orc_z.restype = f32
        L.orc_generate.argtypes = [Seed, u32, u64, u64, vp, vp]
        L.orc_generate.restype = i32
        L.orc_round_f32.argtypes = [ctypes.c_double]
        L.orc_round_f32.restype = f32
        L.orc_round_bf16.argtypes = [ctypes.c_double]
        L.orc_round_bf16.restype = ctypes.c_uint16
        L.orc_signed_log_qmax.argtypes = [f32]
        L.orc_signed_log_qmax.restype = i32
        L.orc_quantize.argtypes = [vp, vp, u32, i32, f32, f32]
        L.orc_quantize.restype = i32
        L.orc_dequantize.argtypes = [vp, vp, u32, i32, f32, f32]
        L.orc_dequantize.restype = i32
        L.orc_coefficients.argtypes = [vp, u32, i32, f32, f32, f32, vp]
        L.orc_coefficients.restype = i32
        L.orc_perturb.argtypes = [vp, i32, u32, vp, u64, u64, Seed, f32]
        L.orc_perturb.restype = i32
        L.orc_update.argtypes = [vp, i32, u32, vp, u64, u64, vp, vp, u32, i32, f32, f32, f32]
        L.orc_update.restype = i32
        L.orc_replay.argtypes = [vp, i32, u32, vp, u64, u64, vp, vp, vp, vp, u32, i32, f32, f32]
        L.orc_replay.restype = i32
        L.orc_box_muller_portable.argtypes = [vp, vp]
        L.orc_box_muller_portable.restype = None
        L.orc_box_muller_blocks.argtypes = [vp, u64, vp]
        L.orc_box_muller_blocks.restype = None
        L.orc_box_muller_portable_blocks.argtypes = [vp, u64, vp]
        L.orc_box_muller_portable_blocks.restype = None
        L.orc_z_portable.argtypes = [Seed, u32, u64]
        L.orc_z_portable.restype = f32
        L.orc_generate_portable.argtypes = [Seed, u32, u64, u64, vp]
        L.orc_generate_portable.restype = i32
        L.orc_perturb_portable.argtypes = [vp, i32, u32, vp, u64, u64, Seed, f32]
        L.orc_perturb_portable.restype = i32
        L.orc_update_portable.argtypes = [vp, i32, u32, vp, u64, u64, vp, vp, u32, i32, f32, f32, f32]
        L.orc_update_portable.restype = i32
        L.orc_replay_portable.argtypes = [vp, i32, u32, vp, u64, u64, vp, vp, vp, vp, u32, i32, f32, f32]
        L.orc_replay_portable.restype = i32
        L.orc_fmix64.argtypes = [u64]
        L.orc_fmix64.restype = u64
        L.orc_checksum.argtypes = [vp, u64, u32]
        L.orc_checksum.restype = u64
        L.orc_set_threads.argtypes = [i32]
        L.orc_set_threads.restype = None
        L.orc_get_threads.argtypes = []
        L.orc_get_threads.restype = i32
        _lib = L
    return _lib


class OracleError(RuntimeError):
    pass


def _check(rc: int, what: str) -> None:
    if rc != 0:
        raise OracleError(f"{what} failed with code {rc}")


def _ptr(a: np.ndarray | None):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _seed(s) -> "ctypes.Structure":
    m, t, j = (int(s["machine"]), int(s["step"]), int(s["sample"])) if isinstance(
        s, np.void) else (int(s[0]), int(s[1]), int(s[2]))
    return lib().Seed(m, t, j)


def seeds_array(seeds) -> np.ndarray:
    """(machine, step, sample) tuples -> contiguous ``SEED_DTYPE`` array."""
    if isinstance(seeds, np.ndarray) and seeds.dtype == SEED_DTYPE:
        return np.ascontiguousarray(seeds)
    out = np.zeros(len(seeds), dtype=SEED_DTYPE)
    for i, s in enumerate(seeds):
        out[i] = (int(s[0]), int(s[1]), int(s[2])) if not isinstance(s, np.void) else s
    return out


def set_threads(n: int) -> None:
    lib().orc_set_threads(int(n))


def get_threads() -> int:
    return int(lib().orc_get_threads())


def philox(ctr, key) -> np.ndarray:
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    lib().orc_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def block_words(seed, tensor_id: int, e: int) -> np.ndarray:
    out = np.zeros(4, dtype=np.uint32)
    lib().orc_block_words(_seed(seed), tensor_id, e, _ptr(out))
    return out


def box_muller(words) -> np.ndarray:
    w = np.ascontiguousarray(words, dtype=np.uint32)
    z = np.zeros(4, dtype=np.float64)
    lib().orc_box_muller(_ptr(w), _ptr(z))
    return z


def generate(seed, tensor_id: int, first: int, count: int, words=True, z=True,
             portable: bool = False):
    """RNG word and fp32 Gaussian of elements ``first .. first+count-1``
    (portable: the binary32-only Gaussian)."""
    w = np.zeros(count, dtype=np.uint32) if words else None
    g = np.zeros(count, dtype=np.float32) if z else None
    _check(lib().orc_generate(_seed(seed), tensor_id, first, count, _ptr(w),
                              None if portable else _ptr(g)), "generate")
    if portable and z:
        _check(lib().orc_generate_portable(_seed(seed), tensor_id, first, count, _ptr(g)),
               "generate_portable")
    return w, g


def box_muller_blocks(words, portable: bool = False) -> np.ndarray:
    """z (fp32) of every block of 4 given words: the fp64 transform rounded
    once, or the portable binary32 one."""
    w = np.ascontiguousarray(words, dtype=np.uint32)
    if w.size % 4:
        raise ValueError("words come in blocks of 4")
    z = np.zeros(w.size, dtype=np.float32)
    fn = lib().orc_box_muller_portable_blocks if portable else lib().orc_box_muller_blocks
    fn(_ptr(w), w.size // 4, _ptr(z))
    return z


def box_muller_portable(words) -> np.ndarray:
    w = np.ascontiguousarray(words, dtype=np.uint32)
    z = np.zeros(4, dtype=np.float32)
    lib().orc_box_muller_portable(_ptr(w), _ptr(z))
    return z


def round_f32(x: float) -> float:
    return float(lib().orc_round_f32(float(x)))


def round_bf16(x: float) -> int:
    return int(lib().orc_round_bf16(float(x)))


def signed_log_qmax(alpha: float) -> int:
    """Largest code magnitude of the signed-log code for slope alpha."""
    return int(lib().orc_signed_log_qmax(float(alpha)))


def quantize(g, kind: int = LINEAR, scale: float = 1.0 / 127.0, alpha: float = LOG2_ALPHA) -> np.ndarray:
    ga = np.ascontiguousarray(g, dtype=np.float32)
    q = np.zeros(ga.size, dtype=np.int8)
    _check(lib().orc_quantize(_ptr(ga), _ptr(q), ga.size, kind, scale, alpha), "quantize")
    return q


def dequantize(q, kind: int = LINEAR, scale: float = 1.0 / 127.0, alpha: float = LOG2_ALPHA) -> np.ndarray:
    qa = np.ascontiguousarray(q, dtype=np.int8)
    g = np.zeros(qa.size, dtype=np.float32)
    _check(lib().orc_dequantize(_ptr(qa), _ptr(g), qa.size, kind, scale, alpha), "dequantize")
    return g


def coefficients(q, lr: float, kind: int = LINEAR, scale: float = 1.0 / 127.0,
                 alpha: float = LOG2_ALPHA) -> np.ndarray:
    qa = np.ascontiguousarray(q, dtype=np.int8)
    c = np.zeros(qa.size, dtype=np.float32)
    _check(lib().orc_coefficients(_ptr(qa), qa.size, kind, scale, alpha, lr, _ptr(c)),
           "coefficients")
    return c


def _theta_args(theta: np.ndarray):
    if theta.dtype == np.float32:
        dt = F32
    elif theta.dtype == np.uint16:
        dt = BF16
    else:
        raise TypeError("theta must be float32 or uint16 (bf16 bits)")
    if not theta.flags.c_contiguous:
        raise ValueError("theta must be contiguous")
    return dt


def _idx(idx):
    return None if idx is None else np.ascontiguousarray(idx, dtype=np.uint64)


def perturb(theta: np.ndarray, tensor_id: int, seed, scale: float, idx=None, first: int = 0,
            portable: bool = False):
    """In place: theta <- round(theta + scale * z(seed)) (PerturbParameters)."""
    dt = _theta_args(theta)
    ix = _idx(idx)
    fn = lib().orc_perturb_portable if portable else lib().orc_perturb
    _check(fn(_ptr(theta), dt, tensor_id, _ptr(ix), first, theta.size, _seed(seed), scale),
           "perturb")
    return theta


def update(theta: np.ndarray, tensor_id: int, seeds, q, lr: float, kind: int = LINEAR,
           scale: float = 1.0 / 127.0, alpha: float = LOG2_ALPHA, idx=None, first: int = 0,
           portable: bool = False):
    """In place: theta <- round(theta + sum_k c_k z_k), c_k = fl32(-lr * deq(q_k))."""
    dt = _theta_args(theta)
    ix = _idx(idx)
    sa = seeds_array(seeds)
    qa = np.ascontiguousarray(q, dtype=np.int8)
    if sa.size != qa.size:
        raise ValueError("seeds and q differ in length")
    fn = lib().orc_update_portable if portable else lib().orc_update
    _check(fn(_ptr(theta), dt, tensor_id, _ptr(ix), first, theta.size,
              _ptr(sa), _ptr(qa), sa.size, kind, scale, alpha, lr), "update")
    return theta


def fmix64(x: int) -> int:
    return int(lib().orc_fmix64(int(x) & 0xFFFFFFFFFFFFFFFF))


def checksum_tensor(data: np.ndarray, tensor_id: int) -> int:
    """Checksum of one tensor's bytes (fp32, or uint16 bf16 bits)."""
    a = np.ascontiguousarray(data)
    return int(lib().orc_checksum(_ptr(a), a.nbytes, int(tensor_id)))


def checksum(tensors, tensor_ids=None) -> int:
    """Checksum of a parameter set: the sum mod 2^64 of its tensors'."""
    ids = range(len(tensors)) if tensor_ids is None else tensor_ids
    return sum(checksum_tensor(t, i) for t, i in zip(tensors, ids)) & 0xFFFFFFFFFFFFFFFF


def replay(theta: np.ndarray, tensor_id: int, steps, kind: int = LINEAR,
           scale: float = 1.0 / 127.0, alpha: float = LOG2_ALPHA, idx=None, first: int = 0,
           portable: bool = False):
    """In place: apply ``steps`` = [(seeds, q, lr), ...] one after another."""
    dt = _theta_args(theta)
    ix = _idx(idx)
    seeds = np.concatenate([seeds_array(s) for s, _, _ in steps]) if steps else \
        np.zeros(0, dtype=SEED_DTYPE)
    qs = np.concatenate([np.asarray(q, dtype=np.int8) for _, q, _ in steps]) if steps else \
        np.zeros(0, dtype=np.int8)
    kt = np.array([len(q) for _, q, _ in steps], dtype=np.uint32)
    lrt = np.array([lr for _, _, lr in steps], dtype=np.float32)
    fn = lib().orc_replay_portable if portable else lib().orc_replay
    _check(fn(_ptr(theta), dt, tensor_id, _ptr(ix), first, theta.size,
              _ptr(seeds), _ptr(qs), _ptr(kt), _ptr(lrt), len(steps),
              kind, scale, alpha), "replay")
    return theta
