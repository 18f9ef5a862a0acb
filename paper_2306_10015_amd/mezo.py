"""Python binding of libmezo (include/mezo.h): argument marshalling only.

Every step of the engine runs in the library's HIP kernels; PyTorch supplies
device memory and the current stream. Importing this module loads
``libmezo.so`` from this directory and raises if it is not built (build it
with ``python -m paper_2306_10015_amd.build``); there is no fallback.

    import torch
    from paper_2306_10015_amd import mezo
    params = [torch.randn(1024, 1024, device="cuda") * 0.02 for _ in range(4)]
    ps = mezo.ParamSet(params)                       # tensor_id = position
    s = (machine_id, step, sample)
    ps.perturb(s, +eps); ...; ps.perturb(s, -2 * eps); ...; ps.perturb(s, +eps)
    q = mezo.quantize_projgrad([(l_plus - l_minus) / (2 * eps)])
    ps.update_multi(seeds, q_all, lr=eta / n_grads)  # Algorithm 1 apply loop
"""
from __future__ import annotations

import ctypes
import math
from pathlib import Path
from typing import Iterable, Sequence

import numpy as np

LIB_PATH = Path(__file__).resolve().parent / "libmezo.so"

OK, EINVAL, EDTYPE, EOVERLAP, EORDER, ERANGE, EHIP, ENOMEM = 0, -1, -2, -3, -4, -5, -6, -7
F32, BF16, NF4 = 0, 1, 2
#: NF4 elements per absmax value.
NF4_BLOCK = 64
GAUSS_FAST, GAUSS_PORTABLE = 0, 1
LINEAR, SIGNED_LOG = 0, 1
#: Signed-log slope of a base-2 log: code 127 decodes just inside fp32.
LOG2_ALPHA = 1.0 / math.log(2.0)
MAX_NUMEL = 1 << 34

#: Layout of mezo_seed_t: (machine u64, step u32, sample u32), 16 bytes.
SEED_DTYPE = np.dtype([("machine", "<u8"), ("step", "<u4"), ("sample", "<u4")])


class Seed(ctypes.Structure):
    _fields_ = [("machine", ctypes.c_uint64), ("step", ctypes.c_uint32),
                ("sample", ctypes.c_uint32)]


class Tensor(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("numel", ctypes.c_uint64),
                ("tensor_id", ctypes.c_uint32), ("dtype", ctypes.c_uint32),
                ("absmax", ctypes.c_void_p), ("first", ctypes.c_uint64)]


class Codec(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_uint32), ("scale", ctypes.c_float), ("alpha", ctypes.c_float)]


class Step(ctypes.Structure):
    _fields_ = [("seeds", ctypes.c_void_p), ("q", ctypes.c_void_p), ("K", ctypes.c_uint32),
                ("lr", ctypes.c_float)]


#: Every symbol include/mezo.h declares.
EXPORTS = ("mezo_paramset_create", "mezo_paramset_destroy", "mezo_paramset_numel",
           "mezo_paramset_set_gaussian",
           "mezo_perturb", "mezo_perturb_multi", "mezo_update_multi", "mezo_replay", "mezo_replay_noalloc",
           "mezo_perturb_from",
           "mezo_update_multi_from", "mezo_checksum", "quantize_projgrad",
           "mezo_dequantize", "mezo_nf4_quantize", "mezo_nf4_dequantize", "mezo_debug_generate", "mezo_debug_box_muller",
           "mezo_strerror", "mezo_last_error", "mezo_version")


def _load() -> ctypes.CDLL:
    # libmezo must run on the same HIP runtime as torch: the streams and device
    # pointers it receives belong to that runtime. torch carries its own copy
    # (same SONAME); importing torch first makes the dynamic loader bind
    # libmezo to it instead of loading a second runtime.
    import torch  # noqa: F401
    if not LIB_PATH.exists():
        raise ImportError(f"{LIB_PATH} is not built: run python -m paper_2306_10015_amd.build")
    L = ctypes.CDLL(str(LIB_PATH))
    vp, u32, u64, i32, f32 = (ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_int,
                               ctypes.c_float)
    L.mezo_paramset_create.argtypes = [ctypes.POINTER(Tensor), u32, ctypes.POINTER(vp)]
    L.mezo_paramset_create.restype = i32
    L.mezo_paramset_destroy.argtypes = [vp]
    L.mezo_paramset_destroy.restype = None
    L.mezo_paramset_numel.argtypes = [vp]
    L.mezo_paramset_numel.restype = u64
    L.mezo_paramset_set_gaussian.argtypes = [vp, u32]
    L.mezo_paramset_set_gaussian.restype = i32
    L.mezo_perturb.argtypes = [vp, Seed, f32, vp]
    L.mezo_perturb.restype = i32
    L.mezo_perturb_multi.argtypes = [vp, vp, vp, u32, vp]
    L.mezo_perturb_multi.restype = i32
    L.mezo_update_multi.argtypes = [vp, vp, vp, u32, ctypes.POINTER(Codec), f32, vp]
    L.mezo_update_multi.restype = i32
    L.mezo_replay.argtypes = [vp, ctypes.POINTER(Step), u32, ctypes.POINTER(Codec), vp]
    L.mezo_replay.restype = i32
    L.mezo_replay_noalloc.argtypes = [vp, ctypes.POINTER(Step), u32, ctypes.POINTER(Codec), vp]
    L.mezo_replay_noalloc.restype = i32
    L.mezo_perturb_from.argtypes = [vp, vp, Seed, f32, vp]
    L.mezo_perturb_from.restype = i32
    L.mezo_update_multi_from.argtypes = [vp, vp, vp, vp, u32, ctypes.POINTER(Codec), f32, vp]
    L.mezo_update_multi_from.restype = i32
    L.mezo_checksum.argtypes = [vp, vp, vp]
    L.mezo_checksum.restype = i32
    L.quantize_projgrad.argtypes = [vp, vp, u32, ctypes.POINTER(Codec)]
    L.quantize_projgrad.restype = i32
    L.mezo_dequantize.argtypes = [vp, vp, u32, ctypes.POINTER(Codec)]
    L.mezo_dequantize.restype = i32
    L.mezo_nf4_quantize.argtypes = [vp, u32, u64, vp, vp, vp]
    L.mezo_nf4_quantize.restype = i32
    L.mezo_nf4_dequantize.argtypes = [vp, vp, u64, vp, u32, vp]
    L.mezo_nf4_dequantize.restype = i32
    L.mezo_debug_generate.argtypes = [Seed, u32, u64, u64, u32, vp, vp, vp]
    L.mezo_debug_generate.restype = i32
    L.mezo_debug_box_muller.argtypes = [vp, u64, u32, vp, vp]
    L.mezo_debug_box_muller.restype = i32
    L.mezo_strerror.argtypes = [i32]
    L.mezo_strerror.restype = ctypes.c_char_p
    L.mezo_last_error.argtypes = []
    L.mezo_last_error.restype = ctypes.c_char_p
    L.mezo_version.argtypes = []
    L.mezo_version.restype = i32
    return L


lib = _load()


class MezoError(RuntimeError):
    def __init__(self, code: int, what: str):
        msg = lib.mezo_strerror(code).decode()
        if code in (EHIP, ENOMEM):
            msg += f" ({lib.mezo_last_error().decode()})"
        super().__init__(f"{what}: {msg} [code {code}]")
        self.code = code


def _check(rc: int, what: str) -> None:
    if rc != OK:
        raise MezoError(rc, what)


def codec(kind: int = LINEAR, scale: float = 1.0 / 127.0, alpha: float = LOG2_ALPHA) -> Codec:
    return Codec(kind, scale, alpha)


DEFAULT_CODEC = codec()


def _seed(s) -> Seed:
    if isinstance(s, Seed):
        return s
    if isinstance(s, np.void):
        return Seed(int(s["machine"]), int(s["step"]), int(s["sample"]))
    m, t, j = s
    return Seed(int(m), int(t), int(j))


def seeds_array(seeds) -> np.ndarray:
    """Any sequence of (machine, step, sample) -> contiguous SEED_DTYPE array."""
    if isinstance(seeds, np.ndarray) and seeds.dtype == SEED_DTYPE:
        return np.ascontiguousarray(seeds)
    out = np.zeros(len(seeds), dtype=SEED_DTYPE)
    for i, s in enumerate(seeds):
        out[i] = s if isinstance(s, np.void) else (int(s[0]), int(s[1]), int(s[2]))
    return out


def _stream_ptr(stream) -> int | None:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported parameter dtype {t.dtype}")


class NF4Tensor:
    """A tensor of ``numel`` elements in 4-bit NormalFloat storage (the 4-bit
    forward-only variant): ``codes`` (uint8, ceil(numel / 2) bytes, element
    2i in the low nibble of byte i) and ``absmax`` (float32, one per block of
    64 elements), both contiguous device tensors owned by torch."""

    def __init__(self, codes, absmax, numel: int):
        import torch
        if codes.dtype != torch.uint8 or absmax.dtype != torch.float32:
            raise TypeError("codes must be uint8 and absmax float32")
        if not (codes.is_cuda and absmax.is_cuda and codes.is_contiguous() and absmax.is_contiguous()):
            raise ValueError("codes and absmax must be contiguous CUDA tensors")
        if codes.numel() < (numel + 1) // 2 or absmax.numel() < (numel + NF4_BLOCK - 1) // NF4_BLOCK:
            raise ValueError("codes / absmax too small for numel")
        self.codes, self.absmax, self._numel = codes, absmax, int(numel)

    @classmethod
    def empty(cls, numel: int, device="cuda") -> "NF4Tensor":
        import torch
        return cls(torch.empty((numel + 1) // 2, dtype=torch.uint8, device=device),
                   torch.empty((numel + NF4_BLOCK - 1) // NF4_BLOCK, dtype=torch.float32, device=device),
                   numel)

    def numel(self) -> int:
        return self._numel

    @property
    def device(self):
        return self.codes.device

    @property
    def is_cuda(self) -> bool:
        return True


def nf4_quantize(values, out: NF4Tensor | None = None, stream=None) -> NF4Tensor:
    """values (contiguous fp32/bf16 device tensor) -> NF4 storage."""
    n = values.numel()
    out = NF4Tensor.empty(n, values.device) if out is None else out
    if out.numel() != n or not values.is_contiguous():
        raise ValueError("size mismatch or non-contiguous values")
    import torch
    with torch.cuda.device(values.device):
        _check(lib.mezo_nf4_quantize(values.data_ptr(), _dtype_code(values), n, out.codes.data_ptr(),
                                     out.absmax.data_ptr(), _stream_ptr(stream)), "mezo_nf4_quantize")
    return out


def nf4_dequantize(t: NF4Tensor, dtype=None, out=None, stream=None):
    """NF4 storage -> a fp32 (default) or bf16 device tensor of numel elements."""
    import torch
    if out is None:
        out = torch.empty(t.numel(), dtype=dtype or torch.float32, device=t.device)
    if out.numel() != t.numel() or not out.is_contiguous():
        raise ValueError("size mismatch or non-contiguous out")
    with torch.cuda.device(t.device):
        _check(lib.mezo_nf4_dequantize(t.codes.data_ptr(), t.absmax.data_ptr(), t.numel(), out.data_ptr(),
                                       _dtype_code(out), _stream_ptr(stream)), "mezo_nf4_dequantize")
    return out


def _tensor_struct(t, tid: int, first: int = 0) -> Tensor:
    if isinstance(t, NF4Tensor):
        return Tensor(t.codes.data_ptr(), t.numel(), tid, NF4, t.absmax.data_ptr(), first)
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError("parameters must be contiguous CUDA tensors")
    return Tensor(t.data_ptr(), t.numel(), tid, _dtype_code(t), None, first)


class ParamSet:
    """A registered set of parameter tensors (device memory owned by torch):
    fp32 / bf16 torch tensors or NF4Tensor objects.

    ``tensor_ids`` default to the position in ``tensors``; they select each
    tensor's noise stream and must be the same on every machine. ``firsts``
    (default all 0) give, for a shard of a tensor split by element range, the
    index of its first element within the whole tensor (a multiple of 8): the
    shard then computes exactly those elements of the whole tensor.
    """

    def __init__(self, tensors: Sequence, tensor_ids: Iterable[int] | None = None,
                 gaussian: int = GAUSS_FAST, firsts: Iterable[int] | None = None):
        self.tensors = list(tensors)
        devices = set()
        for t in self.tensors:
            devices.add(t.device)
            if isinstance(t, NF4Tensor):
                devices.add(t.absmax.device)
        if len(devices) > 1:
            raise ValueError(f"all tensors of a paramset must live on one device, got {sorted(map(str, devices))}")
        #: the device every call of this paramset runs on (made current for the call)
        self.device = devices.pop() if devices else None
        import torch
        self._switch = torch.cuda.device_count() > 1
        ids = list(range(len(self.tensors))) if tensor_ids is None else [int(i) for i in tensor_ids]
        if len(ids) != len(self.tensors):
            raise ValueError("one tensor_id per tensor")
        offs = [0] * len(self.tensors) if firsts is None else [int(f) for f in firsts]
        if len(offs) != len(self.tensors):
            raise ValueError("one first-element offset per tensor")
        arr = (Tensor * max(1, len(self.tensors)))()
        for i, (t, tid, f) in enumerate(zip(self.tensors, ids, offs)):
            arr[i] = _tensor_struct(t, tid, f)
        h = ctypes.c_void_p()
        _check(lib.mezo_paramset_create(arr, len(self.tensors), ctypes.byref(h)),
               "mezo_paramset_create")
        self._h = h
        self.tensor_ids = ids
        if gaussian != GAUSS_FAST:
            self.set_gaussian(gaussian)

    def set_gaussian(self, gaussian: int) -> None:
        """GAUSS_FAST (hardware transcendentals) or GAUSS_PORTABLE (binary32
        operations only: bit-identical on any IEEE device)."""
        _check(lib.mezo_paramset_set_gaussian(self._h, int(gaussian)), "mezo_paramset_set_gaussian")

    def _on_device(self):
        """Make the paramset's device current for a call (a stream or pointer
        of another device would not be valid for its kernels); with a single
        visible device there is nothing to switch."""
        import contextlib
        import torch
        return torch.cuda.device(self.device) if self._switch else contextlib.nullcontext()

    @property
    def handle(self) -> ctypes.c_void_p:
        return self._h

    @property
    def numel(self) -> int:
        return int(lib.mezo_paramset_numel(self._h))

    def close(self) -> None:
        if getattr(self, "_h", None) is not None and self._h.value:
            lib.mezo_paramset_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def perturb(self, seed, scale: float, stream=None) -> None:
        """PerturbParameters: theta += scale * z(seed)."""
        with self._on_device():
            _check(lib.mezo_perturb(self._h, _seed(seed), float(scale), _stream_ptr(stream)),
                   "mezo_perturb")

    def perturb_multi(self, seeds, scales, stream=None) -> None:
        """Perturbs in sequence in one pass: theta += scales[i] * z(seeds[i]),
        rounded after each (e.g. restore sample j and perturb for sample j+1)."""
        sa = seeds_array(seeds)
        sc = np.ascontiguousarray(scales, dtype=np.float32)
        if sa.size != sc.size:
            raise ValueError("seeds and scales differ in length")
        with self._on_device():
            _check(lib.mezo_perturb_multi(self._h, sa.ctypes.data, sc.ctypes.data, sa.size, _stream_ptr(stream)),
                   "mezo_perturb_multi")

    def update_multi(self, seeds, q, lr: float, codec_: Codec = DEFAULT_CODEC, stream=None) -> None:
        """Apply loop of one iteration: theta -= lr * sum_k deq(q_k) z(seed_k)."""
        sa = seeds_array(seeds)
        qa = np.ascontiguousarray(q, dtype=np.int8)
        if sa.size != qa.size:
            raise ValueError("seeds and q differ in length")
        with self._on_device():
            _check(lib.mezo_update_multi(self._h, sa.ctypes.data, qa.ctypes.data, sa.size,
                                         ctypes.byref(codec_), float(lr), _stream_ptr(stream)),
                   "mezo_update_multi")

    def perturb_from(self, src: "ParamSet", seed, scale: float, stream=None) -> None:
        """theta = theta_src + scale * z(seed), src unchanged (out of place)."""
        with self._on_device():
            _check(lib.mezo_perturb_from(self._h, src.handle, _seed(seed), float(scale),
                                         _stream_ptr(stream)), "mezo_perturb_from")

    def update_multi_from(self, src: "ParamSet", seeds, q, lr: float,
                          codec_: Codec = DEFAULT_CODEC, stream=None) -> None:
        """theta = theta_src - lr * sum_k deq(q_k) z(seed_k): restore from the
        backup and apply the iteration's gradients in one pass."""
        sa = seeds_array(seeds)
        qa = np.ascontiguousarray(q, dtype=np.int8)
        if sa.size != qa.size:
            raise ValueError("seeds and q differ in length")
        with self._on_device():
            _check(lib.mezo_update_multi_from(self._h, src.handle, sa.ctypes.data, qa.ctypes.data,
                                              sa.size, ctypes.byref(codec_), float(lr),
                                              _stream_ptr(stream)), "mezo_update_multi_from")

    def checksum_into(self, out, stream=None) -> None:
        """Enqueue the 64-bit checksum of every tensor's bits into `out`, a
        device tensor of 8 bytes (ChecksumMatch, Algorithm 1)."""
        if out.numel() * out.element_size() != 8 or not out.is_cuda:
            raise ValueError("out must be an 8-byte device tensor")
        with self._on_device():
            _check(lib.mezo_checksum(self._h, out.data_ptr(), _stream_ptr(stream)), "mezo_checksum")

    def checksum(self, stream=None) -> int:
        """The checksum as a Python int (waits for the stream it ran on)."""
        import torch
        out = torch.empty(1, dtype=torch.int64, device=self.device)
        self.checksum_into(out, stream)
        if stream is not None:
            # .item() reads on the current stream, which does not wait for `stream`
            if isinstance(stream, torch.cuda.Stream):
                stream.synchronize()
            else:
                torch.cuda.synchronize(self.device)
        return int(out.item()) & 0xFFFFFFFFFFFFFFFF

    def replay(self, steps, codec_: Codec = DEFAULT_CODEC, stream=None) -> None:
        """Late-joiner catch-up: steps = [(seeds, q, lr), ...] in order."""
        self._replay(lib.mezo_replay, "mezo_replay", steps, codec_, stream)

    def replay_noalloc(self, steps, codec_: Codec = DEFAULT_CODEC, stream=None) -> None:
        """replay through mezo_replay_noalloc, the entry point that allocates
        nothing (at most 65536 records; the set must have had a call of
        another engine entry point first)."""
        self._replay(lib.mezo_replay_noalloc, "mezo_replay_noalloc", steps, codec_, stream)

    def _replay(self, fn, what, steps, codec_, stream) -> None:
        keep = []
        arr = (Step * max(1, len(steps)))()
        for i, (s, q, lr) in enumerate(steps):
            sa = seeds_array(s)
            qa = np.ascontiguousarray(q, dtype=np.int8)
            if sa.size != qa.size:
                raise ValueError(f"step {i}: seeds and q differ in length")
            keep.append((sa, qa))
            arr[i] = Step(sa.ctypes.data, qa.ctypes.data, sa.size, float(lr))
        with self._on_device():
            _check(fn(self._h, arr, len(steps), ctypes.byref(codec_), _stream_ptr(stream)), what)


def step_lr(eta: float, n_grads: int, sqrt_scaling: bool = False) -> float:
    """The per-gradient learning rate of one iteration's apply loop: each
    projected gradient is weighted by eta / n_grads (Algorithm 1); with the
    learning rate scaled by the square root of the number of perturbations
    (Section 4) that is eta * sqrt(n) / n = eta / sqrt(n)."""
    if n_grads <= 0:
        raise ValueError("n_grads must be positive")
    return eta / math.sqrt(n_grads) if sqrt_scaling else eta / n_grads


def quantize_projgrad(g, codec_: Codec = DEFAULT_CODEC) -> np.ndarray:
    ga = np.ascontiguousarray(g, dtype=np.float32)
    q = np.zeros(ga.size, dtype=np.int8)
    _check(lib.quantize_projgrad(ga.ctypes.data, q.ctypes.data, ga.size, ctypes.byref(codec_)),
           "quantize_projgrad")
    return q


def dequantize(q, codec_: Codec = DEFAULT_CODEC) -> np.ndarray:
    qa = np.ascontiguousarray(q, dtype=np.int8)
    g = np.zeros(qa.size, dtype=np.float32)
    _check(lib.mezo_dequantize(qa.ctypes.data, g.ctypes.data, qa.size, ctypes.byref(codec_)),
           "mezo_dequantize")
    return g


def debug_generate(seed, tensor_id: int, first: int, count: int, words=True, z=True,
                   stream=None, gaussian: int = GAUSS_FAST):
    """Device tensors (words uint32 as int32 bits, z float32) of elements
    first .. first+count-1 of tensor tensor_id under seed."""
    import torch
    w = torch.empty(count, dtype=torch.int32, device="cuda") if words else None
    zz = torch.empty(count, dtype=torch.float32, device="cuda") if z else None
    _check(lib.mezo_debug_generate(_seed(seed), int(tensor_id), int(first), int(count),
                                   int(gaussian), None if w is None else w.data_ptr(),
                                   None if zz is None else zz.data_ptr(), _stream_ptr(stream)),
           "mezo_debug_generate")
    return w, zz


def debug_box_muller(words, gaussian: int = GAUSS_FAST, stream=None):
    """z (float32 device tensor) of the given words (int32/uint32-bit device
    tensor, a multiple of 4 long), through the library's Gaussian transform."""
    import torch
    if words.numel() % 4 or not words.is_contiguous() or words.element_size() != 4:
        raise ValueError("words: contiguous 32-bit device tensor, a multiple of 4 long")
    z = torch.empty(words.numel(), dtype=torch.float32, device=words.device)
    _check(lib.mezo_debug_box_muller(words.data_ptr(), words.numel() // 4, int(gaussian), z.data_ptr(),
                                     _stream_ptr(stream)), "mezo_debug_box_muller")
    return z


def version() -> int:
    return int(lib.mezo_version())
