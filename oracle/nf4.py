"""Oracle of the 4-bit forward-only variant (Section 3: the layer weights are
dequantized before the noise is added and quantized again afterwards; the
4-bit format is the one of QLoRA, Dettmers et al. 2023, which the paper
cites there).

TEST INFRASTRUCTURE ONLY, like the rest of ``oracle/``: only the tests,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` use it.

Storage (reading of the paper, which names the format only through its
citation): QLoRA's 4-bit NormalFloat (NF4) with blocks of 64 consecutive
elements of a tensor and one fp32 absmax per block (QLoRA's first
quantization level; its second level only compresses the absmax values and is
not used). A tensor of n elements is n 4-bit codes, two per byte (element 2i in
the low nibble of byte i), and ceil(n / 64) absmax values.

One step on a block (every call ends its steps with it):

1. dequantize: w_j = fl32(v[c_j] * a), v the NF4 values, a the block's absmax;
2. apply the step's perturbations exactly as for fp32 storage: the oracle's
   fp32 ``update`` / ``perturb`` (fp64 sum, one rounding to fp32), or their
   portable binary32 forms;
3. quantize again: a' = max_j |w'_j|; if a' = 0 every code is the zero code;
   else r = fl32(1 / a'), x_j = fl32(w'_j * r) and c'_j = the number of NF4
   midpoints m_i = fl32((v_i + v_{i+1}) / 2) below x_j (strictly): the
   nearest value, a tie going to the lower code.

Calls that apply nothing (scale 0, every code zero, no records) leave the
storage as it is, as for the other storage types.
"""
from __future__ import annotations

import numpy as np

import oracle as _orc

BLOCK = 64
ZERO_CODE = 7


def table() -> np.ndarray:
    """The 16 NF4 values as fp32, ascending, from QLoRA's construction:
    quantiles of N(0, 1) for an asymmetric pair of halves (8 positive values
    at probabilities spaced evenly from delta down to 1/2, 7 negative ones
    likewise with one point fewer, 1/2 itself dropped), plus an exact zero,
    divided by the largest value; delta = 1 - (1/32 + 1/30) / 2 puts the
    outermost probabilities halfway between those of 2^4 and 2^4 - 1 equal
    bins. fp64 throughout, one rounding to fp32 at the end."""
    from scipy.stats import norm
    delta = 1.0 - 0.5 * (1.0 / 32.0 + 1.0 / 30.0)
    pos = norm.ppf(np.linspace(delta, 0.5, 9)[:-1])
    neg = -norm.ppf(np.linspace(delta, 0.5, 8)[:-1])
    v = np.sort(np.concatenate([neg, [0.0], pos]))
    return (v / v[-1]).astype(np.float32)


def midpoints(v: np.ndarray | None = None) -> np.ndarray:
    """fl32 of the exact midpoint of each pair of neighbouring values."""
    v = table() if v is None else v
    v64 = v.astype(np.float64)
    return ((v64[:-1] + v64[1:]) * 0.5).astype(np.float32)


def block_lengths(numel: int, blocks) -> np.ndarray:
    b = np.asarray(blocks, dtype=np.int64)
    return np.minimum(BLOCK, numel - BLOCK * b)


def block_elements(numel: int, blocks) -> np.ndarray:
    """Element indices of the listed blocks, concatenated in list order."""
    b = np.asarray(blocks, dtype=np.int64)
    if b.size == 0:
        return np.zeros(0, dtype=np.int64)
    return np.concatenate([np.arange(BLOCK * i, min(BLOCK * (i + 1), numel)) for i in b])


def _blocks(numel: int, blocks):
    nb = (numel + BLOCK - 1) // BLOCK
    return np.arange(nb) if blocks is None else np.asarray(blocks, dtype=np.int64)


def _segments(lens: np.ndarray) -> np.ndarray:
    """Start offset of each block's elements in a concatenated array."""
    return np.concatenate([[0], np.cumsum(lens)[:-1]]).astype(np.int64)


def dequantize(codes: np.ndarray, absmax: np.ndarray, numel: int | None = None, blocks=None) -> np.ndarray:
    """Step 1: w = fl32(v[c] * a) for the elements of the listed blocks (all
    blocks by default); ``codes`` holds one code per element (unpacked)."""
    codes = np.asarray(codes, dtype=np.uint8)
    n = codes.size if numel is None else numel
    b = _blocks(n, blocks)
    lens = block_lengths(n, b)
    if codes.size != lens.sum() or np.asarray(absmax).size != b.size:
        raise ValueError("codes / absmax do not match the blocks")
    a = np.repeat(np.asarray(absmax, dtype=np.float32), lens)
    return table()[codes] * a


def quantize(w: np.ndarray, numel: int | None = None, blocks=None):
    """Step 3: (codes, absmax) of fp32 values w of the listed blocks."""
    w = np.asarray(w, dtype=np.float32)
    n = w.size if numel is None else numel
    b = _blocks(n, blocks)
    lens = block_lengths(n, b)
    if w.size != lens.sum():
        raise ValueError("w does not match the blocks")
    mid = midpoints()
    # blocks as rows of 64, padded with zeros (which change no maximum and
    # whose codes are dropped)
    rows = np.zeros((b.size, BLOCK), dtype=np.float32)
    valid = np.arange(BLOCK)[None, :] < lens[:, None]
    rows[valid] = w
    absmax = np.max(np.abs(rows), axis=1) if b.size else np.zeros(0, np.float32)
    codes = np.full(rows.shape, ZERO_CODE, dtype=np.uint8)
    for lo in range(0, b.size, 4096):
        a = absmax[lo:lo + 4096]
        nz = a != 0
        r = np.ones_like(a)
        r[nz] = np.float32(1.0) / a[nz]
        x = rows[lo:lo + 4096] * r[:, None]
        c = np.sum(x[:, :, None] > mid[None, None, :], axis=2).astype(np.uint8)
        codes[lo:lo + 4096][nz] = c[nz]
    return codes[valid], absmax.astype(np.float32)


def pack(codes: np.ndarray) -> np.ndarray:
    """Two codes per byte, element 2i in the low nibble of byte i."""
    c = np.asarray(codes, dtype=np.uint8)
    if c.size % 2:
        c = np.concatenate([c, np.zeros(1, np.uint8)])
    return (c[0::2] | (c[1::2] << 4)).astype(np.uint8)


def unpack(packed: np.ndarray, numel: int) -> np.ndarray:
    p = np.asarray(packed, dtype=np.uint8)
    c = np.empty(2 * p.size, dtype=np.uint8)
    c[0::2] = p & 0xF
    c[1::2] = p >> 4
    return c[:numel]


def _apply(codes, absmax, numel, blocks, fn):
    n = np.asarray(codes).size if numel is None else numel
    b = _blocks(n, blocks)
    w = dequantize(codes, absmax, n, b)
    fn(w, block_elements(n, b))
    return quantize(w, n, b)


def perturb(codes, absmax, tensor_id: int, seed, scale: float, numel: int | None = None, blocks=None,
            portable: bool = False):
    """PerturbParameters on NF4 storage: (codes', absmax')."""
    if scale == 0:
        return np.array(codes, dtype=np.uint8), np.array(absmax, dtype=np.float32)
    return _apply(codes, absmax, numel, blocks,
                  lambda w, ix: _orc.perturb(w, tensor_id, seed, scale, idx=ix, portable=portable))


def _effective(q, lr, kind, scale, alpha) -> bool:
    return np.any(_orc.coefficients(q, lr, kind, scale, alpha) != 0) if len(q) else False


def update(codes, absmax, tensor_id: int, seeds, q, lr: float, kind: int = _orc.LINEAR,
           scale: float = 1.0 / 127.0, alpha: float = _orc.LOG2_ALPHA, numel: int | None = None,
           blocks=None, portable: bool = False):
    """The fused apply loop on NF4 storage: one dequantize, the K
    perturbations, one quantize."""
    if not _effective(q, lr, kind, scale, alpha):
        return np.array(codes, dtype=np.uint8), np.array(absmax, dtype=np.float32)
    return _apply(codes, absmax, numel, blocks,
                  lambda w, ix: _orc.update(w, tensor_id, seeds, q, lr, kind, scale, alpha, idx=ix,
                                            portable=portable))


def replay(codes, absmax, tensor_id: int, steps, kind: int = _orc.LINEAR, scale: float = 1.0 / 127.0,
           alpha: float = _orc.LOG2_ALPHA, numel: int | None = None, blocks=None, portable: bool = False):
    """Late-joiner replay on NF4 storage: the steps one after another, each
    ending with a quantization."""
    c = np.array(codes, dtype=np.uint8)
    a = np.array(absmax, dtype=np.float32)
    for seeds, q, lr in steps:
        c, a = update(c, a, tensor_id, seeds, q, lr, kind, scale, alpha, numel, blocks, portable)
    return c, a


def image(packed: np.ndarray, absmax: np.ndarray) -> np.ndarray:
    """The bytes a checksum covers: the packed codes zero-padded to a multiple
    of 8 bytes, then the absmax values (little-endian fp32)."""
    p = np.asarray(packed, dtype=np.uint8)
    pad = (-p.size) % 8
    return np.concatenate([p, np.zeros(pad, np.uint8),
                           np.ascontiguousarray(absmax, dtype="<f4").view(np.uint8)])


def checksum_tensor(packed: np.ndarray, absmax: np.ndarray, tensor_id: int) -> int:
    return _orc.checksum_tensor(image(packed, absmax), tensor_id)

