"""Seeded synthetic inputs for the perturbation engine.

This module holds no arithmetic of the method (no RNG of the engine, no
Gaussian transform, no update rule). It only describes the parameter sets and
draws the starting weights, seeds and one-byte gradients with numpy's PCG64,
so that the HIP path and the CPU oracle can be fed identical inputs.

The parameter sets stand in for the models of the paper's experiment (OPT,
Section 3): the same tensor shapes, in registration order (= tensor_id),
with weights drawn from N(0, 0.02), since trained checkpoints are not used.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

#: Memory layout of one seed (machine u64, step u32, sample u32), 16 bytes.
SEED_DTYPE = np.dtype([("machine", "<u8"), ("step", "<u4"), ("sample", "<u4")])

F32, BF16, NF4 = "f32", "bf16", "nf4"
NF4_BLOCK = 64


def _opt_shapes(d: int, ffn: int, layers: int, vocab: int = 50272):
    """OPT-style decoder weights: embedding, per layer q/k/v/o, fc1, fc2 and
    two LayerNorms (weight and bias), then the final LayerNorm."""
    shapes = [("embed_tokens", (vocab, d))]
    for i in range(layers):
        p = f"layers.{i}."
        for n in ("q_proj", "k_proj", "v_proj", "out_proj"):
            shapes.append((p + n, (d, d)))
        shapes.append((p + "fc1", (d, ffn)))
        shapes.append((p + "fc2", (ffn, d)))
        for n in ("ln1.weight", "ln1.bias", "ln2.weight", "ln2.bias"):
            shapes.append((p + n, (d,)))
    shapes.append(("final_ln.weight", (d,)))
    shapes.append(("final_ln.bias", (d,)))
    return shapes


@dataclass(frozen=True)
class Workload:
    name: str
    shapes: list = field(hash=False)
    dtype: str
    K: int
    eps: float = 1e-3
    lr: float = 1e-6
    grad_kind: str = "uniform"      # "uniform": ints in [-127, 127]; "normal40": rne(N(0,40))
    machines: int = 0               # seeds = machines x samples_per_machine
    samples_per_machine: int = 1
    T: int = 0                      # > 0: a replay log of T steps

    @property
    def numel(self) -> int:
        return int(sum(int(np.prod(s)) for _, s in self.shapes))

    @property
    def n_tensors(self) -> int:
        return len(self.shapes)


WORKLOADS = {
    "tiny": Workload("tiny", [(f"w{i}", (256, 1024)) for i in range(4)], F32, K=4,
                     machines=4, samples_per_machine=1),
    "opt125m": Workload("opt125m", _opt_shapes(768, 3072, 12), F32, K=8,
                        machines=8, samples_per_machine=1),
    "opt1.3b": Workload("opt1.3b", _opt_shapes(2048, 8192, 24), BF16, K=16,
                        grad_kind="normal40", machines=4, samples_per_machine=4),
    "opt6.7b": Workload("opt6.7b", _opt_shapes(4096, 16384, 32), BF16, K=64,
                        machines=64, samples_per_machine=1),
    "replay1.3b": Workload("replay1.3b", _opt_shapes(2048, 8192, 24), BF16, K=32,
                           machines=4, samples_per_machine=8, T=200),
    # the 4-bit forward-only variant (Section 3) on the paper's model size
    "opt6.7b-nf4": Workload("opt6.7b-nf4", _opt_shapes(4096, 16384, 32), NF4, K=64,
                            machines=64, samples_per_machine=1),
    "opt1.3b-nf4": Workload("opt1.3b-nf4", _opt_shapes(2048, 8192, 24), NF4, K=16,
                            grad_kind="normal40", machines=4, samples_per_machine=4),
}


def seeds(machines: int, samples_per_machine: int, step: int = 0,
          machine_base: int = 0) -> np.ndarray:
    """(machine, step, sample) for every machine and sample, in ascending
    (machine, step, sample) order: the order the apply loop walks them."""
    out = np.zeros(machines * samples_per_machine, dtype=SEED_DTYPE)
    i = 0
    for m in range(machines):
        for j in range(samples_per_machine):
            out[i] = (machine_base + m, step, j)
            i += 1
    return out


def workload_seeds(w: Workload, step: int = 0) -> np.ndarray:
    return seeds(w.machines, w.samples_per_machine, step=step)


def grads_int8(n: int, kind: str = "uniform", seed: int = 1) -> np.ndarray:
    """One-byte projected gradients: uniform ints in [-127, 127], or
    round-half-even of N(0, 40) clipped to +-127."""
    rng = np.random.Generator(np.random.PCG64(seed))
    if kind == "uniform":
        return rng.integers(-127, 128, size=n, dtype=np.int64).astype(np.int8)
    if kind == "normal40":
        return np.clip(np.rint(rng.normal(0.0, 40.0, size=n)), -127, 127).astype(np.int8)
    raise ValueError(kind)


def projected_grads(n: int, seed: int = 3, spread: float = 0.5) -> np.ndarray:
    """Float projected gradients (l+ - l-)/(2 eps) stand-ins: N(0, spread)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return rng.normal(0.0, spread, size=n).astype(np.float32)


def bf16_bits_truncated(x: np.ndarray) -> np.ndarray:
    """bf16 bit patterns of fp32 draws: the top 16 bits of each (truncation;
    starting weights only, not the method's rounding)."""
    return (np.ascontiguousarray(x, dtype=np.float32).view(np.uint32) >> 16).astype(np.uint16)


def bf16_bits_to_fp32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def theta0_tensor(shape, dtype: str, tensor_id: int, seed: int = 0) -> np.ndarray:
    """Starting weights of one tensor: N(0, 0.02) fp32 from PCG64(seed, tensor_id);
    bf16 storage as the truncated bit patterns of those draws (uint16)."""
    rng = np.random.Generator(np.random.PCG64([seed, tensor_id]))
    x = rng.standard_normal(size=int(np.prod(shape)), dtype=np.float32) * np.float32(0.02)
    return x if dtype == F32 else bf16_bits_truncated(x)


def nf4_theta0_tensor(numel: int, tensor_id: int, seed: int = 0):
    """Starting 4-bit storage of one tensor: packed code bytes uniform over all
    16 codes (NF4's values are quantiles of the normal law, so the codes of
    normal weights are close to uniform) with the unused high nibble of an
    odd-length tensor zero, and absmax = 0.02 * U(2, 3) per 64-element block
    (where the largest |N(0, 0.02)| of 64 draws usually falls)."""
    rng = np.random.Generator(np.random.PCG64([seed, tensor_id, 4]))
    packed = rng.integers(0, 256, size=(numel + 1) // 2, dtype=np.int64).astype(np.uint8)
    if numel % 2:
        packed[-1] &= 0x0F
    absmax = (np.float32(0.02) * rng.uniform(2.0, 3.0, size=(numel + NF4_BLOCK - 1) // NF4_BLOCK)
              .astype(np.float32)).astype(np.float32)
    return packed, absmax


def theta0(w: Workload, seed: int = 0) -> list:
    return [theta0_tensor(s, w.dtype, i, seed) for i, (_, s) in enumerate(w.shapes)]


def sample_indices(numel: int, rng: np.random.Generator, edge: int = 4096,
                   blocks: int = 64) -> np.ndarray:
    """Element indices to check one large tensor on: the first and last `edge`
    elements and `blocks` random 4-aligned blocks of 4 (sorted, unique)."""
    parts = [np.arange(min(edge, numel), dtype=np.uint64),
             np.arange(max(0, numel - edge), numel, dtype=np.uint64)]
    if numel > 8:
        b = rng.integers(0, numel // 4, size=blocks, dtype=np.int64).astype(np.uint64) * 4
        parts.append((b[:, None] + np.arange(4, dtype=np.uint64)[None, :]).ravel())
    ix = np.unique(np.concatenate(parts))
    return ix[ix < numel]
