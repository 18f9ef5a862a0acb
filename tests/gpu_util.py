"""Helpers of the GPU parity tests: moving seeded synthetic tensors between
host and device, and the comparison bars.

Bars: RNG words and int8 codes bit-exact; fp32 weights within
max|theta_gpu - theta_ref| <= 1e-6 * max|theta_ref|; Gaussians within
max|z_gpu - z_ref| <= 1e-6 * max|z_ref|; bf16 weights within one bf16 ulp
at the scale of the operation's operands: ordered-integer distance of the bit
patterns <= 1, or, where theta + delta cancelled to a result smaller than its
input, |theta_gpu - theta_ref| <= one bf16 ulp of max(|theta_in|,
|theta_ref|). (At a cancellation the result's own ulp is smaller than the
error the Gaussian tolerance permits, eps * 1e-6 * max|z|, so no z that is
not bit-exact can meet a result-ulp bar there.)
"""
from __future__ import annotations

import numpy as np

from paper_2306_10015_amd import synth

F32_REL = 1e-6
Z_REL = 1e-6


def to_device(host: np.ndarray):
    import torch
    if host.dtype == np.float32:
        return torch.from_numpy(host.copy()).cuda()
    if host.dtype == np.uint16:
        return torch.from_numpy(host.view(np.int16).copy()).view(torch.bfloat16).cuda()
    raise TypeError(host.dtype)


def to_host(t) -> np.ndarray:
    import torch
    if t.dtype == torch.float32:
        return t.detach().cpu().numpy().copy()
    if t.dtype == torch.bfloat16:
        return t.detach().view(torch.int16).cpu().numpy().view(np.uint16).copy()
    raise TypeError(t.dtype)


def bf16_ordered(bits: np.ndarray) -> np.ndarray:
    b = bits.astype(np.int64)
    mag = b & 0x7FFF
    return np.where(b & 0x8000, -mag, mag)


def bf16_ulp_distance(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    return np.abs(bf16_ordered(a) - bf16_ordered(b))


def bf16_ulp_of(v: np.ndarray) -> np.ndarray:
    """Spacing of bf16 values around |v| (fp64 in, fp64 out)."""
    a = np.abs(np.asarray(v, dtype=np.float64))
    e = np.floor(np.log2(np.maximum(a, 2.0 ** -126)))
    return 2.0 ** (e - 7)


def assert_theta_close(got: np.ndarray, want: np.ndarray, what: str = "",
                       inp: np.ndarray | None = None) -> dict:
    """Apply the parity bar for the storage type; return summary figures.
    `inp` is the operation's input theta (bf16 bits) for the operand-scale
    ulp of the bf16 bar."""
    assert got.shape == want.shape and got.dtype == want.dtype
    if got.dtype == np.float32:
        scale = float(np.max(np.abs(want.astype(np.float64)))) if want.size else 0.0
        err = float(np.max(np.abs(got.astype(np.float64) - want.astype(np.float64)))) if want.size else 0.0
        tol = F32_REL * scale
        assert err <= tol, f"{what}: max abs err {err:.3e} > {tol:.3e}"
        exact = float(np.mean(got.view(np.uint32) == want.view(np.uint32))) if want.size else 1.0
        return {"max_abs_err": err, "tol": tol, "exact_frac": exact}
    d = bf16_ulp_distance(got, want)
    mx = int(d.max()) if d.size else 0
    far = d > 1
    n_cancel = int(far.sum())
    if n_cancel:
        assert inp is not None, f"{what}: bf16 distance {mx} ulp > 1 and no input given"
        g = synth.bf16_bits_to_fp32(got[far]).astype(np.float64)
        w = synth.bf16_bits_to_fp32(want[far]).astype(np.float64)
        i = synth.bf16_bits_to_fp32(inp[far]).astype(np.float64)
        assert np.all(np.abs(w) < np.abs(i)), f"{what}: {mx} ulp off where nothing cancelled"
        lim = bf16_ulp_of(np.maximum(np.abs(i), np.abs(w)))
        assert np.all(np.abs(g - w) <= lim), f"{what}: cancelled elements off by more than an operand ulp"
    return {"max_ulp": mx, "ulp1_frac": float(np.mean(d == 1)) if d.size else 0.0,
            "cancelled_gt1ulp": n_cancel}


def z_close(got: np.ndarray, want: np.ndarray) -> dict:
    scale = float(np.max(np.abs(want.astype(np.float64))))
    err = float(np.max(np.abs(got.astype(np.float64) - want.astype(np.float64))))
    return {"max_abs_err": err, "tol": Z_REL * scale}


def theta_on_device(w: synth.Workload, seed: int = 0, device_rng: bool = False):
    """Seeded theta0 for a workload as a list of device tensors.

    Small sets are drawn with numpy PCG64 (synth.theta0_tensor) and uploaded;
    with device_rng, torch's seeded device generator draws N(0, 0.02) directly
    in HBM (the host reads back whatever elements it needs)."""
    import torch
    out = []
    if not device_rng:
        for i, (_, shape) in enumerate(w.shapes):
            out.append(to_device(synth.theta0_tensor(shape, w.dtype, i, seed)))
        return out
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    dt = torch.float32 if w.dtype == synth.F32 else torch.bfloat16
    for _, shape in w.shapes:
        t = torch.empty(int(np.prod(shape)), dtype=torch.float32, device="cuda")
        t.normal_(0.0, 0.02, generator=g)
        out.append(t.to(dt))
    return out
