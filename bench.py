"""Throughput of the seeded perturbation engine on one MI355X.

One step is one pass of the whole hot path over a synthetic OPT-125m-shaped
fp32 parameter set (123,581,952 elements in 123 tensors, N(0, 0.02)):

  1. PerturbParameters +eps, -2eps, +eps with this machine's seed
     (Algorithm 1, inner inference loop; eps = 1e-3);
  2. quantize_projgrad of the K = 8 projected gradients of the iteration
     (Section 3, one byte each; linear code, scale 1/127);
  3. update_multi: the fused apply loop over the K = 8 (machine, sample)
     seeds (Algorithm 1; lr = 1e-6);
  4. replay: a late joiner's catch-up over a log of T = 4 earlier iterations
     of K = 8 seeds each (Appendix B).

Every parameter is read and written once per call; z is regenerated in
registers. The metric is param-seed updates per second: elements x seeds
applied, summed over the step's calls, divided by the time of the step.

Prints ONE JSON line. Also reports, for the engine kernel (the only kernel of
the step), the ALU roofline fraction against 256 CUs x 4 SIMDs x 16 lanes x
2.4 GHz = 39.3e12 lane-instructions/s, each call timed alone (`ops`), and the
CPU oracle timed on a bounded sample of the same step.

    python bench.py [--gpus 1] [--steps 400] [--warmup 100] [--workload NAME]
                    [--gaussian fast|portable] [--no-ops] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

#: VALU issue capacity of one MI355X: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz
#: = 39.3e12 lane-instructions per second (a wave64 VALU instruction occupies a
#: 16-lane SIMD for 4 cycles when issued singly). It is the published
#: 157.3 TFLOP/s fp32 vector peak / (2 flops per fma x 2 lanes per packed op).
#: gfx950 can dual-issue some VALU instructions, so a kernel can exceed it.
CLOCK_GHZ = 2.4
VALU_LANE_INSTR_PER_S = 256 * 4 * 16 * CLOCK_GHZ * 1e9
HBM_PEAK_GBS = 8000.0
# each call timed alone: OPS_BATCHES batches of back-to-back launches, each
# lasting about OPS_LOOP_MS (at most OPS_MAX_REPS launches); the median batch
OPS_LOOP_MS = 30.0
OPS_MAX_REPS = 400
OPS_BATCHES = 10
# projected gradients per machine per iteration in the paper's runs (Section 3)
SAMPLES_PER_MACHINE = 16

#: VALU instructions per Philox block (4 Gaussians) per seed in the engine's
#: inner loop, the method's minimal sequence on gfx950: round 1 and the
#: element-independent half of round 2 hoisted out of the seed loop; rounds
#: 2..10 cost 17 wide multiplies (v_mad_u64_u32), 16 three-way xors
#: (v_bitop3_b32) and 3 xors; Box-Muller per pair of Gaussians (radius factor
#: sqrt(2 ln 2) folded into the coefficient): 2 shifts, 2 int->float
#: conversions, one fma forming u1, 2 muls (u2's scale, c_k times the radius),
#: log2, sqrt, sin, cos; and one fma per Gaussian accumulating into theta's
#: increment.
INNER_LOOP_MIX = {
    "v_mad_u64_u32": 17, "v_bitop3_b32": 16, "v_xor_b32": 3, "v_lshrrev_b32": 4,
    "v_cvt_f32_u32": 4, "v_fmamk_f32": 2, "v_mul_f32": 4, "v_log_f32": 2, "v_sqrt_f32": 2,
    "v_sin_f32": 2, "v_cos_f32": 2, "v_fmac_f32": 4,
}
#: lane-instructions per param-seed (= 62 / 4)
INSTR_PER_PARAM_SEED = sum(INNER_LOOP_MIX.values()) / 4.0

#: counter profile of the engine kernel on this workload (FETCH_SIZE /
#: WRITE_SIZE per dispatch, calibrated against a plain copy); its traffic is
#: reported only while the kernel sources it was taken on are unchanged.
TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "engine_kernel_{workload}_traffic.json")
KERNEL_SOURCES = ["paper_2306_10015_amd/csrc/kernels.hip", "paper_2306_10015_amd/csrc/engine.hpp",
                  "paper_2306_10015_amd/csrc/records.hpp", "paper_2306_10015_amd/csrc/nf4.hpp",
                  "paper_2306_10015_amd/csrc/launch.hpp"]

T_REPLAY = 4


def parse():
    p = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=400)
    p.add_argument("--warmup", type=int, default=100)
    p.add_argument("--workload", default="opt125m")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-ops", action="store_true",
                   help="skip the per-operation measurements after the timed region (profiling runs)")
    p.add_argument("--gaussian", choices=["fast", "portable"], default="fast",
                   help="how z is computed (portable: binary32 operations only, bit-identical "
                        "on any IEEE device)")
    p.add_argument("--probe", choices=["copy", "rmw"], default=None,
                   help="copy: time a plain device copy of the parameter buffer instead; rmw: an in-place "
                        "streaming read-modify-write of it with the engine's access pattern (the sweep's "
                        "memory ceiling)")
    p.add_argument("--rmw-groups", type=int, choices=[1, 2], default=None,
                   help="rmw probe: 16-byte groups per lane (default 1, the engine's)")
    p.add_argument("--rmw-lanes", type=int, choices=[128, 256, 512], default=256,
                   help="rmw probe: lanes per workgroup (default 256, the engine's)")
    p.add_argument("--cpu-seconds", type=float, default=12.0,
                   help="target CPU work of the oracle baseline sample")
    return p.parse_args()


def flat_views(torch, w, device):
    """One 256-byte-aligned allocation holding every tensor of the set."""
    import math
    esz = 4 if w.dtype == "f32" else 2
    align = 256 // esz
    offs, total = [], 0
    for _, shape in w.shapes:
        n = int(math.prod(shape))
        offs.append((total, n))
        total += (n + align - 1) // align * align
    dt = torch.float32 if w.dtype == "f32" else torch.bfloat16
    flat = torch.empty(total, dtype=dt, device=device)
    views = [flat[a:a + n] for a, n in offs]
    return flat, views, offs


def nf4_buffers(torch, mezo, synth, w, device):
    """4-bit storage of every tensor as views into one code buffer and one
    absmax buffer (each view 256-byte aligned)."""
    import math
    offs, ctot, atot = [], 0, 0
    for _, shape in w.shapes:
        n = int(math.prod(shape))
        cb, nb = (n + 1) // 2, (n + synth.NF4_BLOCK - 1) // synth.NF4_BLOCK
        offs.append((ctot, atot, n))
        ctot += (cb + 255) // 256 * 256
        atot += (nb + 63) // 64 * 64
    codes = torch.empty(ctot, dtype=torch.uint8, device=device)
    absmax = torch.empty(atot, dtype=torch.float32, device=device)

    def views_of(c, a):
        return [mezo.NF4Tensor(c[co:co + (n + 1) // 2], a[ao:ao + (n + synth.NF4_BLOCK - 1) // synth.NF4_BLOCK], n)
                for co, ao, n in offs]

    return codes, absmax, views_of


def storage_bytes(w) -> float:
    """Bytes of one element in storage (NF4: half a code byte plus its share
    of the block's 4-byte absmax)."""
    return {"f32": 4.0, "bf16": 2.0, "nf4": 0.5 + 4.0 / 64}[w.dtype]


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the engine has no multi-GPU path "
              f"(--gpus {args.gpus} requested). Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2306_10015_amd import mezo, synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = synth.WORKLOADS[args.workload]
    K = w.K
    N = w.numel
    gauss = mezo.GAUSS_PORTABLE if args.gaussian == "portable" else mezo.GAUSS_FAST

    # ---- inputs resident in HBM before timing -------------------------------
    if w.dtype == synth.NF4:
        codes, absmax, views_of = nf4_buffers(torch, mezo, synth, w, dev)
        views = views_of(codes, absmax)
        if N <= 200_000_000:
            # numpy PCG64 per tensor (the same storage the tests start from)
            for i, v in enumerate(views):
                p, a = synth.nf4_theta0_tensor(v.numel(), i, 0)
                v.codes.copy_(torch.from_numpy(p))
                v.absmax.copy_(torch.from_numpy(a))
        else:
            # the same distribution drawn in HBM by torch's seeded generator
            g = torch.Generator(device=dev)
            g.manual_seed(0)
            codes.random_(0, 256, generator=g)
            absmax.uniform_(0.04, 0.06, generator=g)
        flat = codes

        def make_backup():
            c2, a2 = codes.clone(), absmax.clone()
            return mezo.ParamSet(views_of(c2, a2), gaussian=gauss), (c2, a2)
    else:
        flat, views, offs = flat_views(torch, w, dev)
        if N <= 200_000_000:
            # numpy PCG64 per tensor (the same theta0 the tests and the oracle use)
            for i, (v, (_, shape)) in enumerate(zip(views, w.shapes)):
                h = synth.theta0_tensor(shape, w.dtype, i, 0)
                if w.dtype == "f32":
                    v.copy_(torch.from_numpy(h))
                else:
                    v.copy_(torch.from_numpy(h.view(np.int16)).view(torch.bfloat16))
        else:
            # billions of elements: N(0, 0.02) drawn in HBM by torch's seeded generator
            g = torch.Generator(device=dev)
            g.manual_seed(0)
            for v in views:
                tmp = torch.empty(v.numel(), dtype=torch.float32, device=dev)
                tmp.normal_(0.0, 0.02, generator=g)
                v.copy_(tmp)
                del tmp

        def make_backup():
            b = flat.clone()
            return mezo.ParamSet([b[a:a + n] for a, n in offs], gaussian=gauss), b
    if args.probe == "copy":
        copy_probe(torch, flat, args)
        return
    if args.probe == "rmw":
        rmw_probe(torch, flat, args)
        return
    ps = mezo.ParamSet(views, gaussian=gauss)
    eps, lr = w.eps, w.lr

    total_steps = args.warmup + args.steps
    proj = [synth.projected_grads(K, seed=1000 + t) for t in range(total_steps)]
    seeds_t = [synth.seeds(w.machines, w.samples_per_machine, step=t) for t in range(total_steps)]
    t_log = w.T if w.T > 0 else T_REPLAY
    log = [(synth.seeds(w.machines, w.samples_per_machine, step=10_000 + t),
            synth.grads_int8(K, "uniform", seed=2000 + t), lr) for t in range(t_log)]
    recs = {"perturb": 1, "update": K, "replay": t_log * K}
    # a replay workload's step is the catch-up alone; otherwise one iteration
    # of Algorithm 1 on this machine plus a short catch-up
    calls = ["replay"] if w.T > 0 else ["perturb", "perturb", "perturb", "update", "replay"]
    ps_per_step = N * sum(recs[c] for c in calls)

    stream = torch.cuda.current_stream()

    def step(t):
        s = (0, t, 0)
        if w.T == 0:
            ps.perturb(s, eps)
            ps.perturb(s, -2 * eps)
            ps.perturb(s, eps)
            q = mezo.quantize_projgrad(proj[t])
            ps.update_multi(seeds_t[t], q, lr)
        ps.replay(log)

    for t in range(args.warmup):
        step(t)
    torch.cuda.synchronize()

    # ---- timed region: exactly `steps` steps ---------------------------------
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record(stream)
    for t in range(args.warmup, total_steps):
        step(t)
    end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_total = start.elapsed_time(end)
    ms_per_step = ms_total / args.steps

    value = ps_per_step * args.steps / (ms_total / 1e3)
    bytes_per_launch = 2 * N * storage_bytes(w)

    # Engine kernel: every call of the step is one launch of it (per storage
    # type; the sets here have one). Its average launch duration is the timed
    # region's GPU time over its launches (the step enqueues nothing else on
    # the stream); achieved ALU work = param-seeds x minimal lane-instructions
    # per param-seed over that time.
    n_launch = len(calls)
    avg_launch_s = ms_per_step / n_launch / 1e3
    ps_per_launch = ps_per_step / n_launch
    achieved = ps_per_launch * INSTR_PER_PARAM_SEED / avg_launch_s / 1e12
    peak = VALU_LANE_INSTR_PER_S / 1e12
    # the step's launches bind differently (the sweeps HBM, the updates the
    # VALU): its ideal time puts every launch at its own roofline, the larger
    # of bytes / HBM peak and instructions / VALU peak
    ideal_ms = 1e3 * sum(max(bytes_per_launch / (HBM_PEAK_GBS * 1e9),
                             N * recs[c] * INSTR_PER_PARAM_SEED / VALU_LANE_INSTR_PER_S) for c in calls)
    ops = None if args.no_ops else measure_ops(torch, mezo, synth, w, ps, make_backup, stream, args,
                                               recs, proj, seeds_t, log, bytes_per_launch, flat)

    out = {
        "metric": "param-seed updates/sec (params x K per s)",
        "value": value,
        "unit": "param-seeds/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"{w.name}: {N} {w.dtype} params in {w.n_tensors} tensors, K={K}; "
                               + (f"step = replay T={t_log}xK={K}" if w.T > 0 else
                                  f"step = perturb +eps,-2eps,+eps; quantize {K} grads; "
                                  f"update_multi K={K}; replay T={t_log}xK={K}"),
                   "params": N, "tensors": w.n_tensors, "K": K, "replay_T": t_log,
                   "storage": w.dtype,
                   "gaussian": args.gaussian,
                   "eps": eps, "lr": lr, "param_seeds_per_step": ps_per_step},
        "roofline": {"bound": "alu", "achieved": achieved, "peak": peak,
                     "unit": "Tinstr/s", "frac": achieved / peak,
                     "traffic": measured_traffic(w.name, args.gaussian),
                     "alg_bytes_per_launch": bytes_per_launch,
                     "kernel": f"engine_kernel<{'inline' if max(recs[c] for c in calls) <= 32 else 'staged'}"
                               f" records, {w.dtype}>",
                     "instr_per_param_seed": INSTR_PER_PARAM_SEED,
                     "param_seeds_per_launch": ps_per_launch,
                     "avg_launch_ms": avg_launch_s * 1e3,
                     "step_ideal_ms": ideal_ms,
                     "combined_frac": ideal_ms / ms_per_step},
        "wall_s_timed": wall,
    }
    if ops is not None:
        out["ops"] = ops
        if "perturb" in ops and "stream_rmw_no_rng" in ops:
            # the memory-bound sweep against the same buffer's streaming ceiling
            out["roofline"]["sweep_frac_of_stream_ceiling"] = (ops["perturb"]["alg_GBps"]
                                                               / ops["stream_rmw_no_rng"]["alg_GBps"])
        out["issue_cycles_isolated"] = {k: round(v, 3) for k, v in issue_costs().items()}
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, recs, calls, log, args.cpu_seconds)
        out["gpu_over_cpu"] = value / out["cpu_baseline"]["value"]
    print(json.dumps(out))


def issue_costs() -> dict:
    """SIMD cycles per wave instruction of each instruction of the inner loop in
    isolation, measured now on this device by libisa_probe.so (8 waves per
    SIMD, 8 independent chains per lane): context for the instruction mix."""
    import ctypes
    from paper_2306_10015_amd import build as b
    if not b.PROBE_LIB.exists():
        raise RuntimeError(f"{b.PROBE_LIB} is not built")
    L = ctypes.CDLL(str(b.PROBE_LIB))
    L.isa_probe_count.restype = ctypes.c_int
    L.isa_probe_name.restype = ctypes.c_char_p
    L.isa_probe_name.argtypes = [ctypes.c_int]
    L.isa_probe_run.argtypes = [ctypes.POINTER(ctypes.c_double), ctypes.c_double]
    n = L.isa_probe_count()
    out = (ctypes.c_double * n)()
    rc = L.isa_probe_run(out, CLOCK_GHZ)
    if rc != 0:
        raise RuntimeError(f"isa_probe_run failed ({rc})")
    return {L.isa_probe_name(i).decode(): float(out[i]) for i in range(n)}


def kernel_source_hash() -> str:
    import hashlib
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(workload: str, gaussian: str = "fast"):
    """HBM bytes per engine launch from the committed counter profile of this
    workload, or None when there is none or the kernel sources changed since
    it was taken."""
    if gaussian != "fast":
        return None
    try:
        with open(TRAFFIC_PROFILE.format(workload=workload)) as f:
            prof = json.load(f)
    except (OSError, ValueError):
        return None
    if prof.get("kernel_source_sha256") != kernel_source_hash():
        return None
    return prof["hbm_bytes_per_dispatch"]


def measure_ops(torch, mezo, synth, w, ps, make_backup, stream, args, recs, proj, seeds_t, log,
                bytes_per_launch, flat):
    """Each operation alone, repeated back to back between two events on the
    kernels' stream (after the timed region, not part of the step)."""
    N, K, lr = w.numel, w.K, w.lr

    def loop(fn, reps):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(reps):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    def timed(fn):
        # warm up, then batches of about OPS_LOOP_MS so that short calls are
        # timed over many launches at the clock a long run settles at; the
        # median batch's average launch
        fn()
        torch.cuda.synchronize()
        once = loop(fn, 1)
        reps = max(1, min(OPS_MAX_REPS, math.ceil(OPS_LOOP_MS / max(once, 1e-3))))
        return statistics.median(loop(fn, reps) for _ in range(OPS_BATCHES))

    def entry(records, ms, nbytes=bytes_per_launch):
        t_s = ms / 1e3
        e = {"ms": round(ms, 4), "alg_GBps": nbytes / t_s / 1e9,
             "hbm_frac": nbytes / t_s / 1e9 / HBM_PEAK_GBS}
        if records:
            e.update({"records": records, "param_seeds_per_s": N * records / t_s,
                      "alu_frac": N * records * INSTR_PER_PARAM_SEED / t_s / VALU_LANE_INSTR_PER_S})
        return e

    q0 = mezo.quantize_projgrad(proj[0])
    ops = {}
    if w.T == 0:
        ops["perturb"] = entry(1, timed(lambda: ps.perturb((0, 0, 0), w.eps)))
        # Algorithm 1 between two samples: restore sample j and perturb for
        # sample j + 1 in one pass (two separate perturbs cost two)
        ops["restore_and_next_perturb"] = entry(
            2, timed(lambda: ps.perturb_multi([(0, 0, 0), (0, 0, 1)], [w.eps, w.eps])))
        ops["update"] = entry(K, timed(lambda: ps.update_multi(seeds_t[0], q0, lr)))
        # one iteration of Algorithm 1 on one machine without its forward
        # passes: SAMPLES_PER_MACHINE samples (Section 3: 16 per machine), each
        # perturbed by -2 eps, the restore of sample j fused with +eps of
        # sample j + 1, then the K-seed update
        samples = [(0, 1, j) for j in range(SAMPLES_PER_MACHINE)]

        def iteration():
            ps.perturb(samples[0], w.eps)
            for j, s in enumerate(samples):
                ps.perturb(s, -2 * w.eps)
                if j + 1 < len(samples):
                    ps.perturb_multi([s, samples[j + 1]], [w.eps, w.eps])
                else:
                    ps.perturb(s, w.eps)
            ps.update_multi(seeds_t[0], q0, lr)
        it_records = 1 + SAMPLES_PER_MACHINE + 2 * (SAMPLES_PER_MACHINE - 1) + 1 + K
        ops["iteration_16_samples"] = entry(it_records, timed(iteration),
                                            bytes_per_launch * (2 * SAMPLES_PER_MACHINE + 2))
    ops["replay"] = entry(recs["replay"], timed(lambda: ps.replay(log)))
    if w.dtype == synth.NF4:
        # the standalone conversions on the largest tensor (the embedding): a
        # QLoRA-style forward pass dequantizes the weights it reads
        big = max(ps.tensors, key=lambda t: t.numel())
        n = big.numel()
        vals = torch.empty(n, dtype=torch.bfloat16, device=big.device)
        spare = mezo.NF4Tensor.empty(n, big.device)
        moved = (n + 1) // 2 + 4 * ((n + 63) // 64) + 2 * n
        ops["nf4_dequantize_to_bf16"] = entry(0, timed(lambda: mezo.nf4_dequantize(big, out=vals, stream=stream)),
                                              moved)
        ops["nf4_quantize_from_bf16"] = entry(0, timed(lambda: mezo.nf4_quantize(vals, out=spare, stream=stream)),
                                              moved)
        del vals, spare
    if w.dtype != synth.NF4:
        # the sweep's memory ceiling on the same buffer: the same tile shape and
        # accesses with no RNG work (every bit kept)
        one, moved = rmw_pass(flat, stream)
        ops["stream_rmw_no_rng"] = entry(0, timed(one), moved)
    ck = torch.empty(1, dtype=torch.int64, device="cuda")
    ops["checksum"] = entry(0, timed(lambda: ps.checksum_into(ck)), bytes_per_launch / 2)
    if w.T == 0:
        # Algorithm 1's restore of the backup fused into the apply loop
        backup, keep = make_backup()
        ops["update_from_backup"] = entry(K, timed(lambda: ps.update_multi_from(backup, seeds_t[0], q0, lr)))
        backup.close()
        del keep
    return ops


def rmw_pass(flat, stream, groups: int = 1, lanes: int = 256):
    """A callable enqueuing one pass of libisa_probe.so's stream_rmw over the
    parameter buffer on stream: read and written in place, an xor with 0 per
    word (every bit kept), the engine's tile shape by default and non-temporal
    16-byte accesses; and the bytes it moves."""
    import ctypes
    from paper_2306_10015_amd import build as b
    L = ctypes.CDLL(str(b.PROBE_LIB))
    L.stream_rmw.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int, ctypes.c_int,
                             ctypes.c_void_p]
    L.stream_rmw.restype = ctypes.c_int
    nbytes = (flat.numel() * flat.element_size()) // 16 * 16

    def one():
        rc = L.stream_rmw(flat.data_ptr(), nbytes, 0, groups, lanes, stream.cuda_stream)
        if rc != 0:
            raise RuntimeError(f"stream_rmw failed ({rc})")
    return one, 2 * nbytes


def rmw_probe(torch, flat, args):
    """What HBM delivers to a sweep with no RNG work: the parameter buffer
    through rmw_pass."""
    groups = args.rmw_groups or 1  # the engine's tile shape: one 16-byte group per lane
    stream = torch.cuda.current_stream()
    one, moved = rmw_pass(flat, stream, groups, args.rmw_lanes)

    def run(n):
        for _ in range(n):
            one()
    run(args.warmup)
    torch.cuda.synchronize()
    a = torch.cuda.Event(enable_timing=True)
    e = torch.cuda.Event(enable_timing=True)
    a.record(stream)
    run(args.steps)
    e.record(stream)
    torch.cuda.synchronize()
    ms = a.elapsed_time(e) / args.steps
    print(json.dumps({"probe": "rmw", "groups_per_lane": groups, "lanes": args.rmw_lanes, "bytes_per_pass": moved,
                      "ms": ms,
                      "GBps": moved / (ms / 1e3) / 1e9,
                      "hbm_frac": moved / (ms / 1e3) / 1e9 / HBM_PEAK_GBS}))


def copy_probe(torch, flat, args):
    """A plain device-to-device copy of the whole parameter buffer: what HBM
    delivers to a streaming read+write of the same size (context for the
    bandwidth figures, and the reference for the traffic counters)."""
    dst = torch.empty_like(flat)
    for _ in range(args.warmup):
        dst.copy_(flat)
    torch.cuda.synchronize()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(args.steps):
        dst.copy_(flat)
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / args.steps
    nbytes = 2 * flat.numel() * flat.element_size()
    print(json.dumps({"probe": "copy", "bytes_per_copy": nbytes, "ms": ms,
                      "GBps": nbytes / (ms / 1e3) / 1e9,
                      "hbm_frac": nbytes / (ms / 1e3) / 1e9 / HBM_PEAK_GBS}))


def cpu_baseline(w, recs, calls, log, target_s):
    """The oracle, as it stands, on a bounded element sample of the same step:
    elements 0 .. n-1 of one tensor (tensor_id 0, the workload's value
    distribution), n sized to about `target_s` of CPU time."""
    import oracle
    from paper_2306_10015_amd import synth
    n_threads = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    n_threads = min(n_threads, 16)
    oracle.set_threads(n_threads)
    seeds = synth.seeds(w.machines, w.samples_per_machine, step=0)
    q = synth.grads_int8(w.K, "uniform", seed=1)
    seeds_per_elem = sum(recs[c] for c in calls)

    def run(n):
        if w.dtype == synth.NF4:
            from oracle import nf4
            p, a = synth.nf4_theta0_tensor(n, 0, 0)
            c = nf4.unpack(p, n)
            t0 = time.perf_counter()
            if w.T == 0:
                c, a = nf4.perturb(c, a, 0, (0, 0, 0), w.eps)
                c, a = nf4.perturb(c, a, 0, (0, 0, 0), -2 * w.eps)
                c, a = nf4.perturb(c, a, 0, (0, 0, 0), w.eps)
                c, a = nf4.update(c, a, 0, seeds, q, w.lr)
            nf4.replay(c, a, 0, log)
            return time.perf_counter() - t0
        th = synth.theta0_tensor((n,), w.dtype, 0, 0)
        t0 = time.perf_counter()
        if w.T == 0:
            oracle.perturb(th, 0, (0, 0, 0), w.eps)
            oracle.perturb(th, 0, (0, 0, 0), -2 * w.eps)
            oracle.perturb(th, 0, (0, 0, 0), w.eps)
            oracle.update(th, 0, seeds, q, w.lr)
        oracle.replay(th, 0, log)
        return time.perf_counter() - t0

    def sized(seconds):
        n = 1 << 10
        dt = run(n)
        while dt < 0.5 and n < w.numel:
            n *= 4
            dt = run(n)
        n_full = int(min(max(n * seconds / max(dt, 1e-6), n), w.numel))
        return n_full, run(n_full)

    n_full, dt = sized(target_s)
    out = {"value": n_full * seeds_per_elem / dt, "unit": "param-seeds/s", "cores": n_threads,
           "kind": "oracle",
           "sample": f"elements 0..{n_full - 1} of one tensor (id 0) through the same step "
                     f"({seeds_per_elem} param-seeds per element), {dt:.1f} s"}
    # the same oracle on one thread (a shorter sample), for the per-core rate
    oracle.set_threads(1)
    n1, dt1 = sized(max(1.0, target_s / 4))
    oracle.set_threads(n_threads)
    out["value_1_thread"] = n1 * seeds_per_elem / dt1
    out["sample_1_thread"] = f"elements 0..{n1 - 1} of one tensor (id 0), {dt1:.1f} s"
    return out


if __name__ == "__main__":
    main()
