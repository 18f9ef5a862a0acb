"""Throughput of the seeded perturbation engine on one MI355X.

One step is one pass of the whole hot path over a synthetic OPT-6.7B-shaped
parameter set in bf16 storage (6,648,897,536 elements in 323 tensors,
N(0, 0.02); fp32 arithmetic):

  1. PerturbParameters +eps, -2eps, +eps with this machine's seed
     (Algorithm 1, inner inference loop; eps = 1e-3);
  2. quantize_projgrad of the K = 64 projected gradients of the iteration
     (Section 3, one byte each; linear code, scale 1/127);
  3. update_multi: the fused apply loop over the K = 64 (machine, sample)
     seeds (Algorithm 1; lr = 1e-6);
  4. replay: a late joiner's catch-up over a log of T = 4 earlier iterations
     of K = 64 seeds each (Appendix B).

Every parameter is read and written once per call; z is regenerated in
registers. The metric is param-seed updates per second: elements x seeds
applied, summed over the step's calls, divided by the time of the step.

Prints ONE JSON line with the engine kernel's ALU roofline (the step is
RNG-bound: its ceiling is the VALU issue rate of the instructions that make z,
below), each call timed alone (`ops`), the memory-bound perturb sweep of the
OPT-125m-shaped fp32 set (`secondary`) and the CPU oracle timed on a bounded
sample of the same step (`cpu_baseline`).

    python bench.py [--gpus 1] [--steps 20] [--warmup 3] [--workload NAME]
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

#: VALU issue ceiling of one MI355X for the engine's instruction stream:
#: every non-transcendental VALU instruction of a wave64 occupies its 16-lane
#: SIMD for 4 cycles, so 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz = 39.3e12
#: lane-instructions per second; transcendentals (log, sqrt, sin, cos) issue
#: on a unit of their own beside them (their 2 per param-seed take 2 x 8
#: cycles per wave on it, less than the 13.5 x 4 of the rest), so they add no
#: time at the ceiling. The counters agree: the dual-issue share of the
#: engine's VALU cycles (14-15%) is its transcendental share (8 of 62).
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
TRANSCENDENTAL = ("v_log_f32", "v_sqrt_f32", "v_sin_f32", "v_cos_f32")
#: lane-instructions per param-seed (= 62 / 4), and the non-transcendental
#: ones that bound the issue rate (= 54 / 4)
INSTR_PER_PARAM_SEED = sum(INNER_LOOP_MIX.values()) / 4.0
NONTRANS_PER_PARAM_SEED = sum(v for k, v in INNER_LOOP_MIX.items() if k not in TRANSCENDENTAL) / 4.0
#: the ceiling in param-seeds per second
PARAM_SEED_PEAK = VALU_LANE_INSTR_PER_S / NONTRANS_PER_PARAM_SEED

#: counter profile of the engine kernel on a workload (traffic per dispatch,
#: VALU counters), quoted only while the kernel's sources are the ones it was
#: taken on
PROFILE = os.path.join(ROOT, "profiles", "engine_kernel_{workload}.json")
ENGINE_UNIT = {"f32": "engine_dense.hip", "bf16": "engine_dense.hip", "nf4": "engine_nf4.hip"}

T_REPLAY = 4
SECONDARY_WORKLOAD = "opt125m"


def parse():
    p = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--workload", default="opt6.7b")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-ops", action="store_true",
                   help="skip the per-operation and secondary measurements after the timed region "
                        "(profiling runs)")
    p.add_argument("--gaussian", choices=["fast", "portable"], default="fast",
                   help="how z is computed (portable: binary32 operations only, bit-identical "
                        "on any IEEE device)")
    p.add_argument("--probe", choices=["copy", "rmw", "checksum", "nf4-dequantize", "nf4-quantize"],
                   default=None,
                   help="copy: time a plain device copy of the parameter buffer instead; rmw: an in-place "
                        "streaming read-modify-write of it with the engine's access pattern (the sweep's "
                        "memory ceiling); checksum: the set's checksum alone; nf4-dequantize / "
                        "nf4-quantize: an NF4 set's largest tensor converted to bf16 and back")
    p.add_argument("--conv-dtype", choices=["bf16", "f32"], default="bf16",
                   help="nf4-dequantize / nf4-quantize probes: the dense side's type")
    p.add_argument("--rmw-groups", type=int, choices=[1, 2], default=None,
                   help="rmw probe: 16-byte groups per lane (default 1, the engine's)")
    p.add_argument("--rmw-lanes", type=int, choices=[128, 256, 512], default=256,
                   help="rmw probe: lanes per workgroup (default 256, the engine's)")
    return p.parse_args()


def flat_views(torch, w, device):
    """One 256-byte-aligned allocation holding every tensor of the set."""
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


def fill_dense(torch, synth, w, views, dev):
    """theta0 ~ N(0, 0.02) of a dense set, resident in HBM."""
    if w.numel <= 200_000_000:
        # numpy PCG64 per tensor (the same theta0 the tests and the oracle use)
        for i, (v, (_, shape)) in enumerate(zip(views, w.shapes)):
            h = synth.theta0_tensor(shape, w.dtype, i, 0)
            if w.dtype == "f32":
                v.copy_(torch.from_numpy(h))
            else:
                v.copy_(torch.from_numpy(h.view(np.int16)).view(torch.bfloat16))
    else:
        # billions of elements: the same law drawn in HBM by torch's seeded generator
        g = torch.Generator(device=dev)
        g.manual_seed(0)
        for v in views:
            tmp = torch.empty(v.numel(), dtype=torch.float32, device=dev)
            tmp.normal_(0.0, 0.02, generator=g)
            v.copy_(tmp)
            del tmp


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the engine's path is the kernel on one GPU's share of the "
              f"parameters, with no collectives (--gpus {args.gpus} requested). Run with --gpus 1.",
              file=sys.stderr)
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
        fill_dense(torch, synth, w, views, dev)

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
    if args.probe is not None:
        kernel_probe(torch, mezo, synth, w, ps, args)
        return
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
    # HIP events on the stream every kernel of the step is enqueued on
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
    # the stream but the record lists' 8 KiB copies); achieved = param-seeds x
    # the non-transcendental lane-instructions per param-seed over that time.
    n_launch = len(calls)
    avg_launch_s = ms_per_step / n_launch / 1e3
    ps_per_launch = ps_per_step / n_launch
    achieved = ps_per_launch * NONTRANS_PER_PARAM_SEED / avg_launch_s / 1e12
    peak = VALU_LANE_INSTR_PER_S / 1e12
    # the step's launches bind differently (a sweep can be memory-bound, the
    # updates are VALU-bound): its ideal time puts every launch at its own
    # roofline, the larger of bytes / HBM peak and param-seeds / ALU peak
    ideal_ms = 1e3 * sum(max(bytes_per_launch / (HBM_PEAK_GBS * 1e9), N * recs[c] / PARAM_SEED_PEAK)
                         for c in calls)
    prof = engine_profile(w, args.gaussian)
    roofline = {"bound": "alu", "achieved": achieved, "peak": peak,
                "unit": "Tinstr/s", "frac": achieved / peak,
                "traffic": prof["hbm_bytes_per_dispatch"] if prof and "hbm_bytes_per_dispatch" in prof else None,
                "alg_bytes_per_launch": bytes_per_launch,
                "kernel": f"engine_kernel<{w.dtype}> ("
                          + ", ".join(f"{recs[c]} record{'s' if recs[c] > 1 else ''}" for c in calls)
                          + " per launch)",
                "peak_basis": "non-transcendental VALU issue: 256 CU x 4 SIMD x 16 lanes x 2.4 GHz; "
                              "transcendentals co-issue on their own unit",
                "instr_per_param_seed": NONTRANS_PER_PARAM_SEED,
                "instr_per_param_seed_with_transcendentals": INSTR_PER_PARAM_SEED,
                "param_seed_peak": PARAM_SEED_PEAK,
                "param_seeds_per_launch": ps_per_launch,
                "avg_launch_ms": avg_launch_s * 1e3,
                "step_ideal_ms": ideal_ms,
                "combined_frac": ideal_ms / ms_per_step}
    if prof and "valu_by_records" in prof:
        # counters of the same kernel sources: the largest record count is the
        # update or replay, where z is nearly all the work
        vr = prof["valu_by_records"]
        kmax = max(vr, key=int)
        roofline["counters"] = {
            "profile": os.path.relpath(PROFILE.format(workload=w.name), ROOT),
            "records": int(kmax),
            "valu_busy_pct": vr[kmax]["busy_pct"],
            "dual_issue_pct": vr[kmax]["dual_issue_pct"],
            "main_pipe_busy_pct": vr[kmax].get("main_pipe_busy_pct"),
            "clock_ghz": vr[kmax].get("clock_ghz"),
            "valu_instr_per_param_seed": vr[kmax]["instr_per_param_seed"],
            "nontrans_instr_per_param_seed": vr[kmax]["instr_per_param_seed"] - vr[kmax]["trans_per_param_seed"],
            "by_records": {r: {"valu_busy_pct": round(v["busy_pct"], 1),
                               "valu_instr_per_param_seed": round(v["instr_per_param_seed"], 3)}
                           for r, v in vr.items()}}
    ops = secondary = None
    if not args.no_ops:
        ops = measure_ops(torch, mezo, synth, w, ps, make_backup, stream, recs, proj, seeds_t, log,
                          bytes_per_launch, flat)
        if w.name != SECONDARY_WORKLOAD and args.gaussian == "fast":
            secondary = measure_secondary(torch, mezo, synth, dev, stream)

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
        "roofline": roofline,
        "wall_s_timed": wall,
    }
    if ops is not None:
        out["ops"] = ops
        if "perturb" in ops and "stream_rmw_no_rng" in ops:
            out["roofline"]["sweep_frac_of_stream_ceiling"] = (ops["perturb"]["alg_GBps"]
                                                               / ops["stream_rmw_no_rng"]["alg_GBps"])
    if secondary is not None:
        out["secondary"] = secondary
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, recs, calls, log)
        out["gpu_over_cpu"] = value / out["cpu_baseline"]["value"]
    print(json.dumps(out))


def engine_profile(w, gaussian: str):
    """The committed counter profile of the engine kernel on this workload,
    or None when there is none or the kernel's sources changed since it was
    taken."""
    if gaussian != "fast":
        return None
    from paper_2306_10015_amd import profile_summary
    try:
        with open(PROFILE.format(workload=w.name)) as f:
            prof = json.load(f)
    except (OSError, ValueError):
        return None
    unit = ENGINE_UNIT[w.dtype]
    if prof.get("kernel_unit") != unit or prof.get("kernel_source_sha256") != profile_summary.source_hash(unit):
        return None
    return prof


def timer(torch, stream):
    """timed(fn): the average duration of one call of fn (enqueuing work on
    stream), from batches of back-to-back calls between two events on the
    stream: each batch lasts about OPS_LOOP_MS, so that short calls are timed
    over many launches at the clock a long run settles at; the median of
    OPS_BATCHES batches."""
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
        fn()
        torch.cuda.synchronize()
        once = loop(fn, 1)
        reps = max(1, min(OPS_MAX_REPS, math.ceil(OPS_LOOP_MS / max(once, 1e-3))))
        return statistics.median(loop(fn, reps) for _ in range(OPS_BATCHES))
    return timed


def measure_ops(torch, mezo, synth, w, ps, make_backup, stream, recs, proj, seeds_t, log,
                bytes_per_launch, flat):
    """Each operation alone, repeated back to back between two events on the
    kernels' stream (after the timed region, not part of the step)."""
    N, K, lr = w.numel, w.K, w.lr
    timed = timer(torch, stream)

    def entry(records, ms, nbytes=bytes_per_launch):
        t_s = ms / 1e3
        e = {"ms": round(ms, 4), "alg_GBps": nbytes / t_s / 1e9,
             "hbm_frac": nbytes / t_s / 1e9 / HBM_PEAK_GBS}
        if records:
            e.update({"records": records, "param_seeds_per_s": N * records / t_s,
                      "alu_frac": N * records / t_s / PARAM_SEED_PEAK})
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
        # the same iteration with the two copies Algorithm 1 holds used as a
        # pair: each sample's weights written out of place from the current
        # ones (theta+ = theta + eps z, then theta- = theta - eps z, the forward
        # passes reading the second copy), the current weights never perturbed
        # and so never restored, then the K-seed update applied to them in
        # place: one record per pass instead of the in-place sequence's
        # -2 eps and restore + next +eps
        cur, nxt = ps, backup
        samples_b = [(0, 1, j) for j in range(SAMPLES_PER_MACHINE)]

        def iteration_out_of_place():
            for s in samples_b:
                nxt.perturb_from(cur, s, w.eps)
                nxt.perturb_from(cur, s, -w.eps)
            cur.update_multi(seeds_t[0], q0, lr)
        ops["iteration_16_samples_out_of_place"] = entry(
            2 * SAMPLES_PER_MACHINE + K, timed(iteration_out_of_place),
            bytes_per_launch * (2 * SAMPLES_PER_MACHINE + 1))
        backup.close()
        del keep
    return ops


def measure_secondary(torch, mezo, synth, dev, stream):
    """The memory-bound regime in the same run: the perturb sweep (one record)
    of the OPT-125m-shaped fp32 set against 8 TB/s and against an in-place
    streaming read-modify-write of the same buffer without RNG; its checksum
    (a read-only stream)."""
    w = synth.WORKLOADS[SECONDARY_WORKLOAD]
    flat, views, _ = flat_views(torch, w, dev)
    fill_dense(torch, synth, w, views, dev)
    ps = mezo.ParamSet(views)
    timed = timer(torch, stream)
    nbytes = 2 * w.numel * storage_bytes(w)
    ms = timed(lambda: ps.perturb((0, 0, 0), w.eps))
    one, moved = rmw_pass(flat, stream)
    ms_rmw = timed(one)
    ck = torch.empty(1, dtype=torch.int64, device="cuda")
    ms_ck = timed(lambda: ps.checksum_into(ck))
    ps.close()
    gbps = nbytes / (ms / 1e3) / 1e9
    rmw_gbps = moved / (ms_rmw / 1e3) / 1e9
    ck_gbps = nbytes / 2 / (ms_ck / 1e3) / 1e9
    return {"workload": f"{w.name}: {w.numel} f32 params in {w.n_tensors} tensors",
            "perturb_sweep": {"ms": round(ms, 4), "alg_GBps": gbps, "hbm_frac": gbps / HBM_PEAK_GBS,
                              "frac_of_stream_ceiling": gbps / rmw_gbps},
            "stream_rmw_no_rng": {"ms": round(ms_rmw, 4), "alg_GBps": rmw_gbps,
                                  "hbm_frac": rmw_gbps / HBM_PEAK_GBS},
            "checksum": {"ms": round(ms_ck, 4), "alg_GBps": ck_gbps, "hbm_frac": ck_gbps / HBM_PEAK_GBS}}


def rmw_pass(flat, stream, groups: int = 1, lanes: int = 256):
    """A callable enqueuing one pass of libstream_probe.so's stream_rmw over
    the parameter buffer on stream: read and written in place, an xor with 0
    per word (every bit kept), the engine's tile shape by default and
    non-temporal 16-byte accesses; and the bytes it moves."""
    import ctypes
    from paper_2306_10015_amd import build as b
    if not b.PROBE_LIB.exists():
        raise RuntimeError(f"{b.PROBE_LIB} is not built")
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


def kernel_probe(torch, mezo, synth, w, ps, args):
    """One of the set's standalone kernels alone, `steps` launches back to back
    after `warmup` (for kernel traces and counters): the checksum of the whole
    set (a read-only stream), or the conversions of an NF4 set's largest
    tensor (the embedding) to bf16 (or fp32: --conv-dtype) and back."""
    stream = torch.cuda.current_stream()
    if args.probe == "checksum":
        ck = torch.empty(1, dtype=torch.int64, device="cuda")
        moved = w.numel * storage_bytes(w)

        def one():
            ps.checksum_into(ck, stream=stream)
    else:
        if w.dtype != synth.NF4:
            raise SystemExit(f"--probe {args.probe} needs an NF4 workload")
        big = max(ps.tensors, key=lambda t: t.numel())
        n = big.numel()
        dense = torch.float32 if args.conv_dtype == "f32" else torch.bfloat16
        vals = mezo.nf4_dequantize(big, dtype=dense, stream=stream)
        spare = mezo.NF4Tensor.empty(n, big.device)
        moved = (n + 1) // 2 + 4 * ((n + synth.NF4_BLOCK - 1) // synth.NF4_BLOCK) + vals.element_size() * n
        if args.probe == "nf4-dequantize":
            def one():
                mezo.nf4_dequantize(big, out=vals, stream=stream)
        else:
            def one():
                mezo.nf4_quantize(vals, out=spare, stream=stream)
    for _ in range(args.warmup):
        one()
    torch.cuda.synchronize()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for _ in range(args.steps):
        one()
    b.record(stream)
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / args.steps
    print(json.dumps({"probe": args.probe, "workload": w.name,
                      **({} if args.probe == "checksum" else {"dense_dtype": args.conv_dtype}),
                      "bytes_per_call": moved, "ms": ms,
                      "GBps": moved / (ms / 1e3) / 1e9,
                      "hbm_frac": moved / (ms / 1e3) / 1e9 / HBM_PEAK_GBS}))


def host_cores():
    """The host cores this process may use, and how many of them the oracle
    runs on: all of them, unless OMP_NUM_THREADS (the GPU machine's share of
    its host for one GPU, set by its environment) says fewer."""
    nproc = os.cpu_count() or 1
    affinity = sorted(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else list(range(nproc))
    threads = len(affinity)
    omp = os.environ.get("OMP_NUM_THREADS", "")
    if omp.isdigit() and int(omp) > 0:
        threads = min(threads, int(omp))
    return threads, {"nproc": nproc, "affinity": len(affinity),
                     "affinity_cpus": f"{affinity[0]}-{affinity[-1]}" if affinity else "",
                     "omp_num_threads": omp or None}


def sample_step(w, recs, calls, log, idx, tids, vals, rounds: int = 1):
    """The oracle through the bench's step on sampled elements: each tensor's
    values at its indices, in place; returns the seconds it took."""
    import oracle
    from paper_2306_10015_amd import synth
    seeds = synth.seeds(w.machines, w.samples_per_machine, step=0)
    q = synth.grads_int8(w.K, "uniform", seed=1)
    t0 = time.perf_counter()
    for _ in range(rounds):
        for tid, ix, th in zip(tids, idx, vals):
            if w.T == 0:
                oracle.perturb(th, tid, (0, 0, 0), w.eps, idx=ix)
                oracle.perturb(th, tid, (0, 0, 0), -2 * w.eps, idx=ix)
                oracle.perturb(th, tid, (0, 0, 0), w.eps, idx=ix)
                oracle.update(th, tid, seeds, q, w.lr, idx=ix)
            oracle.replay(th, tid, log, idx=ix)
    return time.perf_counter() - t0


def cpu_baseline(w, recs, calls, log):
    """The oracle, as it stands, on a bounded sample of the same step: the
    first and last `edge` elements of every tensor plus random 4-aligned
    blocks (PCG64 seed 2), with N(0, 0.02) values in the workload's storage;
    on every host core the process may use, then on one thread (a smaller
    sample)."""
    import oracle
    from paper_2306_10015_amd import synth
    if w.dtype == synth.NF4:
        raise SystemExit("the CPU baseline covers the fp32/bf16 workloads (use --no-cpu-baseline)")
    threads, cores = host_cores()
    seeds_per_elem = sum(recs[c] for c in calls)

    def make(edge, blocks):
        rng = np.random.Generator(np.random.PCG64(2))
        idx, vals = [], []
        for tid, (_, shape) in enumerate(w.shapes):
            ix = synth.sample_indices(int(np.prod(shape)), rng, edge=edge, blocks=blocks)
            x = rng.standard_normal(size=ix.size, dtype=np.float32) * np.float32(0.02)
            idx.append(ix)
            vals.append(x if w.dtype == synth.F32 else synth.bf16_bits_truncated(x))
        return idx, list(range(w.n_tensors)), vals

    # all cores: first/last 4096 elements of every tensor + 2^16 blocks over
    # the set (spread in proportion to the tensors' sizes)
    blocks = [max(1, round(65536 * int(np.prod(s)) / w.numel)) for _, s in w.shapes]
    oracle.set_threads(threads)
    rng = np.random.Generator(np.random.PCG64(2))
    idx, vals = [], []
    for tid, ((_, shape), nb) in enumerate(zip(w.shapes, blocks)):
        ix = synth.sample_indices(int(np.prod(shape)), rng, edge=4096, blocks=nb)
        x = rng.standard_normal(size=ix.size, dtype=np.float32) * np.float32(0.02)
        idx.append(ix)
        vals.append(x if w.dtype == synth.F32 else synth.bf16_bits_truncated(x))
    n_el = sum(ix.size for ix in idx)
    dt = sample_step(w, recs, calls, log, idx, list(range(w.n_tensors)), vals)
    out = {"value": n_el * seeds_per_elem / dt, "unit": "param-seeds/s", "cores": threads,
           "kind": "oracle", "host": cores,
           "sample": f"{n_el} elements: the first and last 4096 of each of the {w.n_tensors} tensors and "
                     f"{sum(blocks)} random 4-aligned blocks, through the same step ({seeds_per_elem} "
                     f"param-seeds per element), {dt:.1f} s on {threads} threads"}
    # one thread, on the first and last 256 elements of every tensor
    oracle.set_threads(1)
    idx1, tids1, vals1 = make(256, 0)
    n1 = sum(ix.size for ix in idx1)
    dt1 = sample_step(w, recs, calls, log, idx1, tids1, vals1)
    oracle.set_threads(threads)
    out["value_1_thread"] = n1 * seeds_per_elem / dt1
    out["sample_1_thread"] = f"{n1} elements (first and last 256 of every tensor), {dt1:.1f} s"
    return out


if __name__ == "__main__":
    main()
