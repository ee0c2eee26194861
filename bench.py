"""Throughput of the block-scaled e4m3 Strassen-type product on one MI355X.

One step = encode + quantize both operands, the T fp8 sub-products, the
W-combine, C written once (fmm_encode, fmm_products, fmm_combine: together
fmm_matmul); fp32 A and B are resident in HBM before the timed region.
Default workload: 8192^3, one level, the Phi-optimal realization T*, e4m3
block 32 along K, power-of-two (E8M0) block scales, A and B iid N(0,1)
(synthetic, seeded).

Prints one JSON line with the effective rate 2MNK / t over exactly --steps
whole steps (after --warmup untimed ones), the relative RMS error of C against
the fp64 product (measured after the timed region), the roofline of the
dominant kernel (the sub-products, fmm_products, against the fp8 dense MFMA
peak) from HIP events on the launch stream, the step's required HBM bytes
against the HBM peak, the comparison arms timed interleaved in batches (the
paired protocol of the paper's Table E.7), the records of the run (device,
versions, sources, seeds), and the oracle timed on this host's cores on a
bounded sample.
"""
from __future__ import annotations

import argparse
import hashlib
import re
import json
import os
import subprocess
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

FP8_DENSE_PEAK_TFLOPS = 5000.0      # MI355X dense fp8 (MX) matrix peak
BF16_DENSE_PEAK_TFLOPS = 2500.0
HBM_PEAK_GBS = 8000.0

METRIC = "effective fp8 TFLOP/s (2mnk/t) at 8192³ 1-level; relative RMS error vs fp64"
SEED = 0          # operand streams SeedSequence([SEED, cfg, trial, operand])


def parse():
    p = argparse.ArgumentParser(description=__doc__)
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--size", type=int, default=8192, help="M = K = N")
    p.add_argument("--shape", type=int, nargs=3, metavar=("M", "K", "N"),
                   help="a rectangular product instead of --size (the other configurations)")
    p.add_argument("--batch", type=int, default=1, help="independent products per step")
    p.add_argument("--depth", type=int, default=1)
    p.add_argument("--block", type=int, default=32)
    p.add_argument("--rule", default="pow2_ceil")
    p.add_argument("--realization", default="tstar",
                   help="cubic8, strassen, winograd, tstar, or a realization of another shape (at depth 1): "
                        "one of fmm_inputs.shapes.CATALOG or cubic_<m><k><n>")
    p.add_argument("--family", default="gaussian")
    p.add_argument("--exact-dot", action="store_true")
    p.add_argument("--large-tile", action="store_true",
                   help="FMM_FLAG_LARGE_TILE: the 256 x 128 sub-product tiles wherever the shape allows")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-arms", action="store_true",
                   help="skip the comparison arms (cubic and Strassen realizations, heavy-tailed "
                        "operands, the deployment granularity, realizations of other shapes)")
    p.add_argument("--arm-batches", type=int, default=4,
                   help="interleaved rounds over the arms (each arm times --arm-steps steps a round)")
    p.add_argument("--arm-steps", type=int, default=5)
    p.add_argument("--calibrate-copy", action="store_true",
                   help="only run a plain 1 GiB device-to-device copy five times (the known-size "
                        "kernel that scales the FETCH_SIZE / WRITE_SIZE counters to bytes)")
    return p.parse_args()


def calibrate_copy():
    import torch
    n = 1 << 28                                   # 2^28 floats = 1 GiB
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": 4 * n, "copy_bytes_written": 4 * n, "launches": 5}))


def source_hash(names=None):
    """sha256 over the library's HIP/C++ sources and its header (the kernels
    a measurement or a counter summary belongs to)."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2609_26077_amd", "csrc")
    if names is None:
        names = sorted(n for n in os.listdir(csrc) if n.endswith((".hip", ".h", ".cpp")))
    for name in names:
        with open(os.path.join(csrc, name), "rb") as fh:
            h.update(fh.read())
    with open(os.path.join(ROOT, "include", "fmm8.h"), "rb") as fh:
        h.update(fh.read())
    return h.hexdigest()


def kernel_source_hash():
    """sha256 over the device code a counter summary measures: the HIP
    sources and headers under csrc/, and the public header with its comments
    removed (host-side sources and comment edits leave the kernels as they
    are; a plan change that runs other kernels shows as other kernel names)."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2609_26077_amd", "csrc")
    for name in sorted(n for n in os.listdir(csrc) if n.endswith((".hip", ".h"))):
        with open(os.path.join(csrc, name), "rb") as fh:
            h.update(fh.read())
    with open(os.path.join(ROOT, "include", "fmm8.h")) as fh:
        text = re.sub(r"/\*.*?\*/", "", fh.read(), flags=re.S)
    h.update(re.sub(r"\s+", " ", text).encode())
    return h.hexdigest()


def recorded_counters(workload_key):
    """Per-launch HBM bytes (FETCH_SIZE, WRITE_SIZE scaled to bytes) of each
    kernel of the step from the committed counter summary of this workload,
    if it was taken on the device code as it is now; otherwise None."""
    path = os.path.join(ROOT, "profiles", f"step_counters_{workload_key}.md")
    if not os.path.exists(path):
        return None
    fields, rows = {}, {}
    with open(path) as fh:
        for l in fh:
            if l.startswith("- ") and ": " in l:
                k, v = l[2:].split(": ", 1)
                fields[k.strip()] = v.strip().strip("`")
            elif l.startswith("| `") and l.count("|") >= 6:
                c = [x.strip() for x in l.strip().strip("|").split("|")]
                try:
                    rows[c[0].strip("`")] = {"role": c[1], "read": float(c[2]) * 1e6, "written": float(c[3]) * 1e6}
                except ValueError:
                    pass
    if fields.get("kernel source sha256") != kernel_source_hash() or not rows:
        return None
    return rows


def run_meta(dev):
    import torch
    props = torch.cuda.get_device_properties(dev)
    rocm = None
    for p in ("/opt/rocm/.info/version", "/opt/rocm/.info/version-dev"):
        try:
            rocm = open(p).read().strip()
            break
        except OSError:
            pass
    commit = None
    try:
        commit = subprocess.run(["git", "-C", ROOT, "rev-parse", "HEAD"], capture_output=True, text=True,
                                timeout=10).stdout.strip() or None
    except Exception:
        pass
    return {"device": torch.cuda.get_device_name(dev), "gcnArchName": getattr(props, "gcnArchName", None),
            "compute_units": props.multi_processor_count, "rocm": rocm, "torch": torch.__version__,
            "torch_hip": torch.version.hip, "numpy": np.__version__, "python": sys.version.split()[0],
            "git_commit": commit, "source_sha256": source_hash(),
            "seeds": {"operands": f"numpy PCG64(SeedSequence([{SEED}, cfg, trial, operand])), "
                                  "cfg 0 (headline), trial 0; operand 0 = A, 1 = B"}}


def time_steps(f, dA, dB, C, stream, steps):
    """Per-step event times (ms) of encode, sub-products, combine and the
    whole step on the launch stream, for `steps` consecutive steps."""
    import torch
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
    for s in range(steps):
        ev[s][0].record(stream)
        f.encode(dA, dB, stream)
        ev[s][1].record(stream)
        f.products(C, stream)
        ev[s][2].record(stream)
        f.combine(C, stream)
        ev[s][3].record(stream)
    torch.cuda.synchronize()
    t = np.array([[e[0].elapsed_time(e[1]), e[1].elapsed_time(e[2]), e[2].elapsed_time(e[3]),
                   e[0].elapsed_time(e[3])] for e in ev])
    return {"encode": t[:, 0], "products": t[:, 1], "combine": t[:, 2], "step": t[:, 3]}


WARM_MS = 150.0   # the least GPU time the warm-up spans, whatever --warmup asks


def warm_up(f, dA, dB, C, stream, min_steps, min_ms=WARM_MS):
    """Untimed steps: at least `min_steps`, and at least `min_ms` of GPU time.
    A burst of work after idle first runs at boost clocks, then dips while
    the power management clamps them (measured: sub-products 0.43 ms for two
    steps, 0.52-0.59 ms around steps 4-10, settling near 0.40 ms after about
    40 steps, i.e. 30 ms); timing must start in the settled state that
    sustained use runs in.  Returns the number of steps run."""
    import torch
    n = 0
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    while True:
        for _ in range(max(1, min_steps - n) if n < min_steps else 10):
            f.matmul(dA, dB, C, stream)
            n += 1
        t1.record(stream)
        t1.synchronize()
        if n >= min_steps and t0.elapsed_time(t1) >= min_ms:
            return n


def interleaved_arms(args, dA, dB, stream):
    """The comparison arms on the same code path and workload size, timed
    interleaved: --arm-batches rounds, each arm --arm-steps steps per round
    (the paired, interleaved protocol of Table E.7), after at least 3
    warm-up steps each.  Arms: the headline itself; cubic (8 products) and Strassen 1969 on
    the same Gaussian operands; the default realization on heavy-tailed
    operands (Student-t, 3 degrees of freedom, unit variance) on the fp8 path
    and on the exact-dot path; the real kernel's quantization (block 128,
    128 x 128 weight blocks with the bfloat16 pre-round) with fp32 amax/448
    scales (exact-dot sub-products) and with E8M0 scales.  Each: effective
    TFLOP/s from the mean event time of its steps, the sub-products' mean, and
    the relative RMS error against fp64."""
    import torch
    import fmm_inputs as gen
    from paper_2609_26077_amd.runner import FMM, error_stats, reference_f64
    n = args.size
    mkn = 2.0 * n ** 3
    t3 = None
    arms = [(args.realization, args.family, args.rule, args.block, 0, False, "headline"),
            ("cubic8", "gaussian", args.rule, args.block, 0, False, "cubic8/gaussian"),
            ("strassen", "gaussian", args.rule, args.block, 0, False, "strassen/gaussian"),
            (args.realization, "student_t3", args.rule, args.block, 0, False,
             f"{args.realization}/student_t3/fp8"),
            (args.realization, "student_t3", args.rule, args.block, 0, True,
             f"{args.realization}/student_t3/exact-dot"),
            (args.realization, "gaussian", "fp32_amax", 128, 2 | 4, False,
             f"{args.realization}/gaussian/deployment-fp32amax-b128x128-bf16"),
            (args.realization, "gaussian", "pow2_ceil", 128, 2 | 4, False,
             f"{args.realization}/gaussian/deployment-e8m0-b128x128-bf16")]
    if args.depth != 1:
        arms = [a for a in arms if not a[4]]
    state = []
    for real, family, rule, block, flags, exact, label in arms:
        if family == args.family:
            xa, xb = dA, dB
        else:
            if t3 is None:
                A, B = gen.operands(family, 1, n, n, n, seed=SEED, cfg=0, trial=0)
                t3 = (torch.from_numpy(A).to(dA.device), torch.from_numpy(B).to(dA.device))
                del A, B
            xa, xb = t3
        f = FMM(real, 1, n, n, n, args.depth, block, rule, exact_dot=exact or args.exact_dot, flags=flags)
        C = torch.empty((1, n, n), dtype=torch.float32, device=dA.device)
        warm_up(f, xa, xb, C, stream, 3, 20.0)
        state.append({"label": label, "f": f, "a": xa, "b": xb, "C": C, "t": []})
    for _ in range(args.arm_batches):
        for s in state:
            s["t"].append(time_steps(s["f"], s["a"], s["b"], s["C"], stream, args.arm_steps))
    out = {}
    for s in state:
        step = np.concatenate([t["step"] for t in s["t"]])
        prod = np.concatenate([t["products"] for t in s["t"]])
        Cref = reference_f64(s["a"], s["b"])
        err2, ref2 = error_stats(s["C"], Cref)
        del Cref
        out[s["label"]] = {"value": mkn / (step.mean() * 1e-3) / 1e12, "unit": "TFLOP/s",
                           "ms_per_step": float(step.mean()), "median_ms": float(np.median(step)),
                           "products_ms": float(prod.mean()),
                           "rel_rms_error_vs_fp64": float(np.sqrt(err2.sum() / ref2.sum())),
                           "steps": int(step.size)}
        s.clear()
        torch.cuda.empty_cache()
    return {"protocol": f"{args.arm_batches} interleaved rounds x {args.arm_steps} steps per arm, "
                        "3 warm-up steps each, same seeded operands across arms", "arms": out}


def shape_arms(args, stream):
    """Realizations of other shapes <m,k,n;R> on the same path, each on
    sub-blocks of the headline's (size / 2 on a side), Gaussian operands, the
    headline's block and rule: <2,2,3;11> (Strassen and T* each beside a
    cubic <2,2,1> part) and the cubic <2,2,3;12> on M = K = size,
    N = 1.5 size; <3,3,3;26> (Strassen on the 2 x 2 x 2 corner) and the cubic
    <3,3,3;27> on 1.5 size cubed.  Timed interleaved as interleaved_arms;
    effective TFLOP/s = 2 M K N / step time."""
    import torch
    import fmm_inputs as gen
    from paper_2609_26077_amd.controls import shaped_realization
    from paper_2609_26077_amd.runner import FMM, error_stats, reference_f64
    h = args.size // 2
    groups = [((2 * h, 2 * h, 3 * h), ["223_11", "223_tstar", "cubic_223"]),
              ((3 * h, 3 * h, 3 * h), ["333_26", "cubic_333"])]
    out = {}
    for (M, K, N), names in groups:
        A, B = gen.operands("gaussian", 1, M, K, N, seed=SEED, cfg=3, trial=0)
        dA, dB = torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda()
        del A, B
        state = []
        for name in names:
            f = FMM(shaped_realization(name), 1, M, K, N, 1, args.block, args.rule, exact_dot=args.exact_dot)
            C = torch.empty((1, M, N), dtype=torch.float32, device=dA.device)
            warm_up(f, dA, dB, C, stream, 3, 20.0)
            state.append({"name": name, "f": f, "C": C, "t": []})
        for _ in range(args.arm_batches):
            for s in state:
                s["t"].append(time_steps(s["f"], dA, dB, s["C"], stream, args.arm_steps))
        Cref = reference_f64(dA, dB)
        for s in state:
            step = np.concatenate([t["step"] for t in s["t"]])
            prod = np.concatenate([t["products"] for t in s["t"]])
            enc = np.concatenate([t["encode"] for t in s["t"]])
            comb = np.concatenate([t["combine"] for t in s["t"]])
            err2, ref2 = error_stats(s["C"], Cref)
            from paper_2609_26077_amd import fmm_realization_metrics, fmm_realization_shape
            shape, rank = fmm_realization_shape(s["f"].real)
            out[s["name"]] = {"shape": list(shape), "rank": rank, "M": M, "K": K, "N": N,
                              "phi": fmm_realization_metrics(s["f"].real, 1)["phi"],
                              "value": 2.0 * M * K * N / (step.mean() * 1e-3) / 1e12, "unit": "TFLOP/s",
                              "ms_per_step": float(step.mean()), "encode_ms": float(enc.mean()),
                              "products_ms": float(prod.mean()), "combine_ms": float(comb.mean()),
                              "rel_rms_error_vs_fp64": float(np.sqrt(err2.sum() / ref2.sum())),
                              "steps": int(step.size)}
            s.clear()
        del Cref, dA, dB, state
        torch.cuda.empty_cache()
    return {"protocol": f"{args.arm_batches} interleaved rounds x {args.arm_steps} steps per arm within each "
                        "shape, 3 warm-up steps each, same seeded operands within a shape", "arms": out}


def paper_context():
    """The paper's own error figures under their stated setup, next to this
    path measured under the same setup (context, not a target): Table E.1's
    <2,2,2> row, an fp32 emulation of fused block-128 e4m3 with fp32
    amax/448 scales, one signed-uniform operand family, eight paired samples
    at block edge 256 (512^3 products), mean relative Frobenius error; the
    re-based realization there is the Phi-minimizing one (T* here)."""
    import torch
    import fmm_inputs as gen
    from paper_2609_26077_amd.runner import FMM, error_stats, reference_f64
    n, trials = 512, 8
    A, B = gen.operands("uniform", trials, n, n, n, seed=SEED, cfg=11, trial=0)
    dA, dB = torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda()
    Cref = reference_f64(dA, dB)
    e = {}
    for real in ("cubic8", "tstar"):
        f = FMM(real, trials, n, n, n, 1, 128, "fp32_amax")
        C = f.matmul(dA, dB)
        err2, ref2 = error_stats(C, Cref)
        e[real] = float(np.mean(np.sqrt(err2 / ref2)))
    return {"source": "Table E.1, <2,2,2> row (fp32 emulator of fused blk128 e4m3, fp32 amax/448 scales, "
                      "signed-uniform operands, 8 paired samples at block edge 256)",
            "paper": {"e_cubic": 0.0874 / 2.4486, "e_rebased_over_e_cubic": 1.7190},
            "measured": {"e_cubic": e["cubic8"], "e_tstar_over_e_cubic": e["tstar"] / e["cubic8"],
                         "trials": trials, "size": f"{n}x{n}x{n}"},
            "note": "context only: the paper's figures come from its own emulator on other hardware"}


def cpu_baseline(args):
    """The oracle, unchanged, timed on this host's cores on a bounded sample
    of the benchmark configurations: the 100 trials of the 256^3
    configuration for the cubic and Strassen 1969 realizations, one trial of
    the 4096^3 configuration (T*) and one trial of the headline workload.
    BLAS threads are held to the cores this process may run on."""
    from threadpoolctl import threadpool_limits
    from oracle import e4m3, fmm
    from oracle import realizations as R
    import fmm_inputs as gen
    cores = len(os.sched_getaffinity(0))
    rule = e4m3.RULES[args.rule]
    flop, t = 0.0, 0.0
    parts = []
    with threadpool_limits(limits=cores):
        A, B = gen.operands("gaussian", 100, 256, 256, 256, seed=SEED, cfg=1, trial=0)
        for name in ("cubic8", "strassen"):
            tabs = R.tables_f32(R.builtin_f64(name), 1)
            t0 = time.perf_counter()
            for b in range(100):
                fmm.fmm(A[b], B[b], tabs, 1, 32, rule, keep=False)
            dt = time.perf_counter() - t0
            t += dt
            flop += 100 * 2.0 * 256 ** 3
            parts.append(f"100 x 256^3 {name} {dt:.2f} s")
        del A, B
        A, B = gen.operands("gaussian", 1, 4096, 4096, 4096, seed=SEED, cfg=2, trial=0)
        tabs = R.tables_f32(R.builtin_f64("tstar"), 1)
        t0 = time.perf_counter()
        fmm.fmm(A[0], B[0], tabs, 1, 32, rule, keep=False)
        dt = time.perf_counter() - t0
        t += dt
        flop += 2.0 * 4096 ** 3
        parts.append(f"1 x 4096^3 tstar {dt:.2f} s")
        del A, B
        n = args.size
        A, B = gen.operands(args.family, 1, n, n, n, seed=SEED, cfg=0, trial=0)
        tabs = R.tables_f32(R.builtin_f64(args.realization), args.depth)
        t0 = time.perf_counter()
        fmm.fmm(A[0], B[0], tabs, args.depth, args.block, rule, keep=False)
        dt = time.perf_counter() - t0
        t += dt
        flop += 2.0 * n ** 3
        parts.append(f"1 x {n}^3 {args.realization} depth {args.depth} {dt:.2f} s")
    cpu = ""
    try:
        with open("/proc/cpuinfo") as f:
            cpu = next((l.split(":", 1)[1].strip() for l in f if l.startswith("model name")), "")
    except OSError:
        pass
    return {"value": flop / t / 1e12, "unit": "TFLOP/s", "cores": cores, "kind": "oracle",
            "sample": "the 100 trials of the 256^3 configuration (N(0,1), block 32, cubic8 and Strassen "
                      f"1969), one trial of the 4096^3 configuration (T*) and one trial of the headline "
                      f"workload ({args.rule}, block {args.block}): "
                      "numpy fp32 encode + e4m3 codec, fp64 BLAS sub-products, W-combine; "
                      + "; ".join(parts),
            "seconds": t, "cpu_model": cpu}


def main():
    args = parse()
    if args.calibrate_copy:
        calibrate_copy()
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the path has no cross-GPU step, and the benchmark times "
              f"a single MI355X (--gpus {args.gpus} is not supported)", file=sys.stderr)
        sys.exit(2)

    import torch
    import fmm_inputs as gen
    from paper_2609_26077_amd import (FMM_LAYOUT_TILE256x64, fmm_operand_views, fmm_realization_metrics,
                                      fmm_realization_terms)
    from paper_2609_26077_amd.runner import FMM, error_stats, reference_f64

    dev = torch.device("cuda:0")
    n = args.size
    M, K, N = args.shape if args.shape else (n, n, n)
    nb = args.batch
    # the comparison arms, the paper context and the oracle baseline go with
    # the headline shape (one cubic product)
    headline = args.shape is None and nb == 1 and args.realization in ("cubic8", "strassen", "winograd", "tstar")
    A, B = gen.operands(args.family, nb, M, K, N, seed=SEED, cfg=0, trial=0)
    dA = torch.from_numpy(A).to(dev)
    dB = torch.from_numpy(B).to(dev)
    del A, B
    from paper_2609_26077_amd import FMM_FLAG_LARGE_TILE
    real = args.realization
    if real not in ("cubic8", "strassen", "winograd", "tstar"):
        # a realization of another shape: fmm_inputs.shapes' catalog or cubic_<m><k><n>
        from paper_2609_26077_amd.controls import shaped_realization
        real = shaped_realization(args.realization)
    f = FMM(real, nb, M, K, N, args.depth, args.block, args.rule, exact_dot=args.exact_dot,
            flags=FMM_FLAG_LARGE_TILE if args.large_tile else 0)
    C = torch.empty((nb, M, N), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream(dev)

    warm_steps = warm_up(f, dA, dB, C, stream, args.warmup)
    torch.cuda.synchronize(dev)

    # timed region: exactly --steps whole steps, bracketed by synchronizations;
    # events around each launch on the launch stream
    t0 = time.perf_counter()
    ev = time_steps(f, dA, dB, C, stream, args.steps)      # ends with a synchronize
    wall = time.perf_counter() - t0
    ms_per_step = wall * 1e3 / args.steps
    enc_ms, prod_ms, comb_ms = (float(ev[k].mean()) for k in ("encode", "products", "combine"))

    # error of the last step's C against the fp64 product (not timed)
    Cref = reference_f64(dA, dB)
    err2, ref2 = error_stats(C, Cref)
    rel_mse = float(err2.sum() / ref2.sum())
    del Cref

    R_, T = fmm_realization_terms(f.real, args.depth)
    phi = fmm_realization_metrics(f.real, args.depth)["phi"]
    a_view, _ = fmm_operand_views(f.plan, f.ws)
    split = a_view.code_layout == FMM_LAYOUT_TILE256x64
    mkn = 2.0 * nb * M * N * K
    from paper_2609_26077_amd import fmm_realization_shape
    (gm, gk, gn), _ = fmm_realization_shape(f.real)
    if (gm, gk, gn) == (2, 2, 2):
        gm = gk = gn = 2 ** args.depth
    mp, kp, np_ = M // gm, K // gk, N // gn
    mfma_flop = 2.0 * nb * T * mp * kp * np_
    sb = 4 if args.rule == "fp32_amax" else 1
    code_bytes = nb * T * (mp + np_) * kp
    scale_bytes = nb * T * (mp + np_) * (kp // args.block) * sb
    ab_bytes = 4 * nb * (M * K + K * N)
    c_bytes = 4 * nb * M * N
    pr_bytes = nb * T * mp * np_ * 4 if split else 0          # P_r written and read back (not required)
    enc_bytes = ab_bytes + code_bytes + scale_bytes
    gemm_required = code_bytes + scale_bytes + c_bytes        # codes and scales read once, C written once
    step_required = enc_bytes + gemm_required
    exact = args.exact_dot or args.rule == "fp32_amax" or args.block == 16
    peak = BF16_DENSE_PEAK_TFLOPS if exact else FP8_DENSE_PEAK_TFLOPS
    achieved = mfma_flop / (prod_ms * 1e-3) / 1e12
    wkey = None
    if headline and not args.exact_dot:
        wkey = f"{M}cube_depth{args.depth}_{args.realization}_b{args.block}_{args.rule}_{args.family}"
    counters = recorded_counters(wkey) if wkey else None
    # the sub-product kernel the plan runs (layout and scale rule decide it)
    if split:
        prod_kernel = ("gemm_exact256x128_kernel" if sb == 4 else
                       "gemm_dq256x128_kernel" if exact else "gemm_tile256x256_kernel")
    elif a_view.code_layout == 2:
        prod_kernel = "gemm_dq8_kernel" if exact else "gemm_mx_fast_kernel"
    else:
        prod_kernel = "gemm_promote_kernel" if exact else "gemm_mx_kernel"
    traffic = None
    step_traffic = None
    if counters:
        for name, c in counters.items():
            if c["role"] == "sub-products":
                traffic = c["read"] + c["written"]
        step_traffic = sum(c["read"] + c["written"] for c in counters.values())

    def hbm(nbytes, ms, note=None):
        gbs = nbytes / (ms * 1e-3) / 1e9 if ms > 0 else 0.0
        d = {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
             "frac": gbs / HBM_PEAK_GBS, "algorithmic_bytes_per_launch": nbytes}
        if note:
            d["note"] = note
        return d

    line = {
        "metric": METRIC,
        "value": mkn / (ms_per_step * 1e-3) / 1e12,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "warmup_steps_run": warm_steps,
        "warmup_note": f"at least --warmup steps and at least {WARM_MS:.0f} ms of GPU time: the clocks dip "
                       "for tens of ms after a burst of work starts, then settle",
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp8",
        "data": "synthetic",
        "config": {"workload": (f"batch {nb} x " if nb > 1 else "") + f"{M}x{K}x{N} product, depth {args.depth}, "
                               f"realization {args.realization} (Phi={phi:.4f}), e4m3 block {args.block} along "
                               f"K, {args.rule} scales, {args.family} operands"
                               + (", exact-dot sub-products" if args.exact_dot else ""),
                   "M": M, "K": K, "N": N, "depth": args.depth, "terms": T, "block": args.block,
                   "rule": args.rule, "realization": args.realization, "family": args.family,
                   "realization_shape": list(fmm_realization_shape(f.real)[0]),
                   "exact_dot": bool(args.exact_dot),
                   "subproduct_path": ("large tiles (" + ("256x128" if exact else "256x256") +
                                       ") + separate W-combine") if split
                   else "128x128 tiles with the W-combine fused"},
        "rel_rms_error_vs_fp64": float(np.sqrt(rel_mse)),
        "rel_mse_vs_fp64": rel_mse,
        "kernels_ms": {"encode": enc_ms, "products": prod_ms, "combine": comb_ms},
        "step_event_ms": {"median": float(np.median(ev["step"])), "min": float(ev["step"].min()),
                          "mean": float(ev["step"].mean())},
        "roofline": {"bound": "mfma", "kernel": f"{prod_kernel} (fmm_products: the T sub-products)",
                     "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                     "frac": achieved / peak, "traffic": traffic,
                     "algorithmic_flop_per_launch": mfma_flop,
                     "algorithmic_bytes_per_launch": gemm_required,
                     "algorithmic_bytes_note": "codes and scales read once + C written once; on the large-tile "
                                               "path C is written by the combine launch and this launch writes "
                                               f"the fp32 P_r instead ({pr_bytes} bytes, not required)",
                     "traffic_over_algorithmic": traffic / gemm_required if traffic else None},
        "encode_roofline": hbm(enc_bytes, enc_ms),
        "step_hbm": {"required_bytes": step_required, "achieved": step_required / (ms_per_step * 1e-3) / 1e9,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": step_required / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS,
                     "pr_round_trip_bytes": 2 * pr_bytes,
                     "traffic": step_traffic,
                     "traffic_over_required": step_traffic / step_required if step_traffic else None,
                     "note": "required = A, B read + codes and scales written + read once + C written once"},
        "meta": run_meta(dev),
    }
    if split:
        line["combine_roofline"] = hbm(pr_bytes + c_bytes, comb_ms,
                                       "the P_r read back is not required work: the pass exists because the "
                                       "W-combine is not fused on the large-tile path")
    if nb > 1:
        line["config"]["batch"] = nb
    if not args.no_arms and headline:
        line["arms"] = interleaved_arms(args, dA, dB, stream)
        if args.depth == 1:
            line["shape_arms"] = shape_arms(args, stream)
        line["paper_context"] = paper_context()
    if not args.no_cpu_baseline and headline:
        del dA, dB, C
        torch.cuda.empty_cache()
        line["cpu_baseline"] = cpu_baseline(args)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
