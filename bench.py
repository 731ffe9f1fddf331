"""Benchmark of the NormPre optimizer step on one MI355X.

A step is one NormPre-G (or NormPre-L) optimizer step over a whole synthetic
layer stack (default: the 196 hidden matrices of Qwen3-1.7B, the largest
single-GPU stack of the workload list), with t incrementing so both
orientations are timed, inputs resident in HBM.

Prints ONE JSON line.  `value` is NormPre-G steps/s of the stack; NormPre-L is
reported in `variants`, and the GPT-2 Small stack (the paper's other
optimizer-latency workload) under `gpt2_small`.  The per-kernel roofline
comes from a second timed region of the same K steps in which the library
brackets every launch with HIP events on the step's stream (the clean region
gives `value`).  For NormPre-G the roofline kernel is the Newton-Schulz GEMM
class: `achieved` is the nominal Newton-Schulz work of the plain iteration,
q (4 s^2 L + 2 s^3) per matrix (s, L the short and long side), over the
class's device time, and `mfma_util_executed` is the MFMA work the launches
actually issue (tiles x tile FLOPs; symmetric products compute only upper
tiles, and the Gram-space schedule does less work than the plain iteration)
over the same time, as a fraction of peak.  The CPU baseline is the float64
oracle timed on one matrix of every shape group of the stack (both
orientations), scaled by the group sizes to whole-stack steps/s.

`roofline.traffic` is the HBM traffic per launch of the roofline kernel,
read from the committed rocprofv3 counter summary for the workload
(FETCH_SIZE and WRITE_SIZE passes, each scaled by what the counter reads for
a plain device copy of known size, `--copy-mib`); it is null when no summary
exists or when the kernel sources changed since the counters were taken.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_FP16_TFLOPS = 2516.6   # MI355X dense fp16/bf16 MFMA (256 CU x 2.4 GHz x 4096)
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E

# The paper's optimizer latency (optimizer.step() of the whole model, one
# A100 80GB; efficiency tables of Sec. 4.2 and App. E) as steps/s, keyed by
# (workload, variant): another machine's figure, reported as context.
PAPER_STEPS_PER_S = {
    ("gpt2_small", "G"): 1000.0 / 119.3, ("gpt2_small", "L"): 1000.0 / 69.8,
    ("qwen3_1p7b", "G"): 1000.0 / 1003.6, ("qwen3_1p7b", "L"): 1000.0 / 402.7,
}


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=100)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--workload", default="qwen3_1p7b")
    p.add_argument("--no-gpt2", action="store_true",
                   help="skip the GPT-2 Small stack reported next to the headline workload")
    p.add_argument("--variants", default="G,L")
    p.add_argument("--rank", type=int, default=None, help="NormPre-L rank r (default: the workload's)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=20.0,
                   help="time bound of the oracle CPU baseline sample (per variant)")
    p.add_argument("--json-out", default=None)
    p.add_argument("--crossover", action="store_true",
                   help="time NormPre-G against NormPre-L at every rank of the large single-matrix "
                        "sweep (one matrix per step) and report the cost crossover instead")
    p.add_argument("--ceiling-mib", type=int, default=256,
                   help="MiB per fp32 array of the streaming-ceiling reference kernels (0: skip)")
    p.add_argument("--copy-mib", type=int, default=0,
                   help="also run a plain device copy of this many MiB (reference kernel for "
                        "calibrating the HBM byte counters) and report its bandwidth")
    return p.parse_args()


CSRC = os.path.join(ROOT, "paper_2609_36692_amd", "csrc")
PROFILES = os.path.join(ROOT, "profiles")


# Sources that decide what a roofline-kernel launch does: the GEMM kernels
# and the host code that sizes and configures their launches.
TRAFFIC_SOURCES = ("np_gemm.hip", "np_internal.h", "normpre_api.cpp")


def kernel_source_hash():
    """SHA-256 over the GEMM kernel and launch-configuration sources."""
    h = hashlib.sha256()
    for name in TRAFFIC_SOURCES:
        h.update(name.encode())
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(workload):
    """Per-launch HBM bytes of each variant's roofline kernel from the counter
    summary `profiles/hbm_traffic_<workload>.txt` ("key: value" lines), or {}
    if it is missing or was taken on other kernel sources."""
    path = os.path.join(PROFILES, f"hbm_traffic_{workload}.txt")
    if not os.path.exists(path):
        return {}
    kv = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith(("#", " ", "|", "`")):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
    if kv.get("source_sha256") != kernel_source_hash():
        return {}
    out = {}
    for v in ("G", "L"):
        try:
            fb = float(kv[f"{v}.fetch_bytes_per_launch"])
            wb = float(kv[f"{v}.write_bytes_per_launch"])
        except (KeyError, ValueError):
            continue
        out[v] = {"bytes_per_launch": fb + wb, "fetch_bytes_per_launch": fb, "write_bytes_per_launch": wb,
                  "source": os.path.relpath(path, ROOT)}
    return out


def copy_reference(torch, mib):
    """Plain device-to-device copy of `mib` MiB: the reference kernel for the
    byte counters, and a practical HBM ceiling."""
    n = mib * (1 << 20) // 4
    src = torch.randn(n, device="cuda:0")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    reps = 10
    times = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        dst.copy_(src)
        e1.record()
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1))
    ms = min(times)
    del src, dst
    torch.cuda.empty_cache()
    return {"mib": mib, "bytes_read": mib << 20, "bytes_written": mib << 20, "launches": reps + 1,
            "ms_per_copy_min": round(ms, 4), "gb_per_s": round(2.0 * (mib << 20) / (ms * 1e-3) / 1e9, 1)}


# Byte mixes of the normalization passes (normpre_stream_ceiling): bytes per
# element and what they stand for.
STREAM_MIXES = {0: (18, "row-active normalize: read 3 fp32, write fp32 + fp16"),
                1: (16, "column-active statistics: read 3 fp32, write fp32"),
                2: (10, "column-active apply: read 2 fp32, write fp16"),
                3: (8, "copy: read fp32, write fp32")}


def stream_ceiling(N, torch, mib):
    """Attainable streaming bandwidth with each normalization byte mix: the
    library's reference kernels over `mib` MiB per fp32 array, best of 10."""
    n = (mib << 20) // 4
    dev = torch.device("cuda:0")
    a, b, c = (torch.randn(n, device=dev) for _ in range(3))
    o32 = torch.empty(n, device=dev)
    o16 = torch.empty(n, device=dev, dtype=torch.float16)
    out = {}
    for mix, (bpe, what) in STREAM_MIXES.items():
        N.normpre_stream_ceiling(mix, a, b, c, o32, o16)
        torch.cuda.synchronize()
        best = None
        for _ in range(10):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            N.normpre_stream_ceiling(mix, a, b, c, o32, o16)
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1)
            best = ms if best is None else min(best, ms)
        out[str(mix)] = {"gb_per_s": round(bpe * n / (best * 1e-3) / 1e9, 1), "bytes_per_element": bpe,
                         "mix": what}
    del a, b, c, o32, o16
    torch.cuda.empty_cache()
    return out


def one_pass_columns(m, n):
    """Whether the library normalizes the columns of an m x n matrix in one
    pass: 16-byte aligned rows and columns of at most 2048 rows padded to a
    multiple of 256 (a strip of them then fits on one CU); longer columns
    take a statistics pass and a normalize pass that reads M and W again."""
    return n % 4 == 0 and -(-m // 256) * 256 <= 2048


def normalize_rooflines(cls, ceiling, shapes):
    """Normalization rooflines per orientation on the algorithmic 18 B per
    element (read G, M_prev, W; write M and fp16 Psi), with the fraction of
    the measured ceiling of the same byte mix; the column-active class also
    on the bytes it moves (18 B per element of one-pass matrices, 26 B =
    statistics 16 B + apply 10 B of two-pass ones) against the ceilings of
    those mixes."""
    out = {}
    total = sum(m * n for m, n in shapes)
    two_pass = sum(m * n for m, n in shapes if not one_pass_columns(m, n)) / total if total else 0.0
    for name, label in (("normalize", "row-active"), ("normalize_col", "column-active")):
        r = roofline_of(cls.get(name), "hbm")
        if not r:
            continue
        r["kernel"] = f"momentum + tangent + normalization, {label}"
        if ceiling:
            c0 = ceiling["0"]["gb_per_s"]
            r["ceiling_gbs_same_mix"] = c0
            r["frac_of_ceiling"] = round(r["achieved"] / c0, 4)
            if name == "normalize_col":
                sec = cls[name]["ms"] / 1e3
                elems = cls[name]["bytes"] / 18.0
                moved = elems * (18.0 + 8.0 * two_pass)
                t_ceil = elems * ((1.0 - two_pass) * 18.0 / (c0 * 1e9) +
                                  two_pass * (16.0 / (ceiling["1"]["gb_per_s"] * 1e9) +
                                              10.0 / (ceiling["2"]["gb_per_s"] * 1e9)))
                r["two_pass_element_share"] = round(two_pass, 4)
                r["moved_gbs"] = round(moved / sec / 1e9, 1)
                r["moved_frac_of_ceiling"] = round(t_ceil / sec, 4)
        out[name] = r
    return out


def kclass_totals(N, ctx):
    out = {}
    for k, name in enumerate(N.KCLASS_NAMES):
        out[name] = N.normpre_kernel_stats(ctx, k, reset=True)
    return out


def time_variant(N, WL, torch, wl, variant, steps, warmup, rank):
    dev = torch.device("cuda:0")
    ws, gs, ms = WL.make_stack(wl, dev)
    torch.cuda.synchronize()
    ctx = N.normpre_init(0)
    # LX: NormPre-L Exact (the leading eigenpairs of the full interaction matrix).
    v = N.VARIANTS["L" if variant == "LX" else variant]
    base_flags = N.NORMPRE_FLAG_L_EXACT if variant == "LX" else 0
    hp = N.normpre_default_hparams(lr=wl.lr, rank=rank, oversample=wl.oversample,
                                   power_iters=wl.power_iters)
    t = 0

    def run(n, flags):
        nonlocal t
        for _ in range(n):
            hp.step = t
            hp.flags = flags | base_flags
            N.normpre_step(ctx, v, ws, gs, ms, hp)
            t += 1

    run(warmup, 0)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    # Clean timed region -> value.
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    e0.record(stream)
    run(steps, 0)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_step = e0.elapsed_time(e1) / steps
    # Instrumented timed region -> per-kernel-class device time.
    kclass_totals(N, ctx)
    torch.cuda.synchronize()
    e0.record(stream)
    run(steps, N.NORMPRE_FLAG_TIME_KERNELS)
    e1.record(stream)
    torch.cuda.synchronize()
    ms_step_instr = e0.elapsed_time(e1) / steps
    classes = kclass_totals(N, ctx)
    N.normpre_destroy(ctx)
    del ws, gs, ms
    torch.cuda.empty_cache()
    return {"ms_per_step": ms_step, "wall_ms_per_step": 1e3 * wall / steps,
            "ms_per_step_instrumented": ms_step_instr, "classes": classes}


def roofline_of(cls, bound):
    if not cls or cls["launches"] == 0 or cls["ms"] <= 0:
        return None
    sec = cls["ms"] / 1e3
    if bound == "mfma":
        ach = cls["flops"] / sec / 1e12
        peak, unit = PEAK_FP16_TFLOPS, "TFLOP/s"
    else:
        ach = cls["bytes"] / sec / 1e9
        peak, unit = PEAK_HBM_GBS, "GB/s"
    return {"bound": bound, "achieved": round(ach, 2), "peak": peak, "unit": unit,
            "frac": round(ach / peak, 4), "traffic": None,
            "launches": cls["launches"], "avg_launch_us": round(1e3 * cls["ms"] / cls["launches"], 2),
            "algorithmic_bytes_per_launch": round(cls["bytes"] / cls["launches"])}


def ns_nominal_flops(shapes, q=5):
    """Nominal Newton-Schulz FLOPs of one step of the plain iteration:
    q (4 s^2 L + 2 s^3) per matrix (Gram 2 s^2 L, A^2 2 s^3, combine 2 s^2 L)."""
    tot = 0.0
    for m, n in shapes:
        sm, lg = float(min(m, n)), float(max(m, n))
        tot += 4.0 * sm * sm * lg + 2.0 * sm ** 3
    return q * tot


def ns_roofline(ns, shapes, steps):
    """Roofline of the Newton-Schulz GEMM class: nominal work (plain
    iteration) per launch over the average launch duration, and the issued
    MFMA work over the same time."""
    if not ns or ns["launches"] == 0 or ns["ms"] <= 0:
        return None
    sec = ns["ms"] / 1e3
    nominal = ns_nominal_flops(shapes) * steps
    ach = nominal / sec / 1e12
    executed = ns["exec_flops"] / sec / 1e12
    return {"bound": "mfma", "achieved": round(ach, 2), "peak": PEAK_FP16_TFLOPS, "unit": "TFLOP/s",
            "frac": round(ach / PEAK_FP16_TFLOPS, 4), "traffic": None,
            "mfma_util_executed": round(executed / PEAK_FP16_TFLOPS, 4),
            "executed_tflops_per_s": round(executed, 2),
            "schedule_tflops_per_s": round(ns["flops"] / sec / 1e12, 2),
            "launches": ns["launches"], "avg_launch_us": round(1e3 * ns["ms"] / ns["launches"], 2),
            "nominal_flops_per_launch": round(nominal / ns["launches"]),
            "executed_flops_per_launch": round(ns["exec_flops"] / ns["launches"]),
            "nominal_flops_per_step": ns_nominal_flops(shapes),
            "algorithmic_bytes_per_launch": round(ns["bytes"] / ns["launches"])}


def merge_classes(classes, names):
    out = {"launches": 0, "ms": 0.0, "flops": 0.0, "exec_flops": 0.0, "bytes": 0.0}
    for n in names:
        c = classes.get(n)
        if c:
            for k in out:
                out[k] += c[k]
    return out


def blas_info():
    """BLAS library numpy calls and its thread count (threadpoolctl)."""
    try:
        from threadpoolctl import threadpool_info
        infos = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        if infos:
            i = infos[0]
            return {"library": f"{i.get('internal_api')} {i.get('version')}", "threads": int(i.get("num_threads", 1)),
                    "arch": i.get("architecture")}
    except Exception:
        pass
    return {"library": "unknown", "threads": len(os.sched_getaffinity(0)), "arch": None}


def cpu_baseline(wl, variant, seconds, rank):
    """Oracle (float64 NumPy) on a bounded sample of the workload: one matrix
    of every shape group of the stack, at t = 0 and t = 1 (both orientations),
    timed per matrix update; the stack step time is the group-size-weighted
    sum, and the rate is reported in whole-stack steps/s.  Stops early (and
    scales what it measured) if `seconds` run out."""
    from oracle import normpre_oracle as O
    from paper_2609_36692_amd import workloads as WL
    blas = blas_info()
    hp = O.HParams(lr=wl.lr, rank=rank, oversample=wl.oversample, power_iters=wl.power_iters)
    groups = {}
    for i, sh in enumerate(wl.shapes):
        groups.setdefault(tuple(sh), []).append(i)
    # A single small matrix (the 256 x 256 case): the median of 10 runs per
    # orientation, and the same with one BLAS thread.
    small = len(wl.shapes) == 1 and wl.shapes[0][0] * wl.shapes[0][1] <= (1 << 20)
    reps = 10 if small else 1

    def one_update(idx, t):
        nonlocal done
        w, g, mp = WL.make_matrix(wl, idx, "cpu")
        runs = []
        for _ in range(reps):
            a = time.perf_counter()
            O.normpre_step(w.numpy(), g.numpy(), mp.numpy(), t, hp, variant, matrix_id=idx)
            runs.append(time.perf_counter() - a)
            done += 1
        return sorted(runs)[len(runs) // 2]

    per_matrix, done = {}, 0
    t0 = time.perf_counter()
    for sh, idx in groups.items():
        times = []
        for t in (0, 1):
            if time.perf_counter() - t0 >= seconds and times:
                break
            times.append(one_update(idx[0], t))
        per_matrix[sh] = sum(times) / len(times)
        if time.perf_counter() - t0 >= seconds:
            break
    measured = [sh for sh in groups if sh in per_matrix]
    covered = sum(len(groups[sh]) for sh in measured)
    est = sum(len(groups[sh]) * per_matrix[sh] for sh in measured) * len(wl.shapes) / covered
    dt = time.perf_counter() - t0
    detail = ", ".join(f"{sh[0]}x{sh[1]} x{len(groups[sh])}: {per_matrix[sh]:.2f} s" for sh in measured)
    out = {"value": round(1.0 / est, 6), "unit": "steps/s", "cores": blas["threads"], "kind": "oracle",
           "sample": f"NormPre-{variant}: one matrix per shape group at t = 0 and 1 ({done} matrix updates"
                     f"{', median of 10 each' if small else ''}, {dt:.1f} s; per matrix {detail}), weighted by "
                     f"group size to the {len(wl.shapes)}-matrix stack ({covered} of {len(wl.shapes)} matrices' "
                     f"groups measured)",
           "blas": blas}
    if small:
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=1):
            one = sum(one_update(0, t) for t in (0, 1)) / 2
        out["one_thread"] = {"value": round(1.0 / one, 6), "unit": "steps/s", "cores": 1}
    return out


def crossover(N, WL, torch, steps, warmup):
    """Per large single matrix: NormPre-G step time against NormPre-L at each
    rank of the sweep, and the rank at which they cost the same (piecewise
    linear between the measured ranks)."""
    import dataclasses
    wl = WL.WORKLOADS["large_sweep"]
    ranks = wl.extra["ranks"]
    rows = []
    for shape in wl.shapes:
        sub = dataclasses.replace(wl, shapes=[shape], name=f"{shape[0]}x{shape[1]}")
        t_g = time_variant(N, WL, torch, sub, "G", steps, warmup, wl.rank)["ms_per_step"]
        t_l = {r: time_variant(N, WL, torch, sub, "L", steps, warmup, r)["ms_per_step"] for r in ranks}
        # Piecewise-linear interpolation of t_L between measured ranks.
        r_star, where = None, "L cheaper at every rank of the sweep"
        if t_l[ranks[0]] > t_g:
            where = "G cheaper at every rank of the sweep"
        else:
            for r0, r1 in zip(ranks, ranks[1:]):
                if t_l[r0] <= t_g < t_l[r1]:
                    r_star = r0 + (r1 - r0) * (t_g - t_l[r0]) / (t_l[r1] - t_l[r0])
                    where = f"crossover between r = {r0} and r = {r1}"
                    break
        rows.append({"shape": list(shape), "ms_G": round(t_g, 4),
                     "ms_L": {str(r): round(t, 4) for r, t in t_l.items()},
                     "crossover_rank": None if r_star is None else round(r_star, 1), "crossover": where})
        print(f"[bench] crossover {shape}: G {t_g:.3f} ms, L {t_l}", file=sys.stderr, flush=True)
    return rows


def main():
    a = parse()
    if a.gpus != 1:
        print(json.dumps({"error": "this library runs on one GPU; --gpus above 1 is not supported "
                                   "(across GPUs the step would shard by matrix ownership)"}))
        sys.exit(2)
    import torch
    from paper_2609_36692_amd import normpre as N
    from paper_2609_36692_amd import workloads as WL
    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    if not os.path.exists(N.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    if a.crossover:
        rows = crossover(N, WL, torch, a.steps, a.warmup)
        line = {"metric": "NormPre-G vs NormPre-L step time on large single matrices (cost crossover in r)",
                "unit": "ms/step", "n_gpus": 1, "steps": a.steps, "warmup": a.warmup, "higher_is_better": False,
                "dtype": "fp16", "precision": "fp16 MFMA operands, fp32 accumulate and state", "data": "synthetic",
                "config": {"workload": "large_sweep: 4096^2, 4096x16384, 8192^2, 8192x28672, power-law spectrum",
                           "ranks": WL.WORKLOADS["large_sweep"].extra["ranks"], "oversample": 8, "power_iters": 1},
                "rows": rows}
        s = json.dumps(line)
        if a.json_out:
            with open(a.json_out, "w") as f:
                f.write(s + "\n")
        print(s)
        return
    wl = WL.WORKLOADS[a.workload]
    rank = a.rank or wl.rank
    variants = [v.strip().upper() for v in a.variants.split(",") if v.strip()]
    traffic = measured_traffic(wl.name)
    ceiling = stream_ceiling(N, torch, a.ceiling_mib) if a.ceiling_mib > 0 else None
    res = {}
    for v in variants:
        r = time_variant(N, WL, torch, wl, v, a.steps, a.warmup, rank)
        cls = r["classes"]
        if v in ("G", "MUON"):
            ns = merge_classes(cls, ["ns_gram", "ns_poly", "ns_combine"])
            roof = ns_roofline(ns, wl.shapes, a.steps)
            roof["kernel"] = "Newton-Schulz GEMMs (gram + poly + Gram-space products + combine, fp16 MFMA)"
        elif v == "NORM":
            roof = roofline_of(merge_classes(cls, ["normalize", "normalize_col"]), "hbm")
            roof["kernel"] = "momentum + tangent + normalization"
        elif v == "LX":
            roof = roofline_of(cls["eigen"], "hbm")
            roof["kernel"] = ("dense eigensolver (tridiagonal reduction, fp32 storage / fp64 arithmetic: one read + write of the trailing "
                              "block per step; bisection, inverse iteration)")
        else:
            roof = roofline_of(cls["sk_stream"], "hbm")
            roof["kernel"] = "sketch products streaming Psi (fp16 MFMA, split-K)"
        if roof and v in traffic:
            roof["traffic"] = round(traffic[v]["bytes_per_launch"], 1)
            roof["traffic_detail"] = traffic[v]
        norm_roof = normalize_rooflines(cls, ceiling, wl.shapes)
        total_dev = sum(c["ms"] for c in cls.values())
        res[v] = {
            "steps_per_s": round(1e3 / r["ms_per_step"], 3),
            "ms_per_step": round(r["ms_per_step"], 4),
            "wall_ms_per_step": round(r["wall_ms_per_step"], 4),
            "ms_per_step_instrumented": round(r["ms_per_step_instrumented"], 4),
            "roofline": roof,
            "normalize_roofline": norm_roof,
            "kernel_ms_per_step": {k: round(c["ms"] / a.steps, 4) for k, c in cls.items() if c["launches"]},
            "kernel_share": {k: round(c["ms"] / total_dev, 4) for k, c in cls.items() if c["launches"]},
        }
        if v in ("G", "MUON"):
            nominal = ns_nominal_flops(wl.shapes)
            res[v]["ns_nominal_tflop_per_step"] = round(nominal / 1e12, 4)
            res[v]["ns_nominal_tflops_per_s_whole_step"] = round(nominal / 1e12 / (r["ms_per_step"] / 1e3), 2)
        print(f"[bench] NormPre-{v}: {res[v]['ms_per_step']:.3f} ms/step", file=sys.stderr, flush=True)

    # Optimizer latency relative to the Muon reference step through the same
    # kernels (the comparison of the paper's efficiency tables).
    rel = None
    if "MUON" in res:
        rel = {f"{v}_vs_MUON": round(res[v]["ms_per_step"] / res["MUON"]["ms_per_step"] - 1.0, 4)
               for v in res if v != "MUON"}
    copy_ref = copy_reference(torch, a.copy_mib) if a.copy_mib > 0 else None

    cpu = None
    if not a.no_cpu_baseline:
        for v in variants:
            if v not in ("G", "L"):
                continue
            cb = cpu_baseline(wl, v, a.cpu_seconds, rank)
            res[v]["cpu_baseline"] = cb
            print(f"[bench] cpu baseline NormPre-{v}: {cb['value']} steps/s ({cb['sample']})", file=sys.stderr,
                  flush=True)
        cpu = res[variants[0]].get("cpu_baseline")

    # The paper's other optimizer-latency workload, for the comparison of its
    # efficiency tables (context).
    gpt2 = None
    if not a.no_gpt2 and wl.name != "gpt2_small":
        g2 = WL.WORKLOADS["gpt2_small"]
        gpt2 = {}
        for v in ("G", "L"):
            r = time_variant(N, WL, torch, g2, v, a.steps, a.warmup, g2.rank)
            entry = {"steps_per_s": round(1e3 / r["ms_per_step"], 3), "ms_per_step": round(r["ms_per_step"], 4)}
            if (g2.name, v) in PAPER_STEPS_PER_S:
                entry["vs_paper_a100"] = round(entry["steps_per_s"] / PAPER_STEPS_PER_S[(g2.name, v)], 2)
            if v == "G":
                ns = merge_classes(r["classes"], ["ns_gram", "ns_poly", "ns_combine"])
                entry["ns_roofline"] = ns_roofline(ns, g2.shapes, a.steps)
            gpt2[v] = entry
            print(f"[bench] gpt2_small NormPre-{v}: {entry['ms_per_step']:.3f} ms/step", file=sys.stderr, flush=True)

    primary = variants[0]
    p = res[primary]
    line = {
        "metric": "optimizer steps/sec per full layer stack + NS GEMM TFLOP/s, % MFMA/HBM peak",
        "value": p["steps_per_s"],
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": p["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": (round(p["steps_per_s"] / PAPER_STEPS_PER_S[(wl.name, primary)], 2)
                        if (wl.name, primary) in PAPER_STEPS_PER_S else None),
        "vs_baseline_ref": ({"value": round(PAPER_STEPS_PER_S[(wl.name, primary)], 3), "unit": "steps/s",
                             "source": "paper's optimizer latency, NVIDIA A100 80GB (context, not a target)"}
                            if (wl.name, primary) in PAPER_STEPS_PER_S else None),
        "dtype": "fp16",
        "precision": "fp16 MFMA operands, fp32 accumulate; fp32 normalization, update and state",
        "data": "synthetic",
        "config": {"workload": f"{wl.name}: {wl.description}", "matrices": len(wl.shapes),
                   "elements": wl.elements, "variant": f"NormPre-{primary}",
                   "ns_iters": 5, "rank": rank, "oversample": wl.oversample,
                   "power_iters": wl.power_iters, "parallelism": "single GPU"},
        "roofline": p["roofline"],
        "cpu_baseline": cpu,
        "variants": res,
    }
    if gpt2:
        line["gpt2_small"] = gpt2
    if ceiling:
        line["stream_ceiling"] = ceiling
    if copy_ref:
        line["copy_reference"] = copy_ref
    if rel:
        line["latency_vs_muon"] = rel
    s = json.dumps(line)
    if a.json_out:
        with open(a.json_out, "w") as f:
            f.write(s + "\n")
    print(s)


if __name__ == "__main__":
    main()
