"""Benchmark: WAMachine-style replans on one MI355X.

A timed step is one closed-loop replan of the large joint video/action DiT
(28 layers, hidden 1536, 24 heads, MLP 6144; 8 frames of 30x40 = 9600 video +
64 action (14-dim) + 512 observation tokens; 20 flow steps; bf16
contractions): Trajectory Remapping of the previous replan's state (entry at
stage 10), an anticipatory prefix of 4 steps under the predicted observation,
the consistency score and rebinding (or restart), and Residual Rescaling
inside every denoising step, all through libwam.  Inputs (weights, noise,
AR(1) observations) are seeded, synthetic and resident in HBM before timing
starts.  `value` counts denoising steps per second.

The same line carries: the native full re-denoise of that model, the
dominant kernel against the bf16 MFMA peak (roofline), the adaptation
kernels against HBM, the achievable-peak probes, the float64 oracle on the
host (cpu_baseline), and the closed-loop replay of the small model (12
layers, hidden 768, T = 864, 10 steps) as extra keys.  --workload selects
another model for the headline.

Prints one JSON line.  --gpus N > 1 is refused: the library runs on one GPU.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16
HBM_PEAK_GBS = 8000.0
ATTN_VARIANTS = {"auto": 0, "running": 1, "bounded": 2, "pingpong": 3, "plain": 4}
CLASS_NAMES = ["gemm_qkv", "gemm_proj", "gemm_fc1", "gemm_fc2", "attention", "rr_gate", "rr_inject",
               "rr_refresh"]


def source_hash() -> str:
    """Hash of the HIP sources; a PMC traffic summary is valid only for these."""
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(ROOT, "paper_2609_34608_amd", "csrc", "*"))):
        with open(f, "rb") as fh:
            h.update(os.path.basename(f).encode())
            h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_path(workload: str) -> str:
    return os.path.join(ROOT, "profiles", f"pmc_traffic_{workload}.json")


def kernel_class(name: str):
    """Kernel class of a rocprofv3 kernel name (None if not a timed class)."""
    m = re.search(r"gemm_bf16_kernel<\s*\d+,\s*\d+,\s*\d+,\s*\d+,\s*\d+,\s*\d+,\s*\d+,\s*(\d+),", name)
    if m:
        return CLASS_NAMES[int(m.group(1))]
    m = re.search(r"gemm_splitk_reduce_kernel<\s*\d+,\s*(\d+)>", name)  # second pass of a split GEMM
    if m:
        return CLASS_NAMES[int(m.group(1))]
    for key, cls in (("attn_bf16", "attention"), ("rr_row_sums_kernel", "rr_gate"),
                     ("rr_finish_kernel", "rr_gate"), ("rr_gate_partials_kernel", "rr_gate"),
                     ("rr_gate_finish_kernel", "rr_gate"), ("rr_inject_kernel", "rr_inject"),
                     ("rr_refresh_kernel", "rr_refresh")):
        if key in name:
            return cls
    return None


def summarize_pmc(fetch_csv, write_csv, probe_mb, workload, commands):
    """Per-class HBM traffic per launch from two rocprofv3 --pmc runs
    (FETCH_SIZE, WRITE_SIZE), each scaled by what the counter reads for the
    plain device copy of probe_mb MiB that the same run performs."""
    def load(path, counter):
        per = {}
        with open(path) as f:
            for r in csv.DictReader(f):
                if r.get("Counter_Name") != counter:
                    continue
                per.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
        return per
    fetch, write = load(fetch_csv, "FETCH_SIZE"), load(write_csv, "WRITE_SIZE")
    probe_bytes = probe_mb * 2.0 ** 20
    f_read = probe_bytes / max(fetch.get("__amd_rocclr_copyBuffer", [1.0]))
    f_write = probe_bytes / max(write.get("__amd_rocclr_copyBuffer", [1.0]))
    classes = {}
    for name in set(fetch) | set(write):
        cls = kernel_class(name)
        if cls is None:
            continue
        fv, wv = fetch.get(name, [0.0]), write.get(name, [0.0])
        c = classes.setdefault(cls, {"kernels": [], "fetch_counter": 0.0, "write_counter": 0.0})
        c["kernels"].append(name)
        c["fetch_counter"] += sum(fv) / len(fv)
        c["write_counter"] += sum(wv) / len(wv)
    for c in classes.values():
        c["traffic_bytes"] = c["fetch_counter"] * f_read + c["write_counter"] * f_write
    out = {"workload": workload, "source_hash": source_hash(), "probe_mib": probe_mb,
           "probe_counter": {"FETCH_SIZE": max(fetch.get("__amd_rocclr_copyBuffer", [0.0])),
                             "WRITE_SIZE": max(write.get("__amd_rocclr_copyBuffer", [0.0]))},
           "scale": {"read": f_read, "write": f_write}, "commands": commands, "classes": classes}
    with open(traffic_path(workload), "w") as f:
        json.dump(out, f, indent=1, sort_keys=True)
    print(json.dumps({k: round(v["traffic_bytes"]) for k, v in classes.items()}))


def class_flops(spec, cls: str) -> float:
    """Algorithmic FLOP of one launch of a contraction class at a workload."""
    M, D, F, T, B = spec.M, spec.D, spec.F, spec.T, spec.B
    return {"gemm_qkv": 2.0 * M * D * 3 * D, "gemm_proj": 2.0 * M * D * D, "gemm_fc1": 2.0 * M * D * F,
            "gemm_fc2": 2.0 * M * F * D, "attention": 4.0 * B * T * T * D}[cls]


def summarize_mfma(pmc_csv, workload, commands, simds=1024, xcds=8):
    """MFMA counters per contraction class from one rocprofv3 --pmc run
    (SQ_INSTS_VALU_MFMA_MOPS_BF16, SQ_VALU_MFMA_BUSY_CYCLES, GRBM_GUI_ACTIVE,
    SQ_BUSY_CU_CYCLES): bf16 MFMA FLOP counted by the hardware against the
    algorithmic FLOP, MFMA-busy fraction of the SIMDs over the dispatch, and
    the shader clock implied by GRBM_GUI_ACTIVE over the dispatch time.
    rocprofv3 reports GRBM_GUI_ACTIVE summed over the 8 XCDs (each has its own
    graphics block), so one XCD's active cycles are the value / 8."""
    from synth import get_workload
    spec = get_workload(workload)
    per = {}
    with open(pmc_csv) as f:
        for r in csv.DictReader(f):
            cls = kernel_class(r["Kernel_Name"])
            if cls is None or not cls.startswith(("gemm", "attention")):
                continue
            d = per.setdefault(cls, {}).setdefault(r["Dispatch_Id"], {"name": r["Kernel_Name"]})
            d[r["Counter_Name"]] = float(r["Counter_Value"])
            d["ns"] = float(r["End_Timestamp"]) - float(r["Start_Timestamp"])
    rows = []
    for cls in CLASS_NAMES:
        if cls not in per:
            continue
        ds = [d for d in per[cls].values() if "SQ_INSTS_VALU_MFMA_MOPS_BF16" in d and "GRBM_GUI_ACTIVE" in d]
        if not ds:
            continue
        n = len(ds)
        avg = lambda k: sum(d[k] for d in ds) / n  # noqa: E731
        ns = avg("ns")
        flop_hw = avg("SQ_INSTS_VALU_MFMA_MOPS_BF16") * 512.0
        flop_alg = class_flops(spec, cls)
        active = avg("GRBM_GUI_ACTIVE") / xcds  # cycles of one XCD
        busy = avg("SQ_VALU_MFMA_BUSY_CYCLES") / (active * simds)
        clock = active / ns  # GHz
        rows.append((cls, n, ns / 1e3, flop_alg / 1e9, flop_hw / 1e9, flop_hw / flop_alg,
                     flop_alg / ns / 1e3, flop_alg / ns / 1e3 / MFMA_BF16_PEAK_TFLOPS, busy, clock,
                     flop_hw / ns / 1e3 / (clock * 1e9 * simds * 1024 / 1e12)))
    path = os.path.join(ROOT, "profiles", f"mfma_counters_{workload}.md")
    with open(path, "w") as f:
        f.write(f"# MFMA counters — {workload} workload (bench.py --workload {workload})\n\n")
        f.write("Commands (repository root, one MI355X, after `cd /tmp && export TMPDIR=/tmp` for the "
                "profiler's files):\n\n")
        for c in commands:
            f.write(f"    {c}\n")
        f.write("\nPer contraction class, averaged over its dispatches (kernels serialised by the counter "
                "collection):\n\n")
        f.write("* hw GFLOP = SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512 (the bf16 MFMA work the hardware issued);\n"
                "* alg GFLOP = the algorithmic work of one launch (2MNK; attention 4 B T^2 D);\n"
                "* TFLOP/s and % of 2.5 PF = alg GFLOP / dispatch time;\n"
                "* MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / 8 x 1024 SIMDs) (rocprofv3 sums "
                "GRBM_GUI_ACTIVE over the 8 XCDs);\n"
                "* clock = GRBM_GUI_ACTIVE / 8 / dispatch time;\n"
                "* issue at clock = hw FLOP / (time x clock x 1024 SIMDs x 1024 FLOP per SIMD-cycle), the "
                "fraction of the dense bf16 rate at the measured clock.\n\n")
        f.write("| class | dispatches | avg us | alg GFLOP | hw GFLOP | hw/alg | TFLOP/s | % of 2.5 PF | "
                "MFMA busy | clock GHz | issue at clock |\n|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|\n")
        for r in rows:
            f.write(f"| {r[0]} | {r[1]} | {r[2]:.2f} | {r[3]:.2f} | {r[4]:.2f} | {r[5]:.4f} | {r[6]:.1f} | "
                    f"{100 * r[7]:.1f}% | {100 * r[8]:.1f}% | {r[9]:.3f} | {100 * r[10]:.1f}% |\n")
        f.write(f"\nSource hash of the HIP kernels: `{source_hash()}`.\n")
    print(open(path).read())


def lookup_traffic(workload: str, cls: str):
    """Traffic per launch of a class from the committed PMC summary, or None
    when there is none or the kernels changed since the counters were taken."""
    try:
        with open(traffic_path(workload)) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("source_hash") != source_hash() or cls not in t.get("classes", {}):
        return None
    return t["classes"][cls]["traffic_bytes"]


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=2)
    p.add_argument("--workload", default="large",
                   help="large (default: the 16-frame model) | mid | replay (small model) | idm (independent "
                        "video / action pair)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-native", action="store_true")
    p.add_argument("--no-probes", action="store_true", help="skip the achievable-peak probes")
    p.add_argument("--no-replay", action="store_true",
                   help="skip the extra small-model closed-loop replay figures")
    p.add_argument("--cpu-sample-steps", type=int, default=5)
    p.add_argument("--tau", type=float, default=None,
                   help="Observation Rebinding threshold tau (default: the workload's, 0.5; 0.3 rejects every "
                        "rebinding on the AR(1) observations, whose score is ~0.44)")
    p.add_argument("--rr-mode", default="auto", choices=["auto", "force_skip", "force_full", "off"],
                   help="residual-rescaling mode of the timed replans")
    p.add_argument("--exec", default="host", choices=["host", "device", "graph"],
                   help="RR decision on the host, on the device, or on the device with graph replay")
    p.add_argument("--attention", default="auto", choices=list(ATTN_VARIANTS),
                   help="bf16 attention kernel: auto, running-max softmax, bounded (fixed reference from the "
                        "QK-norm score bound, software-pipelined), the bounded ping-pong form, or the "
                        "bounded plain loop")
    p.add_argument("--copy-probe-mib", type=int, default=0,
                   help="one plain device copy of this size before timing (PMC calibration)")
    p.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                   help="write the per-class traffic summary of two --pmc runs and exit")
    p.add_argument("--pmc-command", action="append", default=[], help="command lines recorded in the summary")
    p.add_argument("--summarize-mfma", metavar="PMC_CSV",
                   help="write the MFMA-counter summary of one --pmc run (profiles/mfma_counters_<workload>.md) "
                        "and exit")
    p.add_argument("--ablation", action="store_true",
                   help="closed-loop GPU time and observation-to-action latency per variant, then exit")
    p.add_argument("--diagnostics", action="store_true",
                   help="state-continuity diagnostics (layer change, reuse output error, consecutive-replan "
                        "latent similarity, remapped-vs-native action RMSE), then exit")
    p.add_argument("--sweep", action="store_true",
                   help="bandwidth of Trajectory Remapping and the rebinding score at 2^22 .. 2^28 elements, "
                        "then exit")
    p.add_argument("--window-ms", type=float, default=20.0,
                   help="simulated action-execution window between replans (ablation mode)")
    return p.parse_args()


def main():
    args = parse()
    if args.summarize_pmc:
        summarize_pmc(args.summarize_pmc[0], args.summarize_pmc[1], args.copy_probe_mib, args.workload,
                      args.pmc_command)
        return
    if args.summarize_mfma:
        summarize_mfma(args.summarize_mfma, args.workload, args.pmc_command)
        return
    if args.ablation:
        if args.gpus != 1:
            sys.exit(2)
        from synth.workloads import PAIRS
        if args.workload in PAIRS:
            print("the ablation runs on the single-model workloads", file=sys.stderr)
            sys.exit(2)
        ablation(args)
        return
    if args.diagnostics:
        diagnostics(args)
        return
    if args.sweep:
        sweep(args)
        return
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU (asked for {args.gpus}); the library has no "
              "multi-GPU path.", file=sys.stderr)
        sys.exit(2)
    from synth.workloads import PAIRS
    if args.workload in PAIRS:
        idm_main(args)
        return
    out = measure(args, args.workload, args.steps, args.warmup, cpu=not args.no_cpu_baseline,
                  native=not args.no_native, adapt=True, copy_probe_mib=args.copy_probe_mib)
    if not args.no_probes:
        out["achievable"] = achievable_peaks()
        ach = out["achievable"]["mfma_bf16_16x16x32_tflops"]
        out["roofline"]["frac_of_achievable"] = round(out["roofline"]["achieved"] / ach, 5)
        out["mfma_frac_dit_of_achievable"] = round(out["dit_tflops"] / ach, 5)
        cg = out["achievable"]["copy_gbs"]
        for v in out.get("adaptation_kernels", {}).values():
            v["frac_of_achievable_copy"] = round(v["GB/s"] / cg, 4)
    if not args.no_replay and args.workload != "replay":
        r = measure(args, "replay", 30, 5, cpu=False, native=not args.no_native, adapt=False)
        out["replay"] = {k: r[k] for k in ("value", "unit", "ms_per_step", "action_chunks_per_s",
                                           "denoise_steps_per_replan", "dit_tflops", "mfma_frac_dit",
                                           "native_chunk_ms", "reuse_latency_speedup", "reuse_stats")
                         if k in r}
        out["replay"]["workload"] = r["config"]["workload"]
        out["replay"]["dominant_kernel"] = {k: r["roofline"][k]
                                            for k in ("kernel", "achieved", "frac", "avg_launch_us")}
    print(json.dumps(out), flush=True)


def sweep(args):
    """Trajectory Remapping (wam_remap_noalloc: rms runs, their sum, the
    remapped initialisation) and the Observation Rebinding score
    (wam_consistency_score: run sums on the device, their sum on the host)
    over 2^22 .. 2^28 trajectory / condition elements, beside a plain copy of
    the same size: the bandwidth of these operators once they are not
    latency-bound.  Algorithmic bytes: remap 20 per element (the rms pass
    reads x^r and x_bar, the remap reads them again and writes x; no slot is
    shifted out, so no noise is read), score 8 (u_hat and u), copy 8."""
    import numpy as np
    import torch

    from paper_2609_34608_amd import runtime as R
    from synth import get_workload, make_weights
    dev = torch.device("cuda:0")
    tiny = get_workload("tiny")
    m = R.WamModel(R.config_of(tiny), make_weights(tiny), device=dev)
    rows = []
    for lg in range(22, 29):
        n = 1 << lg
        spec = tiny.replace(B=1, Nv=n // 16, Cv=16, Na=0, A=1)
        cfg = R.config_of(spec)
        g = torch.Generator(device=dev).manual_seed(lg)
        xb = torch.randn(1, n, device=dev, generator=g)
        xr = torch.randn(1, n, device=dev, generator=g)
        eps = torch.randn(1, n, device=dev, generator=g)
        out = torch.empty_like(xb)
        reps = 20
        R.remap_noalloc(cfg, xb, xr, 0.6, 0.75, 0, 0, eps, out)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            R.remap_noalloc(cfg, xb, xr, 0.6, 0.75, 0, 0, eps, out)
        e1.record()
        e1.synchronize()
        t_tr = e0.elapsed_time(e1) / reps
        m.consistency_score([xb], [xr], [1.0], [1.0])
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(reps):
            m.consistency_score([xb], [xr], [1.0], [1.0])
        t_or = (time.perf_counter() - t0) / reps * 1e3
        gbs_copy, t_cp = R.probe_copy(n * 4, reps=reps)
        r = {"log2_elements": lg, "remap_us": round(1e3 * t_tr, 2),
             "remap_GBs": round(20.0 * n / (t_tr * 1e-3) / 1e9, 1),
             "score_us": round(1e3 * t_or, 2), "score_GBs": round(8.0 * n / (t_or * 1e-3) / 1e9, 1),
             "copy_us": round(1e3 * t_cp, 2), "copy_GBs": round(gbs_copy, 1)}
        r["remap_frac_hbm"] = round(r["remap_GBs"] / HBM_PEAK_GBS, 4)
        r["score_frac_hbm"] = round(r["score_GBs"] / HBM_PEAK_GBS, 4)
        rows.append(r)
        print(json.dumps(r), flush=True)
        del xb, xr, eps, out
    m.close()
    print(json.dumps({"sweep": rows}), flush=True)


def progress(msg: str) -> None:
    """One progress line on stderr (the JSON result stays the only stdout line)."""
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def achievable_peaks():
    """What the chip reaches in practice: the bf16 MFMA issue rate on register
    operands (both MFMA shapes) and a streaming copy of 1 GiB."""
    from paper_2609_34608_amd import runtime as R
    # each timed launch lasts ~90 ms after a warm-up launch of the same length:
    # launches of a few ms end before the shader clock has ramped up from idle
    # and read ~20% low
    iters = 400_000
    t16, _ = R.probe_mfma_bf16(shape=0, iters=iters)
    t32, _ = R.probe_mfma_bf16(shape=1, iters=iters)
    gbs, _ = R.probe_copy(1 << 30, reps=100)
    return {"mfma_bf16_16x16x32_tflops": round(t16, 1), "mfma_bf16_32x32x16_tflops": round(t32, 1),
            "copy_gbs": round(gbs, 1),
            "method": f"wam_probe_mfma_bf16 (1024 blocks x 4 waves, {iters} rounds of independent MFMA chains "
                      "on register operands, one timed launch after a warm-up launch) and wam_probe_copy "
                      "(1 GiB device copy, one 16-byte element per thread, read + write bytes counted, 100 "
                      "timed copies), HIP events"}


def measure(args, name, steps, warmup, cpu, native, adapt, copy_probe_mib=0):
    """Closed-loop replans of workload `name` (one timed step = one replan);
    returns the bench record."""
    import numpy as np
    import torch

    from paper_2609_34608_amd import _lib as L
    from paper_2609_34608_amd import runtime as R
    from synth import get_workload, make_weights, make_initial_noise, make_observations, make_remap_noise

    spec = get_workload(name)
    if args.tau is not None:
        spec = spec.replace(or_tau=args.tau)
    dev = torch.device("cuda:0")
    progress(f"{name}: generating weights")
    W = make_weights(spec)
    progress(f"{name}: weights ready")
    m = R.WamModel(R.config_of(spec), W, device=dev, own_stream=args.exec == "graph")
    m.set_option(L.WAM_OPT_ATTENTION, ATTN_VARIANTS[args.attention])
    if args.exec in ("device", "graph"):
        m.set_option(L.WAM_OPT_DEVICE_DECISION, 1)
    if args.exec == "graph":
        m.set_option(L.WAM_OPT_GRAPHS, 1)
    K = spec.K
    s = np.arange(K + 1, dtype=np.float64)
    sig = (1.0 - s / K)  # uniform flow schedule sigma_k = 1 - k/K
    m.set_schedule(sig)
    q, s_, e = spec.rr_bounds
    modes = {"auto": L.WAM_RR_AUTO, "force_skip": L.WAM_RR_FORCE_SKIP, "force_full": L.WAM_RR_FORCE_FULL,
             "off": L.WAM_RR_OFF}
    rr = R.rr_profile(q, s_, e, modes[args.rr_mode], spec.rr_alpha_min, spec.rr_alpha_max, spec.rr_eps,
                      spec.rr_gamma_cos, spec.rr_gamma_fit)
    n_ctrl = 1 + warmup + steps
    obs = make_observations(spec, n_ctrl)
    rho = spec.ar_rho
    delta = 1.0 / np.sqrt(1.0 - rho * rho)
    obs_d = torch.from_numpy(obs).to(dev)
    pred_d = torch.from_numpy((rho * obs[:-1]).astype(np.float32)).to(dev)
    noise_first = torch.from_numpy(make_initial_noise(spec)).to(dev)
    remap_noise = torch.from_numpy(np.stack([make_remap_noise(spec, t) for t in range(n_ctrl)])).to(dev)
    x_out = m.new_traj()
    ra = dict(b0=spec.tr_b0, r=spec.tr_r, shift_action=spec.shift_action, shift_video=spec.shift_video,
              k1=spec.or_k1, tau=spec.or_tau, kappa_max=spec.or_kappa_max)

    def replan(t, rr=rr):
        cr = obs_d[t]
        cp = pred_d[t - 1] if t > 0 else obs_d[t]
        return m.replan(cr, x_out, remap_noise[t], cond_pred=cp, u_hat=[cp], u=[cr], delta=[delta],
                        weight=[1.0], noise_first=noise_first, rr=rr, **ra)

    if copy_probe_mib:
        n = copy_probe_mib * 2 ** 18
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    torch.cuda.synchronize()
    t = 0
    replan(t)  # first replan: native K steps from noise
    t += 1
    for _ in range(warmup):
        replan(t)
        t += 1
    # untimed attribution pass over one replan: which kernel class dominates
    classes = [L.WAM_KC_GEMM_QKV, L.WAM_KC_GEMM_PROJ, L.WAM_KC_GEMM_FC1, L.WAM_KC_GEMM_FC2,
               L.WAM_KC_ATTENTION]
    for kc in classes:
        m.profile_enable(kc, True, 4096)
    replan(t - 1 if t > 1 else t)
    tot = {kc: m.profile_read(kc)[0] for kc in classes}
    for kc in classes:
        m.profile_enable(kc, False)
    dom = max(tot, key=tot.get)
    m.reset_all()
    replan(0)
    for tt in range(1, t):
        replan(tt)
    # timed region: events around the dominant kernel's launches only
    m.profile_enable(dom, True, 200000)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    infos = []
    per_replan = []  # wall time of each replan, chunk ready (a control step waits for it)
    for _ in range(steps):
        ts = time.perf_counter()
        infos.append(replan(t))
        torch.cuda.synchronize()
        per_replan.append(time.perf_counter() - ts)
        t += 1
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    dom_ms, dom_n, dom_work = m.profile_read(dom)
    m.profile_enable(dom, False)
    progress(f"{name}: timed region done ({steps} replans in {elapsed:.2f} s)")

    n_steps = sum(i.steps for i in infos)
    layers_eval = sum(i.steps * spec.L - i.layers_skipped for i in infos)
    flops = spec.flops_per_layer() * layers_eval
    ms_per_step = 1000.0 * elapsed / steps
    steps_per_s = n_steps / elapsed
    chunks_per_s = steps / elapsed
    n_att = sum(i.rr_attempts for i in infos)
    n_reuse = sum(i.rr_reuses for i in infos)
    skip = sum(i.layers_skipped for i in infos)
    dense = sum(i.layers_dense for i in infos)
    n_start = sum(i.n_start for i in infos)
    n_bind = sum(i.n_bind for i in infos)

    dom_tflops = dom_work / (dom_ms * 1e-3) / 1e12 if dom_ms > 0 else 0.0
    out = {
        "metric": "denoise steps/s + action chunks/s per MI355X; MFMA % of bf16 peak",
        "value": round(steps_per_s, 3),
        "unit": "denoise steps/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if spec.dtype == "bf16" else "f32",
        "data": "synthetic (seeded random-init weights N(0,0.02), N(0,1) noise, AR(1) observations)",
        "config": {
            "workload": (f"{spec.name}: closed-loop replan with TR+OR+RR on a joint video/action DiT "
                         f"B{spec.B} L{spec.L} D{spec.D} H{spec.H} F{spec.F} T{spec.T} "
                         f"(video {spec.Nv}, action {spec.Na}x{spec.A}, obs {spec.No}) K{spec.K} "
                         f"b0={spec.tr_b0} k1={spec.or_k1} tau={spec.or_tau} shift={spec.shift_action}"),
            "step": "one replan (control step)",
            "exec": args.exec,
            "attention": args.attention,
        },
        "action_chunks_per_s": round(chunks_per_s, 3),
        "denoise_steps_per_replan": n_steps / steps,
        "ms_per_replan_median": round(1000.0 * float(np.median(per_replan)), 4),
        "ms_per_replan_min_max": [round(1000.0 * min(per_replan), 4), round(1000.0 * max(per_replan), 4)],
        # a batched step denoises B samples (and a replan yields B chunks)
        "batch": spec.B,
        "sample_steps_per_s": round(steps_per_s * spec.B, 3),
        "sample_chunks_per_s": round(chunks_per_s * spec.B, 3),
        "mfma_frac_dit": round(flops / elapsed / 1e12 / MFMA_BF16_PEAK_TFLOPS, 5),
        "dit_tflops": round(flops / elapsed / 1e12, 3),
        "reuse_stats": {"rr_accept": n_reuse / n_att if n_att else None,
                        "rr_skip_frac": skip / dense if dense else None,
                        "or_accept": n_bind / n_start if n_start else None,
                        "or_coverage": n_bind / steps},
        "roofline": {
            "kernel": L.KERNEL_CLASS_NAMES[dom],
            "bound": "mfma",
            "achieved": round(dom_tflops, 3),
            "peak": MFMA_BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(dom_tflops / MFMA_BF16_PEAK_TFLOPS, 5),
            "traffic": lookup_traffic(spec.name, L.KERNEL_CLASS_NAMES[dom]),
            "launches": dom_n,
            "avg_launch_us": round(1000.0 * dom_ms / dom_n, 3) if dom_n else None,
            "class_ms_one_replan": {L.KERNEL_CLASS_NAMES[k]: round(v, 4) for k, v in tot.items()},
        },
    }

    if adapt:
        out["adaptation_kernels"] = adaptation_kernels(m, spec, replan, t)

    if native:
        # full re-denoise of the same model: K native steps from noise per chunk
        xn = m.new_traj()
        nrep = max(3, steps // 5)
        m.reset_all()
        xn.copy_(noise_first)
        m.continue_(0, K, xn, obs_d[0])
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(nrep):
            xn.copy_(noise_first)
            m.continue_(0, K, xn, obs_d[i + 1])
        torch.cuda.synchronize()
        nat = (time.perf_counter() - t0) / nrep
        out["native_chunk_ms"] = round(1000.0 * nat, 4)
        out["native_steps_per_s"] = round(K / nat, 3)
        out["reuse_latency_speedup"] = round(nat / (elapsed / steps), 4)

    if cpu:
        progress(f"{name}: float64 oracle on the host")
        # models whose float64 step would take minutes are timed one layer at a time
        out["cpu_baseline"] = (cpu_baseline_layer(spec, W) if spec.flops_per_step() > 1e12
                               else cpu_baseline(spec, W, obs, args.cpu_sample_steps))
    m.close()
    return out


def adaptation_kernels(m, spec, replan, t):
    """Residual-Rescaling kernels at the workload's size: two extra (untimed)
    replans with reuse forced, so that the gate, the injection and the refresh
    all run, each launch timed by its dispatch stamps."""
    from paper_2609_34608_amd import _lib as L
    from paper_2609_34608_amd import runtime as R
    q, s_, e = spec.rr_bounds
    rr_force = R.rr_profile(q, s_, e, L.WAM_RR_FORCE_SKIP, spec.rr_alpha_min, spec.rr_alpha_max, spec.rr_eps,
                            spec.rr_gamma_cos, spec.rr_gamma_fit)
    ad = [L.WAM_KC_RR_GATE, L.WAM_KC_RR_INJECT, L.WAM_KC_RR_REFRESH]
    for kc in ad:
        m.profile_enable(kc, True, 4096)
    for _ in range(2):
        replan(t - 1, rr=rr_force)
    adapt = {}
    for kc in ad:
        ms_, n_, bytes_ = m.profile_read(kc)
        m.profile_enable(kc, False)
        if n_:
            gbs = bytes_ / (ms_ * 1e-3) / 1e9
            adapt[L.KERNEL_CLASS_NAMES[kc]] = {"launches": n_, "avg_us": round(1000.0 * ms_ / n_, 3),
                                               "bytes_per_launch": bytes_ / n_, "GB/s": round(gbs, 1),
                                               "frac_hbm": round(gbs / HBM_PEAK_GBS, 4)}
    return adapt


def idm_main(args):
    """Independent execution of the video and action branches (Sec. 3.3,
    Fast-WAM-IDM profiles): one step = one control step of the pair (video
    replan under the observation, action replan under the observation and the
    video latent).  value counts the denoising steps of both models."""
    import numpy as np
    import torch

    from paper_2609_34608_amd import _lib as L
    from paper_2609_34608_amd import runtime as R
    from synth import get_pair, make_weights, make_initial_noise, make_observations, make_remap_noise

    sv, sa = get_pair(args.workload)
    dev = torch.device("cuda:0")
    Wv, Wa = make_weights(sv), make_weights(sa)
    models = [R.WamModel(R.config_of(sp), W, device=dev, own_stream=args.exec == "graph")
              for sp, W in ((sv, Wv), (sa, Wa))]
    mv, ma = models
    K = sv.K
    for m in models:
        m.set_option(L.WAM_OPT_ATTENTION, ATTN_VARIANTS[args.attention])
        m.set_option(L.WAM_OPT_DEVICE_DECISION, int(args.exec in ("device", "graph")))
        m.set_option(L.WAM_OPT_GRAPHS, int(args.exec == "graph"))
        m.set_schedule(1.0 - np.arange(K + 1, dtype=np.float64) / K)
    pair = R.IdmPair(mv, ma, sv.No, sv.Co)
    modes = {"auto": L.WAM_RR_AUTO, "force_skip": L.WAM_RR_FORCE_SKIP, "force_full": L.WAM_RR_FORCE_FULL,
             "off": L.WAM_RR_OFF}

    def rrp(sp, mode):
        q, s_, e = sp.rr_bounds
        return R.rr_profile(q, s_, e, mode, sp.rr_alpha_min, sp.rr_alpha_max, sp.rr_eps, sp.rr_gamma_cos,
                            sp.rr_gamma_fit, branches=L.WAM_RR_SINGLE)

    rr = (rrp(sv, modes[args.rr_mode]), rrp(sa, modes[args.rr_mode]))
    n_ctrl = 2 + args.warmup + args.steps  # first, warm-up, attribution and timed replans
    obs = make_observations(sv, n_ctrl)
    rho = sv.ar_rho
    delta = 1.0 / np.sqrt(1.0 - rho * rho)
    obs_d = torch.from_numpy(obs).to(dev)
    pred_d = torch.from_numpy((rho * obs[:-1]).astype(np.float32)).to(dev)
    nf = [torch.from_numpy(make_initial_noise(sp)).to(dev) for sp in (sv, sa)]
    rn = [torch.from_numpy(np.stack([make_remap_noise(sp, t) for t in range(n_ctrl)])).to(dev) for sp in (sv, sa)]
    xv, xa = mv.new_traj(), ma.new_traj()

    def replan(t, rr=rr):
        cr = obs_d[t]
        cp = pred_d[t - 1] if t > 0 else cr
        return pair.replan(
            cr, xv, xa, rn[0][t], rn[1][t],
            video_kw=dict(cond_pred=cp, u_hat=[cp], u=[cr], delta=[delta], weight=[1.0], noise_first=nf[0],
                          rr=rr[0], b0=sv.tr_b0, r=sv.tr_r, shift_action=0, shift_video=sv.shift_video,
                          k1=sv.or_k1, tau=sv.or_tau, kappa_max=sv.or_kappa_max),
            action_kw=dict(noise_first=nf[1], rr=rr[1], b0=sa.tr_b0, r=sa.tr_r, shift_action=sa.shift_action,
                           shift_video=0, k1=0, or_enabled=False))

    t = 0
    replan(t)
    t += 1
    for _ in range(args.warmup):
        replan(t)
        t += 1
    classes = [L.WAM_KC_GEMM_QKV, L.WAM_KC_GEMM_PROJ, L.WAM_KC_GEMM_FC1, L.WAM_KC_GEMM_FC2, L.WAM_KC_ATTENTION]
    for m in models:
        for kc in classes:
            m.profile_enable(kc, True, 4096)
    replan(t)
    t += 1
    tot = {}
    for mi, m in enumerate(models):
        for kc in classes:
            tot[(mi, kc)] = m.profile_read(kc)[0]
            m.profile_enable(kc, False)
    dmod, dom = max(tot, key=tot.get)
    models[dmod].profile_enable(dom, True, 200000)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    infos = []
    for _ in range(args.steps):
        infos.append(replan(t))
        t += 1
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    dom_ms, dom_n, dom_work = models[dmod].profile_read(dom)
    models[dmod].profile_enable(dom, False)

    steps_v = sum(iv.steps for iv, _ in infos)
    steps_a = sum(ia.steps for _, ia in infos)
    flops = sum(sp.flops_per_layer() * sum(i[j].steps * sp.L - i[j].layers_skipped for i in infos)
                for j, sp in enumerate((sv, sa)))
    dom_tflops = dom_work / (dom_ms * 1e-3) / 1e12 if dom_ms > 0 else 0.0

    def reuse(j):
        att = sum(i[j].rr_attempts for i in infos)
        dense = sum(i[j].layers_dense for i in infos)
        st = sum(i[j].n_start for i in infos)
        return {"rr_accept": sum(i[j].rr_reuses for i in infos) / att if att else None,
                "rr_skip_frac": sum(i[j].layers_skipped for i in infos) / dense if dense else None,
                "or_accept": sum(i[j].n_bind for i in infos) / st if st else None}

    name = {0: "video", 1: "action"}
    out = {
        "metric": "denoise steps/s + action chunks/s per MI355X; MFMA % of bf16 peak",
        "value": round((steps_v + steps_a) / elapsed, 3),
        "unit": "denoise steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(1000.0 * elapsed / args.steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if sv.dtype == "bf16" else "f32",
        "data": "synthetic (seeded random-init weights N(0,0.02), N(0,1) noise, AR(1) observations)",
        "config": {
            "workload": (f"{args.workload}: independently executed video / action DiTs, closed-loop replan per "
                         f"model (video: L{sv.L} D{sv.D} T{sv.T}, b0={sv.tr_b0} r={sv.tr_r} prefix {sv.or_k1}+"
                         f"{K - sv.tr_b0 - sv.or_k1}; action: L{sa.L} D{sa.D} T{sa.T} (obs {sv.No} + video "
                         f"{sv.Nv} condition tokens), b0={sa.tr_b0} shift={sa.shift_action}) K{K}, "
                         "single-branch RR per model"),
            "step": "one control step of the pair (video replan, then action replan)",
            "exec": args.exec,
            "attention": args.attention,
        },
        "action_chunks_per_s": round(args.steps / elapsed, 3),
        "denoise_steps_per_replan": {"video": steps_v / args.steps, "action": steps_a / args.steps},
        "mfma_frac_dit": round(flops / elapsed / 1e12 / MFMA_BF16_PEAK_TFLOPS, 5),
        "dit_tflops": round(flops / elapsed / 1e12, 3),
        "reuse_stats": {"video": reuse(0), "action": reuse(1)},
        "roofline": {
            "kernel": f"{name[dmod]} {L.KERNEL_CLASS_NAMES[dom]}",
            "bound": "mfma",
            "achieved": round(dom_tflops, 3),
            "peak": MFMA_BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(dom_tflops / MFMA_BF16_PEAK_TFLOPS, 5),
            "traffic": lookup_traffic(args.workload, L.KERNEL_CLASS_NAMES[dom]),
            "launches": dom_n,
            "avg_launch_us": round(1000.0 * dom_ms / dom_n, 3) if dom_n else None,
            "class_ms_one_replan": {f"{name[mi]} {L.KERNEL_CLASS_NAMES[k]}": round(v, 4)
                                    for (mi, k), v in tot.items()},
        },
    }
    if not args.no_native:
        # full re-denoise of both models: K steps of video from noise, the
        # condition packing, K steps of action
        nrep = max(3, args.steps // 5)
        vv, aa = mv.new_traj(), ma.new_traj()

        def native(i):
            vv.copy_(nf[0])
            mv.continue_(0, K, vv, obs_d[i])
            ma.pack_condition(obs_d[i], sv.No, sv.Co, vv, sv.Nv, sv.Cv, mv.traj, pair.cond_action)
            aa.copy_(nf[1])
            ma.continue_(0, K, aa, pair.cond_action)

        for m in models:
            m.reset_all()
        native(0)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(nrep):
            native(i + 1)
        torch.cuda.synchronize()
        nat = (time.perf_counter() - t0) / nrep
        out["native_chunk_ms"] = round(1000.0 * nat, 4)
        out["native_steps_per_s"] = round(2 * K / nat, 3)
        out["reuse_latency_speedup"] = round(nat / (elapsed / args.steps), 4)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(sv, Wv, obs, args.cpu_sample_steps, single=True)
        out["cpu_baseline"]["sample"] += " (video model of the pair)"
    print(json.dumps(out), flush=True)
    for m in models:
        m.close()


def ablation(args):
    """Closed-loop replans per variant, mirroring the paper's ablation of the
    three mechanisms and graph replay: GPU time per replan (foreground +
    anticipatory, HIP events on the handle's stream) and observation-to-action
    latency (host clock from the real observation to the ready chunk, Eq.
    app-o2a).  The anticipatory prefix is enqueued by wam_replan_begin right
    after the previous chunk and runs during a simulated action window."""
    import numpy as np
    import torch

    from paper_2609_34608_amd import _lib as L
    from paper_2609_34608_amd import runtime as R
    from synth import get_workload, make_weights, make_initial_noise, make_observations, make_remap_noise

    spec = get_workload(args.workload)
    dev = torch.device("cuda:0")
    W = make_weights(spec)
    m = R.WamModel(R.config_of(spec), W, device=dev, own_stream=True)
    K = spec.K
    m.set_schedule(1.0 - np.arange(K + 1) / K)
    q, s_, e = spec.rr_bounds
    n = args.warmup + args.steps + 1
    obs = make_observations(spec, n)
    rho = spec.ar_rho
    delta = 1.0 / np.sqrt(1.0 - rho * rho)
    obs_d = torch.from_numpy(obs).to(dev)
    pred_d = torch.from_numpy((rho * obs[:-1]).astype(np.float32)).to(dev)
    noise_first = torch.from_numpy(make_initial_noise(spec)).to(dev)
    remap_noise = torch.from_numpy(np.stack([make_remap_noise(spec, t) for t in range(n)])).to(dev)
    x_out = m.new_traj()
    k2 = K - spec.tr_b0 - spec.or_k1  # steps under the real condition after an accepted prefix
    variants = [  # name, exec, tr, or, rr mode
        ("native", "host", False, False, L.WAM_RR_OFF),
        ("native+graph", "graph", False, False, L.WAM_RR_OFF),
        ("wamachine", "graph", True, True, L.WAM_RR_AUTO),
        ("w/o TR", "graph", False, True, L.WAM_RR_AUTO),
        ("w/o OR", "graph", True, False, L.WAM_RR_AUTO),
        ("w/o RR", "graph", True, True, L.WAM_RR_OFF),
        ("w/o graph", "host", True, True, L.WAM_RR_AUTO),
    ]
    table = {}
    for name, ex, tr, orb, rrm in variants:
        m.set_option(L.WAM_OPT_GRAPHS, 0)
        m.set_option(L.WAM_OPT_DEVICE_DECISION, int(ex != "host"))
        m.set_option(L.WAM_OPT_GRAPHS, int(ex == "graph"))
        rr = R.rr_profile(q, s_, e, rrm, spec.rr_alpha_min, spec.rr_alpha_max, spec.rr_eps, spec.rr_gamma_cos,
                          spec.rr_gamma_fit)
        # without remapping the replan enters at stage 0; the prefix then covers
        # all steps before the last k2, as the paper's w/o-TR variant keeps the
        # native rebinding stage
        kw = dict(rr=rr, b0=spec.tr_b0 if tr else 0, r=spec.tr_r, shift_action=spec.shift_action,
                  shift_video=spec.shift_video, k1=spec.or_k1 if tr else K - k2, tau=spec.or_tau,
                  kappa_max=spec.or_kappa_max, tr_enabled=tr, or_enabled=orb)
        m.reset_all()
        gpu, o2a, steps, infos = [], [], [], []
        for t in range(n):
            cp = pred_d[t - 1] if t > 0 else obs_d[t]
            a = m.replan_args(obs_d[t], x_out, remap_noise[t], cond_pred=cp, u_hat=[cp], u=[obs_d[t]],
                              delta=[delta], weight=[1.0], noise_first=noise_first, **kw)
            e0, e1, e2, e3 = (torch.cuda.Event(enable_timing=True) for _ in range(4))
            e0.record(m.stream)
            m.replan_begin(a)
            e1.record(m.stream)
            time.sleep(args.window_ms * 1e-3)  # action execution; the prefix runs meanwhile
            t_obs = time.perf_counter()
            e2.record(m.stream)
            info = m.replan_end(a)
            e3.record(m.stream)
            m.stream.synchronize()
            t_ready = time.perf_counter()
            if t > args.warmup:
                gpu.append(e0.elapsed_time(e1) + e2.elapsed_time(e3))
                o2a.append(1000.0 * (t_ready - t_obs))
                steps.append(info.steps)
                infos.append(info)
        n_start = sum(i.n_start for i in infos)
        n_bind = sum(i.n_bind for i in infos)
        att = sum(i.rr_attempts for i in infos)
        table[name] = {"gpu_ms": round(float(np.mean(gpu)), 4), "o2a_ms": round(float(np.mean(o2a)), 4),
                       "steps_per_replan": float(np.mean(steps)),
                       "or_accept": n_bind / n_start if n_start else None,
                       "or_coverage": n_bind / len(infos),
                       "rr_accept": sum(i.rr_reuses for i in infos) / att if att else None}
        print(f"ablation {name}: {table[name]['gpu_ms']:.3f} ms GPU, {table[name]['o2a_ms']:.3f} ms O2A",
              file=sys.stderr, flush=True)
    base = table["native"]
    for v in table.values():
        v["gpu_speedup"] = round(base["gpu_ms"] / v["gpu_ms"], 3)
        v["o2a_speedup"] = round(base["o2a_ms"] / v["o2a_ms"], 3)
    print(json.dumps({"workload": spec.name, "window_ms": args.window_ms, "replans": args.steps,
                      "variants": table}), flush=True)
    m.close()


def rel_l2(a, ref) -> float:
    """||a - ref|| / ||ref|| in float64 (device tensors)."""
    a, ref = a.double(), ref.double()
    return float((a - ref).norm() / ref.norm())


def layer_diagnostics(m, spec, x0, cond, rr_force, n_steps):
    """Layer-state diagnostics along the native trajectory from x0 under cond
    (Eq. app-layer-errors): at step i, Delta_l(i) = ||h_{l+1} - h_l|| / ||h_l||
    for every layer l, and E_out(i) = ||y_reuse - y_full|| / ||y_full||, the
    output of the residual-reuse path (reuse forced, retained state from the
    previous step) against full computation on the same input.  Returns
    (delta [n_steps][L], e_out [n_steps]); step 0 only establishes the
    retained state, so its E_out is that of a full evaluation (0)."""
    x = x0.clone()
    m.reset_layer_state()
    delta, e_out = [], []
    for i in range(n_steps):
        hs = [m.hidden(i, x, cond, n) for n in range(spec.L + 1)]
        delta.append([rel_l2(hs[l + 1], hs[l]) for l in range(spec.L)])
        v_full, _ = m.velocity(i, x, cond)
        v_reuse, _ = m.velocity(i, x, cond, rr=rr_force)
        e_out.append(rel_l2(v_reuse, v_full))
        m.denoise_step(i, x, cond)
    return delta, e_out


def action_part(spec, x):
    """[B, Na, A] action slots of trajectories [B, traj] (video first)."""
    return x[:, spec.Nv * spec.Cv:].reshape(x.shape[0], spec.Na, spec.A)


def diagnostics(args):
    """State-continuity diagnostics of the paper's analysis protocols on the
    synthetic model: layer change and reuse output error along a native
    trajectory; cos and relative L2 of the retained latent x^r between
    consecutive closed-loop replans (Eq. app-trajectory-similarity); action
    RMSE of remapped inference (K - b0 steps, OR and RR off) against native
    inference (K steps) under the same observation and initial noise, both
    continuing from the native replan of the previous observation (Eq.
    app-action-rmse)."""
    import numpy as np
    import torch

    from paper_2609_34608_amd import _lib as L
    from paper_2609_34608_amd import runtime as R
    from synth import get_workload, make_weights, make_initial_noise, make_observations, make_remap_noise

    spec = get_workload(args.workload)
    dev = torch.device("cuda:0")
    W = make_weights(spec)
    m = R.WamModel(R.config_of(spec), W, device=dev)
    K = spec.K
    m.set_schedule(1.0 - np.arange(K + 1) / K)
    q, s_, e = spec.rr_bounds
    rr_kw = (spec.rr_alpha_min, spec.rr_alpha_max, spec.rr_eps, spec.rr_gamma_cos, spec.rr_gamma_fit)
    rr_auto = R.rr_profile(q, s_, e, L.WAM_RR_AUTO, *rr_kw)
    rr_force = R.rr_profile(q, s_, e, L.WAM_RR_FORCE_SKIP, *rr_kw)
    n = max(3, min(args.steps, 8))
    obs = make_observations(spec, n + 1)
    rho = spec.ar_rho
    delta_or = 1.0 / np.sqrt(1.0 - rho * rho)
    obs_d = torch.from_numpy(obs).to(dev)
    pred_d = torch.from_numpy((rho * obs[:-1]).astype(np.float32)).to(dev)
    noise_first = torch.from_numpy(make_initial_noise(spec)).to(dev)
    remap_noise = torch.from_numpy(np.stack([make_remap_noise(spec, t) for t in range(n + 1)])).to(dev)
    ra = dict(b0=spec.tr_b0, r=spec.tr_r, shift_action=spec.shift_action, shift_video=spec.shift_video,
              k1=spec.or_k1, tau=spec.or_tau, kappa_max=spec.or_kappa_max)

    delta, e_out = layer_diagnostics(m, spec, noise_first, obs_d[0], rr_force, K)
    print(f"diagnostics: layer change and output error over {K} steps", file=sys.stderr, flush=True)

    # consecutive closed-loop replans (TR + OR + RR as in the replay workload)
    m.reset_all()
    x_out = m.new_traj()
    cos_r, rel_r, prev = [], [], None
    for t in range(n):
        cp = pred_d[t - 1] if t > 0 else obs_d[t]
        m.replan(obs_d[t], x_out, remap_noise[t], cond_pred=cp, u_hat=[cp], u=[obs_d[t]], delta=[delta_or],
                 weight=[1.0], noise_first=noise_first, rr=rr_auto, **ra)
        _, xr, _ = m.get_replan_state()
        if prev is not None:
            a, b = xr.double().flatten(), prev.double().flatten()
            cos_r.append(float(a.dot(b) / (a.norm() * b.norm())))
            rel_r.append(rel_l2(xr, prev))
        prev = xr.clone()
    print(f"diagnostics: {n} consecutive replans", file=sys.stderr, flush=True)

    # remapped (K - b0 steps) against native (K steps), OR and RR off
    rmse, x_tr, x_nat = [], m.new_traj(), m.new_traj()
    for t in range(1, n):
        m.reset_all()  # the next replan is native (K steps from noise) and leaves the replan state
        m.replan(obs_d[t - 1], x_nat, remap_noise[t - 1], noise_first=noise_first, or_enabled=False, **ra)
        m.replan(obs_d[t], x_tr, remap_noise[t], noise_first=noise_first, or_enabled=False, **ra)
        m.reset_all()
        m.replan(obs_d[t], x_nat, remap_noise[t], noise_first=noise_first, or_enabled=False, **ra)
        d = action_part(spec, x_tr).double() - action_part(spec, x_nat).double()
        rmse.append(float(d.pow(2).mean().sqrt()))
    m.close()
    out = {"diagnostics": spec.name, "data": "synthetic (seeded random-init weights)",
           "layer_change_mean": [round(float(v), 6) for v in np.mean(delta, axis=0)],
           "layer_change_per_step": [[round(v, 6) for v in row] for row in delta],
           "output_error_reuse_vs_full": [round(v, 6) for v in e_out],
           "replan_latent_cos": [round(v, 6) for v in cos_r],
           "replan_latent_rel_l2": [round(v, 6) for v in rel_r],
           "action_rmse_remapped_vs_native": [round(v, 6) for v in rmse],
           "protocol": {"steps": K, "replans": n, "remapped_steps": K - spec.tr_b0, "native_steps": K}}
    print(json.dumps(out), flush=True)


def host_info():
    """Host cores, CPU model and BLAS threads of the machine the oracle runs on."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        from threadpoolctl import threadpool_info
        blas = max((i.get("num_threads", 1) for i in threadpool_info()), default=1)
    except Exception:
        blas = None
    try:
        affinity = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        affinity = None
    return {"host_cpus": os.cpu_count(), "affinity_cpus": affinity, "cpu_model": model, "blas_threads": blas}


def cpu_baseline(spec, W, obs, n_steps, single=False):
    """The float64 oracle on the host: a bounded sample of Euler steps of the
    same model (the continuation of one accepted replan), timed."""
    from oracle import method as OM
    from synth import make_initial_noise
    info = host_info()
    sig = OM.flow_schedule(spec.K)
    q, s, e = spec.rr_bounds
    rr = OM.RRProfile(q, s, e, spec.rr_alpha_min, spec.rr_alpha_max, spec.rr_eps, spec.rr_gamma_cos,
                      spec.rr_gamma_fit, single=single)
    x = make_initial_noise(spec)
    k0 = spec.K - n_steps
    t0 = time.perf_counter()
    OM.denoise(W, spec, x, obs[0], sig, k0, spec.K, rr, OM.LayerState())
    dt = time.perf_counter() - t0
    return {"value": round(n_steps / dt, 5), "unit": "denoise steps/s", "cores": info["blas_threads"],
            "kind": "oracle",
            "sample": f"{n_steps} float64 Euler steps with residual rescaling of the same model "
                      f"(steps {k0}..{spec.K - 1}), {dt:.1f} s", **info}


def cpu_baseline_layer(spec, W):
    """The float64 oracle on the host at the large workload: one DiT layer of
    the model (full sequence, every head, the oracle's serial head loop),
    timed, and scaled to one denoising step of L layers.  The embedding and
    the output heads of a step are under 1% of its work and are left out."""
    import numpy as np
    from oracle import dit as OD
    from synth import make_initial_noise, make_observations
    info = host_info()
    x = make_initial_noise(spec)
    cond = make_observations(spec, 0)[0]
    c = OD.cond_vector(W, 1.0)
    h = OD.embed_tokens(W, spec, x, cond)
    t0 = time.perf_counter()
    h1 = OD.dit_layer(W, spec, 0, h, c)
    dt = time.perf_counter() - t0
    assert np.isfinite(h1).all()
    step_s = dt * spec.L
    return {"value": round(1.0 / step_s, 6), "unit": "denoise steps/s", "cores": info["blas_threads"],
            "kind": "oracle",
            "sample": f"one float64 DiT layer of the {spec.name} model (T={spec.T}, {spec.H} heads), "
                      f"{dt:.1f} s, x {spec.L} layers = {step_s:.0f} s per denoising step; the oracle's "
                      f"matrix products use {info['blas_threads']} BLAS threads, its elementwise work one",
            **info}


if __name__ == "__main__":
    main()
