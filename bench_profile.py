#!/usr/bin/env python3
"""Summarise rocprofv3 runs of ``bench.py`` into the text files under ``profiles/``.

Inputs are the CSV folders rocprofv3 writes:
  --trace DIR   ``rocprofv3 --kernel-trace --stats --output-format csv -d DIR -o kt -- python bench.py ...``
  --fetch DIR   ``rocprofv3 --pmc FETCH_SIZE --output-format csv -d DIR -o f -- python bench.py ... --copy-probe-gib 1``
  --write DIR   the same with ``--pmc WRITE_SIZE``

Writes ``profiles/kernels_<workload>.md`` (per-launch kernel durations, warm-up launches dropped) and,
with the counter runs, ``profiles/traffic_<workload>.json`` + ``.md``: HBM bytes per entry-point
call, calibrated against the plain 1 GiB copy that ``bench.py --copy-probe-gib 1`` runs after timing
(FETCH_SIZE and WRITE_SIZE are in KiB; each is scaled by true bytes / counter bytes of that copy).
The JSON carries the digest of the HIP sources it was measured on; ``bench.py`` reports ``traffic``
only while that digest matches.
"""
from __future__ import annotations

import argparse
import collections
import csv
import glob
import json
import os
import statistics

import bench

ROOT = os.path.dirname(os.path.abspath(__file__))
# kernel-name fragment -> step (first match wins: the aligner's hidden layer inside the Patch step
# before the unfolded aligner timed beside it)
PHASES = {"encode_bf16_kernel": "encode", "reuse_decode": "reuse_decode",
          "patch_kv": "patch", "patch_align_act": "patch", "patch_align": "aligner",
          "patch_fold": "fold", "EncodeKV": "encode", "EncodeH": "encode",
          "ReuseDecode": "reuse_decode", "PatchKV": "patch", "PatchAlign": "patch",
          "fit_gram": "fit_gram", "fit_prep": "fit_solve", "fit_tridiag": "fit_solve",
          "fit_bisect": "fit_solve", "fit_inverse": "fit_solve", "fit_back": "fit_solve",
          "fit_project": "fit_solve", "fit_normal": "fit_solve", "fit_chol": "fit_solve",
          "fit_out": "fit_solve"}


def phase_of(name: str):
    for frag, ph in PHASES.items():
        if frag in name:
            return ph
    return None


def short(name: str) -> str:
    name = name.replace("scd::(anonymous namespace)::", "").replace("(scd::GemmParams)", "")
    return name.replace("void ", "")[:70]


def one_csv(folder: str, suffix: str) -> str:
    found = glob.glob(os.path.join(folder, "**", f"*{suffix}"), recursive=True)
    if not found:
        raise SystemExit(f"no *{suffix} under {folder}")
    return found[0]


def kernel_table(trace_dir: str, warmup_launches: int, aligner_calls: int = 0):
    """Per (kernel, grid) group of codec kernels: launches, mean/min/max microseconds, with the first
    ``warmup_launches`` launches of each group dropped."""
    rows = list(csv.DictReader(open(one_csv(trace_dir, "kernel_trace.csv"))))
    groups = collections.OrderedDict()
    for r in rows:
        if phase_of(r["Kernel_Name"]) is None:
            continue
        grid = r.get("Grid_Size") or r.get("Grid_Size_X") or 0
        # the solve's per-column launches shrink their grids step by step: one row per kernel
        key = (r["Kernel_Name"], 0 if phase_of(r["Kernel_Name"]) == "fit_solve" else int(grid))
        dur = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        groups.setdefault(key, []).append(dur)
    out = []
    for (name, grid), d in groups.items():
        if phase_of(name) == "aligner" and aligner_calls and len(d) == 2 * aligner_calls:
            # both products of the MLP ran on this kernel (two launches per call, possibly with
            # the same grid): split them by their order within the call
            d = d[2 * warmup_launches:] or d
            for i, part in enumerate(("first product", "second product")):
                di = d[i::2]
                if di:
                    out.append({"kernel": f"{short(name)} ({part})", "phase": "aligner",
                                "grid": grid, "launches": len(di), "mean_us": statistics.mean(di),
                                "min_us": min(di), "max_us": max(di)})
            continue
        d = d[warmup_launches:] or d
        out.append({"kernel": short(name), "phase": phase_of(name), "grid": grid, "launches": len(d),
                    "mean_us": statistics.mean(d), "min_us": min(d), "max_us": max(d)})
    return out


def fit_solve_table(trace_dir: str):
    """The fp64 solve's kernels per call: launches and total microseconds per call (a call starts at
    its one `fit_prep_kernel` launch; the first call, a warm-up, is dropped)."""
    rows = sorted(csv.DictReader(open(one_csv(trace_dir, "kernel_trace.csv"))),
                  key=lambda r: int(r["Start_Timestamp"]))
    calls, cur = [], None
    for r in rows:
        name = r["Kernel_Name"]
        if phase_of(name) != "fit_solve":
            continue
        if "fit_prep_kernel" in name:
            cur = {"start": int(r["Start_Timestamp"]), "k": collections.OrderedDict()}
            calls.append(cur)
        if cur is None:
            continue
        k = short(name).replace("(scd::(anonymous namespace)::SolveArgs)", "")
        k = k.replace("(scd::FitSolveParams)", "")
        n, t = cur["k"].get(k, (0, 0.0))
        cur["k"][k] = (n + 1, t + (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
        cur["end"] = int(r["End_Timestamp"])
    calls = [c for c in calls if "end" in c][1:] or calls
    names = list(calls[0]["k"].keys()) if calls else []
    out = []
    for k in names:
        out.append({"kernel": k, "launches": statistics.median(c["k"].get(k, (0, 0))[0] for c in calls),
                    "us": statistics.median(c["k"].get(k, (0, 0.0))[1] for c in calls)})
    wall = statistics.median((c["end"] - c["start"]) / 1e3 for c in calls) if calls else 0.0
    return out, wall, len(calls)


def counters(folder: str, counter: str):
    rows = list(csv.DictReader(open(one_csv(folder, "counter_collection.csv"))))
    return [r for r in rows if r["Counter_Name"] == counter]


def calibration(rows, true_bytes: int) -> float:
    """true bytes / counter bytes of the probe copy (the last three elementwise launches with the
    probe's element count)."""
    probe = [r for r in rows if "elementwise" in r["Kernel_Name"]
             and int(r["Grid_Size"]) * 16 == true_bytes]
    if not probe:
        raise SystemExit("copy probe dispatches not found (run bench.py with --copy-probe-gib 1)")
    kib = statistics.median(float(r["Counter_Value"]) for r in probe[-3:])
    return true_bytes / (kib * 1024.0)


def per_phase_bytes(rows, scale: float):
    """Median counter bytes per (kernel, grid) group, summed per phase (one entry-point call)."""
    groups = collections.defaultdict(list)
    for r in rows:
        ph = phase_of(r["Kernel_Name"])
        if ph is not None:
            groups[(ph, r["Kernel_Name"], r["Grid_Size"])].append(float(r["Counter_Value"]))
    out = collections.defaultdict(float)
    for (ph, _, _), v in groups.items():
        out[ph] += statistics.median(v) * 1024.0 * scale
    return dict(out)


N_XCD, N_SIMD = 8, 256 * 4


def mfma_table(folder: str):
    """Per (kernel, grid): median duration, MFMA flops from SQ_INSTS_VALU_MFMA_MOPS_BF16 (512 flops
    per op), MFMA-busy cycles per SIMD over the kernel's cycles (GRBM_GUI_ACTIVE is summed over the
    XCDs), and the clock those cycles imply."""
    rows = list(csv.DictReader(open(one_csv(folder, "counter_collection.csv"))))
    vals = collections.defaultdict(lambda: collections.defaultdict(list))
    durs = collections.defaultdict(list)
    for r in rows:
        if phase_of(r["Kernel_Name"]) is None:
            continue
        key = (r["Kernel_Name"], int(r["Grid_Size"]))
        vals[key][r["Counter_Name"]].append(float(r["Counter_Value"]))
        durs[key].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    out = []
    for key, cs in vals.items():
        med = {c: statistics.median(v) for c, v in cs.items()}
        dur_us = statistics.median(durs[key])
        cycles = med.get("GRBM_GUI_ACTIVE", 0.0) / N_XCD
        busy = med.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) / N_SIMD
        wave = med.get("SQ_WAVE_CYCLES", 0.0)
        out.append({"kernel": short(key[0]), "phase": phase_of(key[0]), "grid": key[1],
                    "us": dur_us, "gflop": med.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0) * 512 / 1e9,
                    "busy": busy / cycles if cycles else 0.0,
                    "ghz": cycles / (dur_us * 1e3) if dur_us else 0.0,
                    "wait": med.get("SQ_WAIT_ANY", 0.0) / wave if wave else 0.0,
                    "valu": med.get("SQ_ACTIVE_INST_VALU", 0.0) / wave if wave else 0.0})
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--workload", default="llama3_8b_bf16")
    ap.add_argument("--trace")
    ap.add_argument("--trace-cmd", default="")
    ap.add_argument("--warmup-launches", type=int, default=3)
    ap.add_argument("--bench-log", help="log whose first JSON line is the traced bench run's")
    ap.add_argument("--fetch")
    ap.add_argument("--write")
    ap.add_argument("--pmc-cmd", default="")
    ap.add_argument("--probe-gib", type=float, default=1.0)
    ap.add_argument("--mfma", help="rocprofv3 --pmc folder with SQ_VALU_MFMA_BUSY_CYCLES, "
                    "SQ_INSTS_VALU_MFMA_MOPS_BF16, GRBM_GUI_ACTIVE")
    ap.add_argument("--mfma-cmd", default="")
    ap.add_argument("--fit-md", help="also write profiles/fit_solve_<name>.md from --trace (the "
                    "traced run timed the fit at --fit-shape)")
    ap.add_argument("--fit-shape", default="fit_llama3_8b_head_shared_bf16")
    args = ap.parse_args()

    from synth import workloads as W
    wl = {w.name: w for w in (*W.CONFIGS, *W.MODEL_SCALE_EXTRA, *W.TEST_WORKLOADS)}[args.workload]
    alg = dict(bench.algorithmic(wl))
    digest = bench.source_digest()
    os.makedirs(os.path.join(ROOT, "profiles"), exist_ok=True)

    if args.trace:
        aligner_calls = 0
        if args.bench_log:
            for line in open(args.bench_log):
                if line.startswith("{"):
                    rec = json.loads(line)
                    aligner_calls = (rec["steps"] + rec["warmup"]
                                     if "aligner_unfolded" in rec else 0)
                    break
        tab = kernel_table(args.trace, args.warmup_launches, aligner_calls)
        lines = [f"# Codec kernels, {wl.name} (T={wl.n_tokens}, L={wl.n_layers}, d={wl.d_model}, "
                 f"{wl.n_kv_heads}x{wl.head_dim}, r={sorted(set(wl.ranks))}, Patch layers "
                 f"{list(wl.patch_layers)})", "",
                 f"Command: `{args.trace_cmd}`", "",
                 f"Source digest of csrc/: `{digest}`. Durations from the kernel trace, first "
                 f"{args.warmup_launches} launches of each kernel (the warm-up steps) dropped.", "",
                 "| kernel | step | grid (work-items) | launches | mean us | min us | max us |",
                 "|---|---|---|---|---|---|---|"]
        per_phase = collections.defaultdict(float)
        for t in tab:
            lines.append(f"| `{t['kernel']}` | {t['phase']} | {t['grid']} | {t['launches']} | "
                         f"{t['mean_us']:.1f} | {t['min_us']:.1f} | {t['max_us']:.1f} |")
            per_phase[t["phase"]] += t["mean_us"]
        events = {}
        if args.bench_log:
            for line in open(args.bench_log):  # the first JSON line is the traced run's
                if line.startswith("{"):
                    rec = json.loads(line)
                    events = rec.get("phase_ms", {})
                    events = {k: (v["mean"] if isinstance(v, dict) else v)
                              for k, v in events.items()}
                    if "aligner_unfolded" in rec:  # timed beside the step, with its own figures
                        al = rec["aligner_unfolded"]
                        alg["aligner"] = (al["alg_bytes"], al["alg_flops"])
                        events["aligner"] = al["ms_per_call"]
                    break
        lines += ["", "Per entry-point call (sum of its launches) and the algorithmic roofline; "
                  "\"bench events\" is bench.py's own HIP-event time of the same call in the "
                  "same traced run:", "",
                  "| step | us per call | bench events us | algorithmic | achieved | fraction of peak |",
                  "|---|---|---|---|---|---|"]
        for ph, us in per_phase.items():
            if ph not in alg:
                continue
            ev = f"{events[ph] * 1e3:.1f}" if ph in events else "-"
            b, f = alg[ph]
            bound = bench.KERNELS[ph][1] if ph in bench.KERNELS else "mfma"
            if bound == "hbm":
                ach = b / (us * 1e-6) / 1e9
                lines.append(f"| {ph} | {us:.1f} | {ev} | {b / 1e9:.4f} GB | {ach:.0f} GB/s | "
                             f"{ach / bench.HBM_PEAK_GBPS:.3f} of 8 TB/s |")
            else:
                ach = f / (us * 1e-6) / 1e12
                peak = bench.MFMA_PEAK_TFLOPS[wl.dtype]
                lines.append(f"| {ph} | {us:.1f} | {ev} | {f / 1e9:.1f} GFLOP | {ach:.0f} TFLOP/s | "
                             f"{ach / peak:.3f} of {peak:.0f} TFLOP/s |")
        path = os.path.join(ROOT, "profiles", f"kernels_{wl.name}.md")
        open(path, "w").write("\n".join(lines) + "\n")
        print("wrote", path)

    if args.trace and args.fit_md:
        tab, wall, n_calls = fit_solve_table(args.trace)
        lines = [f"# fp64 fit solve kernels, {args.fit_shape}", "",
                 f"Command: `{args.trace_cmd}`", "",
                 f"Source digest of csrc/: `{digest}`. Per call (one branch, every Reuse layer), "
                 f"medians over {n_calls} calls after a warm-up call; kernel times from the trace.",
                 "", "| kernel | launches per call | us per call |", "|---|---|---|"]
        for t in tab:
            lines.append(f"| `{t['kernel']}` | {t['launches']:.0f} | {t['us']:.1f} |")
        lines += ["", f"Sum of kernel time per call: {sum(t['us'] for t in tab):.1f} us; first "
                  f"launch start to last launch end: {wall:.1f} us."]
        path = os.path.join(ROOT, "profiles", f"fit_solve_{args.fit_md}.md")
        open(path, "w").write("\n".join(lines) + "\n")
        print("wrote", path)

    if args.mfma:
        write_mfma(args, wl, alg, digest)

    if args.fetch and args.write:
        true_bytes = int(args.probe_gib * (1 << 30))
        frows, wrows = counters(args.fetch, "FETCH_SIZE"), counters(args.write, "WRITE_SIZE")
        fs, ws = calibration(frows, true_bytes), calibration(wrows, true_bytes)
        fb, wb = per_phase_bytes(frows, fs), per_phase_bytes(wrows, ws)
        steps = {}
        for ph in bench.PHASES:
            if ph in fb and ph in wb:
                tot = fb[ph] + wb[ph]
                steps[ph] = {"fetch_bytes": round(fb[ph]), "write_bytes": round(wb[ph]),
                             "hbm_bytes_per_launch": round(tot),
                             "algorithmic_bytes": alg[ph][0],
                             "ratio_to_algorithmic": round(tot / alg[ph][0], 4)}
        rec = {"workload": wl.name, "source_digest": digest, "command": args.pmc_cmd,
               "calibration": {"probe_bytes": true_bytes, "fetch_scale": round(fs, 4),
                               "write_scale": round(ws, 4)},
               "unit": "bytes per entry-point call (sum of its launches)", "steps": steps}
        jpath = os.path.join(ROOT, "profiles", f"traffic_{wl.name}.json")
        json.dump(rec, open(jpath, "w"), indent=1)
        lines = [f"# HBM traffic per entry-point call, {wl.name}", "",
                 f"Command (one pass per counter): `{args.pmc_cmd}`", "",
                 f"Source digest of csrc/: `{digest}`. Calibration: a plain copy of "
                 f"{true_bytes} bytes reads FETCH_SIZE x {fs:.4f} and WRITE_SIZE x {ws:.4f} of its "
                 f"true bytes; both scales are applied below.", "",
                 "| step | fetch (GB) | write (GB) | total (GB) | algorithmic (GB) | ratio |",
                 "|---|---|---|---|---|---|"]
        for ph, s in steps.items():
            lines.append(f"| {ph} | {s['fetch_bytes'] / 1e9:.4f} | {s['write_bytes'] / 1e9:.4f} | "
                         f"{s['hbm_bytes_per_launch'] / 1e9:.4f} | "
                         f"{s['algorithmic_bytes'] / 1e9:.4f} | {s['ratio_to_algorithmic']:.3f} |")
        open(os.path.join(ROOT, "profiles", f"traffic_{wl.name}.md"), "w").write(
            "\n".join(lines) + "\n")
        print("wrote", jpath)


def write_mfma(args, wl, alg, digest):
    rows = mfma_table(args.mfma)
    lines = [f"# MFMA counters per kernel, {wl.name}", "",
             f"Command: `{args.mfma_cmd}`", "",
             f"Source digest of csrc/: `{digest}`. Medians over the run's launches.",
             "- `SQ_INSTS_VALU_MFMA_MOPS_BF16` counts MFMA work in units of 512 flops: the flop "
             "column checks the algorithmic count.",
             "- MFMA busy = `SQ_VALU_MFMA_BUSY_CYCLES` per SIMD (1024 SIMDs) over the kernel's "
             "cycles (`GRBM_GUI_ACTIVE` over 8 XCDs).",
             "- The clock is those cycles over the kernel's duration; the 2.5 PFLOP/s bf16 peak "
             "assumes 2.4 GHz.",
             "- Waiting and VALU issue are `SQ_WAIT_ANY` and `SQ_ACTIVE_INST_VALU` over "
             "`SQ_WAVE_CYCLES` (fractions of the waves' lifetimes).", "",
             "| kernel | step | grid | us | MFMA GFLOP | MFMA busy | clock GHz | flops / peak at 2.4 GHz | flops / peak at that clock | waves waiting | waves issuing VALU |",
             "|---|---|---|---|---|---|---|---|---|---|---|"]
    for r in rows:
        pk = 2500.0e12 * r["us"] * 1e-6
        frac = r["gflop"] * 1e9 / pk if pk else 0.0
        frac_clk = frac * 2.4 / r["ghz"] if r["ghz"] else 0.0
        lines.append(f"| `{r['kernel']}` | {r['phase']} | {r['grid']} | {r['us']:.1f} | "
                     f"{r['gflop']:.1f} | {r['busy']:.3f} | {r['ghz']:.2f} | {frac:.3f} | "
                     f"{frac_clk:.3f} | {r['wait']:.2f} | {r['valu']:.2f} |")
    if "patch" in alg:
        lines += ["", f"Algorithmic Patch flops per call: {alg['patch'][1] / 1e9:.1f} GFLOP "
                  f"(hidden layer {alg['patch_act'][1] / 1e9:.1f}, folded product "
                  f"{alg['patch_gemm'][1] / 1e9:.1f})."]
    path = os.path.join(ROOT, "profiles", f"mfma_{wl.name}.md")
    open(path, "w").write("\n".join(lines) + "\n")
    print("wrote", path)


if __name__ == "__main__":
    main()
