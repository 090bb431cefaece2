#!/usr/bin/env python3
"""Throughput of the SCD KV-state codec's hot path on one MI355X.

One step is one pass of the whole path over one batch already resident in HBM:
  producer encode    scd_encode        K/V of every Reuse layer -> codes, H of every Patch layer -> Z_H
  consumer Reuse     scd_reuse_decode  codes -> K (RoPE) / V straight into the consumer's KV cache
  consumer Patch     scd_patch_kv      H_hat -> K (RoPE) / V through the consumer's W_K / W_V
The Reuse decode consumes the codes the encode of the same step produced.

Prints one JSON line.  ``value`` is reconstructed-KV GB/s over the whole step (KV bytes written by
Reuse + Patch divided by the full step time, encode included), ``tokens_per_s`` the prefix tokens
per second, both from K uninstrumented steps.  ``roofline`` is the dominant kernel's achieved
fraction of its bound, from a second pass of K steps with HIP events between the entry points on
the stream the kernels run on; ``cpu_baseline`` is the fp64 oracle timed on this host.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}


def algorithmic(wl):
    """Minimum bytes and flops of each step for workload ``wl`` (read every input once, write every
    output once; the RoPE table and re-reads are not counted)."""
    eb, T, D, d, w, g = wl.elem_bytes, wl.n_tokens, wl.kv_width, wl.d_model, wl.w, wl.g
    dec_b = dec_f = pat_b = pat_f = enc_b = enc_f = 0
    for l in range(wl.n_layers):
        if wl.is_patch[l]:
            r = wl.rank(l, "h")
            pat_b += (T * d + 2 * D * d + 2 * T * D + (2 * D if wl.with_bias else 0)) * eb
            pat_f += 2 * T * d * 2 * D
            enc_b += (T * d + r * d + T * r) * eb
            enc_f += 2 * T * d * r
        else:
            mu = w if wl.with_mu else 0
            for br in ("k", "v"):
                r = wl.rank(l, br)
                dec_b += (T * g * r + w * r + mu + T * D) * eb
                dec_f += 2 * T * g * r * w
                enc_b += (T * D + r * w + mu + T * g * r) * eb
                enc_f += 2 * T * g * w * r
    kv_bytes = wl.n_layers * 2 * T * D * eb
    return {"reuse_decode": (dec_b, dec_f), "patch_kv": (pat_b, pat_f),
            "encode": (enc_b, enc_f), "kv_bytes": kv_bytes}


KERNELS = {  # step -> (kernel symbol of the bf16 path, bound)
    "encode": ("encode_bf16_kernel", "hbm"),
    "reuse_decode": ("reuse_decode_bf16_kernel", "hbm"),
    "patch_kv": ("patch_kv_bf16_kernel", "mfma"),
}


def source_digest() -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2606_07684_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode() + f.read())
    return h.hexdigest()[:16]


def traffic_for(workload: str, step: str, digest: str):
    """HBM bytes per launch from committed counter runs, if they were taken on this source."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("source_digest") != digest:
        return None
    ent = rec.get("steps", {}).get(step)
    return None if ent is None else ent.get("hbm_bytes_per_launch")


def cpu_baseline(wl, inp, budget_s=25.0):
    """The fp64 oracle on this host's cores over the same workload, layer by layer; stops after
    ``budget_s`` seconds of oracle time and extrapolates per layer kind."""
    import numpy as np
    import torch

    from oracle import scd_oracle as O

    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # noqa: BLE001
        threads = None
    cores = len(os.sched_getaffinity(0))
    pos = O.positions(wl.cu_seqlens, wl.pos0)
    H, dh, th, D = wl.n_kv_heads, wl.head_dim, wl.rope_theta, wl.kv_width
    f64 = lambda t: None if t is None else t.detach().to("cpu", torch.float64).numpy()  # noqa: E731
    t_reuse, n_reuse, t_patch, n_patch = 0.0, 0, 0.0, 0
    # interleave layer kinds so a budget cut still samples both
    order = sorted(range(wl.n_layers), key=lambda l: (0 if wl.is_patch[l] else 1, l))
    patch_layers = [l for l in order if wl.is_patch[l]]
    reuse_layers = [l for l in order if not wl.is_patch[l]]
    seq = []
    while patch_layers or reuse_layers:
        if patch_layers:
            seq.append(patch_layers.pop(0))
        for _ in range(7):
            if reuse_layers:
                seq.append(reuse_layers.pop(0))
    for l in seq:
        if t_reuse + t_patch > budget_s:
            break
        if wl.is_patch[l]:
            hin, eh, hh, wk, wv = (f64(inp.h_in[l]), f64(inp.w_enc_h[l]), f64(inp.h_hat[l]),
                                   f64(inp.w_k[l]), f64(inp.w_v[l]))
            t0 = time.perf_counter()
            O.encode_h(hin, eh)
            O.patch_k(hh, wk, f64(inp.b_k[l]), pos, H, dh, th)
            O.patch_v(hh, wv, f64(inp.b_v[l]))
            t_patch += time.perf_counter() - t0
            n_patch += 1
        else:
            ka, va = f64(inp.k_in[l]), f64(inp.v_in[l])
            ek, ev, fk, fv = (f64(inp.w_enc_k[l]), f64(inp.w_enc_v[l]), f64(inp.w_dec_k[l]),
                              f64(inp.w_dec_v[l]))
            mk, mv = f64(inp.mu_k[l]), f64(inp.mu_v[l])
            t0 = time.perf_counter()
            zk = O.encode_k(ka, pos, ek, mk, H, dh, th)
            zv = O.encode_v(va, ev, mv)
            O.decode_k(zk, fk, mk, pos, H, dh, th)
            O.decode_v(zv, fv, mv, D)
            t_reuse += time.perf_counter() - t0
            n_reuse += 1
    n_r_all = sum(1 for p in wl.is_patch if not p)
    n_p_all = sum(1 for p in wl.is_patch if p)
    est = (t_reuse / max(n_reuse, 1)) * n_r_all + (t_patch / max(n_patch, 1)) * n_p_all
    kv = algorithmic(wl)["kv_bytes"]
    return {
        "value": round(kv / est / 1e9, 4), "unit": "GB/s", "cores": threads or cores,
        "host_cpus": cores, "kind": "oracle",
        "sample": (f"fp64 numpy oracle, full step of encode + Reuse decode + Patch over "
                   f"{n_reuse}/{n_r_all} Reuse and {n_patch}/{n_p_all} Patch layers at "
                   f"T={wl.n_tokens} (timed {t_reuse + t_patch:.1f} s), extrapolated per layer "
                   f"kind to the whole step; inputs converted to fp64 outside the timed region"),
        "est_step_s": round(est, 3),
    }


def time_aligner(wl, dev, steps, warmup, stream):
    """``scd_patch_align`` over every Patch layer (hidden width = the workload's), HIP events on
    the stream it runs on; algorithmic flops 2T(r_H h + h d) and bytes of every operand read and
    every result written once (the activations are written and read back once)."""
    import torch

    import paper_2606_07684_amd as scd
    from synth import workloads as W

    L, T, h, d = wl.n_layers, wl.n_tokens, wl.hidden_width, wl.d_model
    z_h, w1, b1, w2, b2, act, hh = ([None] * L for _ in range(7))
    flops = nbytes = 0
    for l in range(L):
        if not wl.is_patch[l]:
            continue
        r = wl.rank(l, "h")
        z_h[l] = W.patch_codes(wl, l, dev)
        w1[l], b1[l], w2[l], b2[l] = W.aligner_weights(wl, l, dev)
        act[l] = torch.empty((T, h), dtype=wl.torch_dtype, device=dev)
        hh[l] = torch.empty((T, d), dtype=wl.torch_dtype, device=dev)
        flops += 2 * T * (r * h + h * d)
        nbytes += (T * r + h * r + h + 2 * T * h + d * h + d + T * d) * wl.elem_bytes
    model = scd.Model(n_layers=L, d_model=d, n_kv_heads=wl.n_kv_heads, head_dim=wl.head_dim,
                      rope_theta=wl.rope_theta, dtype=wl.dtype, is_patch=wl.is_patch,
                      rank_k=wl.ranks, rank_v=wl.rank_v, rank_h=wl.ranks, basis_width=wl.w)
    cu = W.cu_seqlens(wl, dev) if wl.n_seqs > 1 or wl.pos0 is not None else None
    batch = scd.Batch(n_tokens=T, cu_seqlens=cu, pos0=W.pos0(wl, dev))
    run = scd.prepare_patch_align(model, batch, h, z_h, w1, b1, w2, b2, act, hh)
    for _ in range(warmup):
        run(stream)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ev[0].record(stream)
    for _ in range(steps):
        run(stream)
    ev[1].record(stream)
    torch.cuda.synchronize()
    ms = ev[0].elapsed_time(ev[1]) / steps
    ach = flops / (ms * 1e-3) / 1e12
    peak = MFMA_PEAK_TFLOPS[wl.dtype]
    return {"kernel": "patch_align_bf16_kernel", "hidden": h, "ms_per_call": round(ms, 4),
            "bound": "mfma", "achieved": round(ach, 2), "peak": peak, "unit": "TFLOP/s",
            "frac": round(ach / peak, 4), "alg_flops": flops, "alg_bytes": nbytes}


def time_fit(dev, steps, warmup, stream):
    """The offline Reuse fit at the Llama-3-8B shape with the head-shared basis (w = d_h = 128:
    8192 tokens x 8 heads = 65,536 calibration rows per layer, 28 Reuse layers): ``scd_fit_gram``
    and ``scd_fit_solve`` for keys and values, HIP events on the stream they run on.  The Gram is
    HBM-bound (2w = 256 columns: about 128 flops per byte of the symmetric product); algorithmic
    bytes read both caches once and write the Gram and column sums once.  The solve is the
    O(w^3) fp64 step, one workgroup per layer, reported as time per call."""
    import torch

    import paper_2606_07684_amd as scd
    from synth import workloads as W

    wl = W.FIT_LLAMA3_8B
    L, T, D, w, g = wl.n_layers, wl.n_tokens, wl.kv_width, wl.w, wl.g
    R = [l for l in range(L) if not wl.is_patch[l]]
    model = scd.Model(n_layers=L, d_model=wl.d_model, n_kv_heads=wl.n_kv_heads,
                      head_dim=wl.head_dim, rope_theta=wl.rope_theta, dtype=wl.dtype,
                      is_patch=wl.is_patch, rank_k=wl.ranks, rank_v=wl.rank_v, rank_h=wl.ranks,
                      basis_width=w)
    batch = scd.Batch(n_tokens=T)
    rope = scd.scd_rope_table(model, wl.max_position)
    ws = torch.empty(scd.scd_fit_workspace_bytes(model, T), dtype=torch.uint8, device=dev)
    n2 = 2 * w
    grams, solves = [], []
    keep = []  # every tensor the prepared calls point to stays alive until the timing ends
    for br, code in (("k", scd.FIT_KEYS), ("v", scd.FIT_VALUES)):
        a_in, b_in, gram, colsum, w_enc, w_dec, mu_e, mu_d = ([None] * L for _ in range(8))
        keep.append((a_in, b_in, gram, colsum, w_enc, w_dec, mu_e, mu_d))
        ranks = wl.ranks if br == "k" else wl.rank_v
        for l in R:
            a_in[l], b_in[l] = W.fit_pair(wl, l, br, dev)
            gram[l] = torch.empty((n2, n2), dtype=torch.float32, device=dev)
            colsum[l] = torch.empty((n2,), dtype=torch.float32, device=dev)
            w_enc[l] = torch.empty((ranks[l], w), dtype=wl.torch_dtype, device=dev)
            w_dec[l] = torch.empty((w, ranks[l]), dtype=wl.torch_dtype, device=dev)
            mu_e[l] = torch.empty((w,), dtype=wl.torch_dtype, device=dev)
            mu_d[l] = torch.empty((w,), dtype=wl.torch_dtype, device=dev)
        grams.append(scd.prepare_fit_gram(model, batch, rope if br == "k" else None, code, a_in,
                                          b_in, gram, colsum, ws))
        solves.append(scd.prepare_fit_solve(model, code, T * g, 0.05 * T * g, True, gram, colsum,
                                            w_enc, w_dec, mu_e, mu_d, ws))
    torch.cuda.synchronize()

    def timed(calls, n, nw):
        for _ in range(nw):
            for c in calls:
                c(stream)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ev[0].record(stream)
        for _ in range(n):
            for c in calls:
                c(stream)
        ev[1].record(stream)
        torch.cuda.synchronize()
        return ev[0].elapsed_time(ev[1]) / n

    gram_k = timed(grams[:1], steps, warmup)
    gram_v = timed(grams[1:], steps, warmup)
    gram_ms = gram_k + gram_v
    solve_ms = timed(solves, max(1, steps // 4), 1)
    nbytes = 2 * len(R) * (2 * T * D * wl.elem_bytes + (n2 * n2 + n2) * 4)  # both branches
    flops = 2 * len(R) * (T * g) * n2 * (n2 + 1)  # symmetric X^T X
    ach = nbytes / (gram_ms * 1e-3) / 1e9
    return {"config": {"workload": wl.name, "n_tokens": T, "rows_per_layer": T * g,
                       "basis_width": w, "reuse_layers": len(R), "rank_k": wl.ranks[R[0]],
                       "rank_v": wl.rank_v[R[0]]},
            "gram": {"kernel": "fit_gram_bf16_kernel", "ms_per_call": round(gram_ms / 2, 4),
                     "ms_keys": round(gram_k, 4), "ms_values": round(gram_v, 4),
                     "calls": 2, "bound": "hbm", "achieved": round(ach, 2),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBPS, 4),
                     "alg_bytes": nbytes, "alg_flops": flops,
                     "tflops": round(flops / (gram_ms * 1e-3) / 1e12, 2)},
            "solve": {"kernel": "fit_solve_kernel", "ms_per_call": round(solve_ms / 2, 3),
                      "calls": 2, "layers_per_call": len(R)}}


def time_receive(wl, dev, steps, warmup, stream, model, batch, rope, inp, z_k, z_v, z_h,
                 k_cache, v_cache):
    """The consumer's receipt of the packed payload from pinned host memory (PCIe-inclusive;
    reported beside the step, never as ``value``): the plain host-to-device copy of the whole
    payload, the copy followed by the one-call decode, and ``scd_reuse_decode_streamed`` (copy by
    layer groups on a side stream, each group decoded as it lands) for several group sizes.  HIP
    events on ``stream``, which every variant ends on."""
    import torch

    import paper_2606_07684_amd as scd

    L, T = wl.n_layers, wl.n_tokens
    total, _ = scd.scd_payload_bytes(model, T)
    staged = torch.empty(total, dtype=torch.uint8, device=dev)
    pz_k, pz_v, pz_h = scd.scd_payload_views(model, T, staged)
    for l in range(L):  # this step's codes, packed
        for dst, src in ((pz_k, z_k), (pz_v, z_v), (pz_h, z_h)):
            if dst[l] is not None:
                dst[l].copy_(src[l])
    host = torch.empty(total, dtype=torch.uint8, pin_memory=True)
    host.copy_(staged)
    dst = torch.empty_like(staged)
    copy_stream = torch.cuda.Stream(device=dev)

    def timed(fn):
        for _ in range(warmup):
            fn()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ev[0].record(stream)
        for _ in range(steps):
            fn()
        ev[1].record(stream)
        torch.cuda.synchronize()
        return ev[0].elapsed_time(ev[1]) / steps

    def copy_only():
        with torch.cuda.stream(stream):
            dst.copy_(host, non_blocking=True)

    def receipt(group, side):
        return scd.prepare_reuse_decode_streamed(model, batch, rope, host, dst, group,
                                                 inp.w_dec_k, inp.w_dec_v, inp.mu_k, inp.mu_v,
                                                 k_cache, v_cache), (copy_stream if side else stream)

    copy_ms = timed(copy_only)
    serial, cs = receipt(L, False)
    serial_ms = timed(lambda: serial(cs, stream))
    by_group = {}
    for group in sorted({1, 2, 4, 8, 16, scd.DEFAULT_LAYERS_PER_GROUP}):
        if group > L:
            continue
        run, cs = receipt(group, True)
        by_group[group] = timed(lambda: run(cs, stream))
    default = by_group[min(scd.DEFAULT_LAYERS_PER_GROUP, L)] if by_group else serial_ms
    reuse_kv = sum(2 * T * wl.kv_width * wl.elem_bytes for l in range(L) if not wl.is_patch[l])
    del staged, host, dst
    return {"source": "pinned host memory", "payload_bytes": total,
            "layers_per_group": scd.DEFAULT_LAYERS_PER_GROUP,
            "copy_ms": round(copy_ms, 4), "h2d_GBps": round(total / (copy_ms * 1e-3) / 1e9, 2),
            "copy_then_decode_ms": round(serial_ms, 4), "streamed_ms": round(default, 4),
            "streamed_ms_by_group": {str(k): round(v, 4) for k, v in by_group.items()},
            "reuse_kv_GBps_pcie_inclusive": round(reuse_kv / (default * 1e-3) / 1e9, 2)}


def copy_ceiling(dev, gib=1.0, reps=10):
    """Attainable HBM bandwidth on this GPU: a plain device-to-device copy of ``gib`` GiB (read +
    write bytes over time), timed with HIP events on the current stream."""
    import torch

    n = int(gib * (1 << 30)) // 4
    src = torch.empty(n, dtype=torch.float32, device=dev).uniform_()
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(reps):
        dst.copy_(src)
    end.record()
    torch.cuda.synchronize()
    gbps = 2 * n * 4 * reps / (start.elapsed_time(end) * 1e-3) / 1e9
    del src, dst
    torch.cuda.empty_cache()
    return gbps


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="llama3_8b_bf16")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-receive", action="store_true",
                    help="skip the receipt timing (its decode launches share the step's kernel "
                         "and grid, so kernel traces of the step leave it out)")
    ap.add_argument("--no-fit", action="store_true",
                    help="skip the offline fit timing (it runs after the step's timing)")
    ap.add_argument("--copy-probe-gib", type=float, default=0.0,
                    help="after timing, run a plain copy of this many GiB (counter calibration)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the codec is measured on one MI355X and is not "
              f"sharded (asked for --gpus {args.gpus})", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2606_07684_amd as scd
    from synth import workloads as W

    wl = {w.name: w for w in (*W.CONFIGS, *W.MODEL_SCALE_EXTRA, *W.TEST_WORKLOADS)}[args.workload]
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    scd.load_library()
    print(f"[bench] building inputs for {wl.name} (T={wl.n_tokens}, L={wl.n_layers})",
          file=sys.stderr, flush=True)

    inp = W.Inputs(wl, dev, decode=False)  # the decode consumes this step's encoded codes
    model = scd.Model(n_layers=wl.n_layers, d_model=wl.d_model, n_kv_heads=wl.n_kv_heads,
                      head_dim=wl.head_dim, rope_theta=wl.rope_theta, dtype=wl.dtype,
                      is_patch=wl.is_patch, rank_k=wl.ranks, rank_v=wl.rank_v, rank_h=wl.ranks,
                      basis_width=wl.w)
    cu = W.cu_seqlens(wl, dev) if wl.n_seqs > 1 or wl.pos0 is not None else None
    batch = scd.Batch(n_tokens=wl.n_tokens, cu_seqlens=cu, pos0=W.pos0(wl, dev))
    rope = scd.scd_rope_table(model, wl.max_position)
    z_k, z_v, z_h = W.alloc_codes(wl, dev)
    k_cache, v_cache = W.alloc_caches(wl, dev)
    enc = scd.prepare_encode(model, batch, rope, inp.k_in, inp.v_in, inp.h_in, inp.w_enc_k,
                             inp.w_enc_v, inp.w_enc_h, inp.mu_k, inp.mu_v, z_k, z_v, z_h)
    dec = scd.prepare_reuse_decode(model, batch, rope, z_k, z_v, inp.w_dec_k, inp.w_dec_v,
                                   inp.mu_k, inp.mu_v, k_cache, v_cache)
    pat = scd.prepare_patch_kv(model, batch, rope, inp.h_hat, inp.w_k, inp.w_v, inp.b_k,
                               inp.b_v, k_cache, v_cache)
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        enc(stream)
        if ev is not None:
            ev[1].record(stream)
        dec(stream)
        if ev is not None:
            ev[2].record(stream)
        pat(stream)
        if ev is not None:
            ev[3].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    print("[bench] warmup done", file=sys.stderr, flush=True)

    # the headline: K whole steps back to back, bracketed by synchronizations, no instrumentation
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    print("[bench] timed steps done", file=sys.stderr, flush=True)
    # per-step breakdown: the same steps again, with HIP events between the entry points
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    for i in range(args.steps):
        step(events[i])
    torch.cuda.synchronize()

    phase = {"encode": [], "reuse_decode": [], "patch_kv": []}
    for ev in events:
        phase["encode"].append(ev[0].elapsed_time(ev[1]))
        phase["reuse_decode"].append(ev[1].elapsed_time(ev[2]))
        phase["patch_kv"].append(ev[2].elapsed_time(ev[3]))
    mean = {k: sum(v) / len(v) for k, v in phase.items()}

    alg = algorithmic(wl)
    ms_per_step = wall * 1e3 / args.steps
    kv = alg["kv_bytes"]
    digest = source_digest()
    rooflines = {}
    for k, (sym, bound) in KERNELS.items():
        b, f = alg[k]
        t = mean[k] * 1e-3
        if bound == "hbm":
            ach, peak, unit = b / t / 1e9, HBM_PEAK_GBPS, "GB/s"
        else:
            ach, peak, unit = f / t / 1e12, MFMA_PEAK_TFLOPS[wl.dtype], "TFLOP/s"
        rooflines[k] = {"kernel": sym, "bound": bound, "achieved": round(ach, 2),
                        "peak": peak, "unit": unit, "frac": round(ach / peak, 4),
                        "traffic": traffic_for(wl.name, k, digest),
                        "ms_per_launch": round(mean[k], 4), "alg_bytes": b, "alg_flops": f}
    dominant = max(mean, key=mean.get)
    dom = rooflines[dominant]

    out = {
        "metric": "reconstructed KV GB/s & tokens/s (Reuse+Patch decode); % of HBM roofline",
        "value": round(kv / (ms_per_step * 1e-3) / 1e9, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic (seeded, model-shaped; no weights or datasets)",
        "config": {"workload": wl.name, "n_layers": wl.n_layers, "d_model": wl.d_model,
                   "n_kv_heads": wl.n_kv_heads, "head_dim": wl.head_dim,
                   "n_tokens": wl.n_tokens, "n_requests": wl.n_seqs,
                   "ranks": sorted(set(wl.ranks)), "ranks_v": sorted(set(wl.rank_v)),
                   "patch_layers": list(wl.patch_layers),
                   "basis_width": wl.w, "rope_theta": wl.rope_theta},
        "tokens_per_s": round(wl.n_tokens / (ms_per_step * 1e-3), 1),
        "phase_ms": {k: round(v, 4) for k, v in mean.items()},
        "decode_patch_GBps": round(kv / ((mean["reuse_decode"] + mean["patch_kv"]) * 1e-3) / 1e9,
                                   2),
        "roofline": {k: dom[k] for k in ("bound", "achieved", "peak", "unit", "frac", "traffic")},
        "roofline_kernel": dom["kernel"],
        "rooflines": rooflines,
        "source_digest": digest,
    }

    # The Patch aligner (Eq. aligner, the row after the hot path): timed on its own over the same
    # step count, reported beside the step and not part of ``value``.
    if any(wl.is_patch):
        print("[bench] timing the aligner", file=sys.stderr, flush=True)
        out["aligner"] = time_aligner(wl, dev, args.steps, args.warmup, stream)

    # The consumer's receipt from host memory (PCIe-inclusive), beside the step.
    if not args.no_receive:
        print("[bench] timing the streamed receipt", file=sys.stderr, flush=True)
        out["receive"] = time_receive(wl, dev, args.steps, args.warmup, stream, model, batch, rope,
                                      inp, z_k, z_v, z_h, k_cache, v_cache)

    # The offline Reuse fit (Section 4.3.1), at the head-shared calibration shape, beside the step.
    if not args.no_fit:
        print("[bench] timing the offline fit", file=sys.stderr, flush=True)
        out["fit"] = time_fit(dev, args.steps, args.warmup, stream)

    # The combined readings of the decode-side target (Reuse decode + Patch at this workload):
    #   reuse_hbm_frac:   Reuse algorithmic bytes / t_reuse / 8 TB/s
    #   patch_mfma_frac:  Patch flops / t_patch / 2.5 PFLOP/s
    #   roofline_time_frac: (t_HBM(Reuse) + t_MFMA(Patch)) / (t_reuse + t_patch), the fraction of the
    #                     serial roofline time the two steps achieve together
    #   literal_hbm_frac: (Reuse + Patch algorithmic bytes) / (t_reuse + t_patch) / 8 TB/s
    # and the same decode and copy rates against a plain device copy timed in this run.
    t_r, t_p = mean["reuse_decode"] * 1e-3, mean["patch_kv"] * 1e-3
    b_r, b_p = alg["reuse_decode"][0], alg["patch_kv"][0]
    f_p = alg["patch_kv"][1]
    peak_flops = MFMA_PEAK_TFLOPS[wl.dtype] * 1e12
    copy_gbps = copy_ceiling(dev)
    out["decode_readings"] = {
        "reuse_hbm_frac": round(b_r / t_r / (HBM_PEAK_GBPS * 1e9), 4),
        "patch_mfma_frac": round(f_p / t_p / peak_flops, 4),
        "roofline_time_frac": round((b_r / (HBM_PEAK_GBPS * 1e9) + f_p / peak_flops) / (t_r + t_p),
                                    4),
        "literal_hbm_frac": round((b_r + b_p) / (t_r + t_p) / (HBM_PEAK_GBPS * 1e9), 4),
        "copy_ceiling_GBps": round(copy_gbps, 1),
        "reuse_frac_of_copy_ceiling": round(b_r / t_r / 1e9 / copy_gbps, 4),
    }

    if args.copy_probe_gib > 0:
        n = int(args.copy_probe_gib * (1 << 30)) // 4
        src = torch.empty(n, dtype=torch.float32, device=dev).uniform_()
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        out["copy_probe_bytes"] = {"read": n * 4, "write": n * 4}
        del src, dst

    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle baseline", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(wl, inp)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
