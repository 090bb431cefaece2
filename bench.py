#!/usr/bin/env python3
"""Throughput of the SCD KV-state codec's hot path on one MI355X.

One step is one pass of the whole path over one batch already resident in HBM:
  producer encode    scd_encode               K/V of every Reuse layer -> codes, H of every
                                              Patch layer -> Z_H
  consumer Reuse     scd_reuse_decode         codes -> K (RoPE) / V straight into the KV cache
  consumer Patch     scd_patch_kv_from_codes  Z_H -> aligner hidden layer -> K (RoPE) / V through
                                              the aligner's output layer folded into W_K / W_V
The consumer half consumes the codes the encode of the same step produced.  The fold of the
aligner's output layer into the projections is weights-only and runs once before timing.

Prints one JSON line.  ``value`` is reconstructed-KV GB/s: the KV bytes Reuse + Patch write divided
by the consumer's time (Reuse decode + Patch), from HIP events recorded between the entry points on
the stream they run on inside the K timed steps.  An event recorded between two launches leaves the
GPU idle for about 5 us, so the consumer span is taken on the odd steps, which record no event
between the decode and Patch calls, and the per-phase split on the even steps, which do.
``ms_per_step`` is the whole step (encode included) by wall clock around those K steps, and
``whole_step_GBps`` the same bytes over it.
``roofline`` is the dominant phase's achieved fraction of its bound; ``configs`` repeats the
measurement for every model-shaped workload; ``cpu_baseline`` is the fp64 oracle on this host.
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
    """Minimum bytes and flops of each phase for workload ``wl`` (read every input once, write every
    output once; the RoPE table and re-reads are not counted).  The Patch phase from the codes is
    the aligner's hidden layer act = SiLU(Z_H W1^T + b1) (written once) and the folded product
    act W_fold^T + c into the K/V cache (act read once)."""
    eb, T, D, d, w, g = wl.elem_bytes, wl.n_tokens, wl.kv_width, wl.d_model, wl.w, wl.g
    h = wl.hidden_width
    dec_b = dec_f = pat_b = pat_f = enc_b = enc_f = act_b = act_f = 0
    for l in range(wl.n_layers):
        if wl.is_patch[l]:
            r = wl.rank(l, "h")
            act_b += (T * r + h * r + h + T * h) * eb
            act_f += 2 * T * r * h
            pat_b += (T * h + 2 * D * h + 2 * D + 2 * T * D) * eb
            pat_f += 2 * T * h * 2 * D
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
    return {"reuse_decode": (dec_b, dec_f), "patch": (act_b + pat_b, act_f + pat_f),
            "patch_act": (act_b, act_f), "patch_gemm": (pat_b, pat_f),
            "encode": (enc_b, enc_f), "kv_bytes": kv_bytes}


PHASES = ("encode", "reuse_decode", "patch")
KERNELS = {  # phase -> (kernel symbols of the bf16 path, bound)
    "encode": ("encode_bf16_kernel", "hbm"),
    "reuse_decode": ("reuse_decode_bf16_kernel", "hbm"),
    "patch": ("patch_align_act_bf16_kernel + patch_kv_bf16_kernel", "mfma"),
}


def pct(vals, q):
    """The q-th percentile (linear interpolation) of a list."""
    v = sorted(vals)
    if len(v) == 1:
        return v[0]
    x = (len(v) - 1) * q / 100.0
    i = int(x)
    j = min(i + 1, len(v) - 1)
    return v[i] + (v[j] - v[i]) * (x - i)


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


def cpu_baseline(wl, inp, aligner, budget_s=25.0, max_tokens=None):
    """The fp64 oracle on this host's cores over the same workload, layer by layer: the consumer's
    Reuse decode and Patch from the codes (the literal aligner, then W_K / W_V), each on the codes
    the oracle's own encode produced.  Stops after ``budget_s`` seconds of oracle time and
    extrapolates per layer kind; the encode is timed too but not counted in ``value``.  With
    ``max_tokens`` the oracle runs on the first that many packed tokens (every map is row-wise, so
    its cost is linear in the token count) and the time is scaled to the whole batch."""
    import torch

    from oracle import scd_oracle as O

    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # noqa: BLE001
        threads = None
    cores = len(os.sched_getaffinity(0))
    S = wl.n_tokens if max_tokens is None else min(wl.n_tokens, max_tokens)
    pos = O.positions(wl.cu_seqlens, wl.pos0)[:S]
    H, dh, th, D = wl.n_kv_heads, wl.head_dim, wl.rope_theta, wl.kv_width
    f64 = lambda t: None if t is None else t.detach().to("cpu", torch.float64).numpy()  # noqa: E731
    rows = lambda t: None if t is None else f64(t[:S])  # noqa: E731
    t_enc = {True: 0.0, False: 0.0}
    t_con = {True: 0.0, False: 0.0}
    n_done = {True: 0, False: 0}
    # interleave layer kinds so a budget cut still samples both
    patch_layers = [l for l in range(wl.n_layers) if wl.is_patch[l]]
    reuse_layers = [l for l in range(wl.n_layers) if not wl.is_patch[l]]
    seq = []
    while patch_layers or reuse_layers:
        if patch_layers:
            seq.append(patch_layers.pop(0))
        for _ in range(7):
            if reuse_layers:
                seq.append(reuse_layers.pop(0))
    spent = 0.0
    for l in seq:
        if spent > budget_s:
            break
        kind = bool(wl.is_patch[l])
        if kind:
            w1, b1, w2, b2 = (f64(x) for x in aligner[l])
            hin, eh, wk, wv = rows(inp.h_in[l]), f64(inp.w_enc_h[l]), f64(inp.w_k[l]), f64(inp.w_v[l])
            t0 = time.perf_counter()
            zh = O.encode_h(hin, eh)
            t1 = time.perf_counter()
            hh, _ = O.align(zh, w1, b1, w2, b2)
            O.patch_k(hh, wk, f64(inp.b_k[l]), pos, H, dh, th)
            O.patch_v(hh, wv, f64(inp.b_v[l]))
            t2 = time.perf_counter()
        else:
            ka, va = rows(inp.k_in[l]), rows(inp.v_in[l])
            ek, ev, fk, fv = (f64(inp.w_enc_k[l]), f64(inp.w_enc_v[l]), f64(inp.w_dec_k[l]),
                              f64(inp.w_dec_v[l]))
            mk, mv = f64(inp.mu_k[l]), f64(inp.mu_v[l])
            t0 = time.perf_counter()
            zk = O.encode_k(ka, pos, ek, mk, H, dh, th)
            zv = O.encode_v(va, ev, mv)
            t1 = time.perf_counter()
            O.decode_k(zk, fk, mk, pos, H, dh, th)
            O.decode_v(zv, fv, mv, D)
            t2 = time.perf_counter()
        t_enc[kind] += t1 - t0
        t_con[kind] += t2 - t1
        n_done[kind] += 1
        spent += t2 - t0
    n_all = {True: sum(1 for p in wl.is_patch if p), False: sum(1 for p in wl.is_patch if not p)}
    est = lambda t: sum(t[k] / max(n_done[k], 1) * n_all[k] for k in (True, False))  # noqa: E731
    scale = wl.n_tokens / max(S, 1)
    est_con, est_enc = est(t_con) * scale, est(t_enc) * scale
    kv = algorithmic(wl)["kv_bytes"]
    return {
        "value": round(kv / est_con / 1e9, 4), "unit": "GB/s", "cores": threads or cores,
        "host_cpus": cores, "kind": "oracle",
        "sample": (f"fp64 numpy oracle on {n_done[False]}/{n_all[False]} Reuse and "
                   f"{n_done[True]}/{n_all[True]} Patch layers over {S} of {wl.n_tokens} tokens "
                   f"(timed {spent:.1f} s), extrapolated per layer kind and token count: value = "
                   f"KV bytes over the "
                   f"consumer's Reuse decode + Patch (aligner, then W_K/W_V) on the oracle's own "
                   f"codes; inputs converted to fp64 outside the timed region"),
        "est_consumer_s": round(est_con, 3), "est_encode_s": round(est_enc, 3),
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


def time_fit(dev, steps, warmup, stream, fit_workload="fit_llama3_8b_head_shared_bf16"):
    """The offline Reuse fit at the Llama-3-8B shape with the head-shared basis (w = d_h = 128:
    8192 tokens x 8 heads = 65,536 calibration rows per layer, 28 Reuse layers): ``scd_fit_gram``
    and ``scd_fit_solve`` for keys and values, HIP events on the stream they run on.  The Gram is
    HBM-bound (2w = 256 columns: about 128 flops per byte of the symmetric product); algorithmic
    bytes read both caches once and write the Gram and column sums once.  The solve is the
    O(w^3) fp64 step (each stage one launch over all layers; the tridiagonalisation and the
    Cholesky one launch per column), reported as time per call."""
    import torch

    import paper_2606_07684_amd as scd
    from synth import workloads as W

    wl = {w.name: w for w in (W.FIT_LLAMA3_8B, *W.FIT_WORKLOADS, W.FIT_W1024_BF16)}[fit_workload]
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
            "solve": {"kernels": "fit_prep/tridiag/bisect/inverse/back/project/normal/chol/out",
                      "ms_per_call": round(solve_ms / 2, 3), "calls": 2,
                      "layers_per_call": len(R),
                      # prep, the per-column Householder steps until 128 rows remain, their
                      # one-launch tail, five stages, the Cholesky (one launch up to 128), the solves
                      "launches_per_call": 1 + max(n2 - 128, 0) + 1 + 5 + (1 if w <= 128 else w) + 1}}


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




def make_model(wl):
    import paper_2606_07684_amd as scd

    return scd.Model(n_layers=wl.n_layers, d_model=wl.d_model, n_kv_heads=wl.n_kv_heads,
                     head_dim=wl.head_dim, rope_theta=wl.rope_theta, dtype=wl.dtype,
                     is_patch=wl.is_patch, rank_k=wl.ranks, rank_v=wl.rank_v, rank_h=wl.ranks,
                     basis_width=wl.w)


def make_batch(wl, dev):
    import paper_2606_07684_amd as scd
    from synth import workloads as W

    cu = W.cu_seqlens(wl, dev) if wl.n_seqs > 1 or wl.pos0 is not None else None
    return scd.Batch(n_tokens=wl.n_tokens, cu_seqlens=cu, pos0=W.pos0(wl, dev))


class Codec:
    """Every buffer of one workload on the GPU and the step's three prepared entry-point calls."""

    def __init__(self, wl, dev):
        import torch

        import paper_2606_07684_amd as scd
        from synth import workloads as W

        self.wl = wl
        L, T, D, h = wl.n_layers, wl.n_tokens, wl.kv_width, wl.hidden_width
        dt = wl.torch_dtype
        self.inp = W.Inputs(wl, dev, decode=False)  # the decode consumes this step's own codes
        self.model, self.batch = make_model(wl), make_batch(wl, dev)
        self.rope = scd.scd_rope_table(self.model, wl.max_position)
        self.z_k, self.z_v, self.z_h = W.alloc_codes(wl, dev)
        self.k_cache, self.v_cache = W.alloc_caches(wl, dev)
        inp = self.inp
        # aligner weights and their fold into the consumer's projections (once, weights only)
        self.aligner = [None] * L
        fk, fv, ck, cv = ([None] * L for _ in range(4))
        w2, b2 = [None] * L, [None] * L
        for l in wl.patch_layers:
            self.aligner[l] = W.aligner_weights(wl, l, dev)
            w2[l], b2[l] = self.aligner[l][2], self.aligner[l][3]
            fk[l] = torch.empty((D, h), dtype=dt, device=dev)
            fv[l] = torch.empty((D, h), dtype=dt, device=dev)
            ck[l] = torch.empty((D,), dtype=dt, device=dev)
            cv[l] = torch.empty((D,), dtype=dt, device=dev)
        self.fold = scd.prepare_patch_fold(self.model, h, w2, b2, inp.w_k, inp.w_v, inp.b_k,
                                           inp.b_v, fk, fv, ck, cv)
        self.folded = (fk, fv, ck, cv)
        # one act buffer per Patch layer: the layers then run as one launch of each product
        self.act = [torch.empty((T, h), dtype=dt, device=dev) if wl.is_patch[l] else None
                    for l in range(L)]
        w1 = [a[0] if a is not None else None for a in self.aligner]
        b1 = [a[1] if a is not None else None for a in self.aligner]
        self.enc = scd.prepare_encode(self.model, self.batch, self.rope, inp.k_in, inp.v_in,
                                      inp.h_in, inp.w_enc_k, inp.w_enc_v, inp.w_enc_h, inp.mu_k,
                                      inp.mu_v, self.z_k, self.z_v, self.z_h)
        self.dec = scd.prepare_reuse_decode(self.model, self.batch, self.rope, self.z_k, self.z_v,
                                            inp.w_dec_k, inp.w_dec_v, inp.mu_k, inp.mu_v,
                                            self.k_cache, self.v_cache)
        self.pat = scd.prepare_patch_kv_from_codes(self.model, self.batch, self.rope, h, self.z_h,
                                                   w1, b1, fk, fv, ck, cv, self.act,
                                                   self.k_cache, self.v_cache)

    def step(self, stream, ev=None, split=True):
        """One step; with events, ev[0..3] around encode, decode and Patch (ev[2], between the
        consumer's two calls, only if split)."""
        if ev is not None:
            ev[0].record(stream)
        self.enc(stream)
        if ev is not None:
            ev[1].record(stream)
        self.dec(stream)
        if ev is not None and split:
            ev[2].record(stream)
        self.pat(stream)
        if ev is not None:
            ev[3].record(stream)


def reduce_events(events, split):
    """Per-phase times and consumer spans (ms) from each step's four events: encode from every
    step, the decode/Patch split from the steps with an event between them (split), the consumer
    span (decode start to Patch end) from the others, or from every step if all are split."""
    phase = {k: [] for k in PHASES}
    consumer = []
    every = all(split)
    for ev, sp in zip(events, split):
        phase["encode"].append(ev[0].elapsed_time(ev[1]))
        if sp:
            phase["reuse_decode"].append(ev[1].elapsed_time(ev[2]))
            phase["patch"].append(ev[2].elapsed_time(ev[3]))
        if not sp or every:
            consumer.append(ev[1].elapsed_time(ev[3]))
    return phase, consumer


def measure(wl, dev, steps, warmup, stream, codec=None):
    """W warm-up steps, then K timed steps bracketed by synchronisations (wall clock), with HIP
    events on the stream between the entry points.  Returns the workload's block."""
    import torch

    codec = codec or Codec(wl, dev)
    torch.cuda.synchronize()
    ev_fold = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ev_fold[0].record(stream)
    codec.fold(stream)
    ev_fold[1].record(stream)
    for _ in range(warmup):
        codec.step(stream)
    torch.cuda.synchronize()
    fold_ms = ev_fold[0].elapsed_time(ev_fold[1])
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    # even steps: an event between decode and Patch (the phase split); odd steps: none (the
    # consumer span without the event's idle gap)
    split = [i % 2 == 0 or steps == 1 for i in range(steps)]
    for i in range(steps):
        codec.step(stream, events[i], split[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    phase, consumer = reduce_events(events, split)
    mean = {k: sum(v) / len(v) for k, v in phase.items()}
    cons_ms = sum(consumer) / len(consumer)
    alg = algorithmic(wl)
    kv = alg["kv_bytes"]
    ms_per_step = wall * 1e3 / steps
    digest = source_digest()
    rooflines = {}
    for k in PHASES:
        sym, bound = KERNELS[k]
        b, f = alg[k]
        t = mean[k] * 1e-3
        if bound == "hbm":
            ach, peak, unit = b / t / 1e9, HBM_PEAK_GBPS, "GB/s"
        else:
            ach, peak, unit = f / t / 1e12, MFMA_PEAK_TFLOPS[wl.dtype], "TFLOP/s"
        rooflines[k] = {"kernel": sym, "bound": bound, "achieved": round(ach, 2), "peak": peak,
                        "unit": unit, "frac": round(ach / peak, 4),
                        "traffic": traffic_for(wl.name, k, digest),
                        "ms_per_launch": round(mean[k], 4), "alg_bytes": b, "alg_flops": f}
    stats = lambda v: {"mean": round(sum(v) / len(v), 4), "median": round(pct(v, 50), 4),  # noqa
                       "p10": round(pct(v, 10), 4), "p90": round(pct(v, 90), 4)}
    # the combined readings of the decode-side target (Reuse decode + Patch from the codes):
    #   reuse_hbm_frac:     Reuse algorithmic bytes / t_reuse / 8 TB/s
    #   patch_mfma_frac:    Patch flops (aligner hidden layer + folded product) / t_patch / peak
    #   roofline_time_frac: the serial roofline time of the two phases (Reuse bytes at 8 TB/s, the
    #                       aligner's hidden layer bytes at 8 TB/s, the folded product's flops at
    #                       the MFMA peak) over the consumer span
    #   literal_hbm_frac:   (Reuse + Patch algorithmic bytes) / consumer span / 8 TB/s
    t_r, t_p = mean["reuse_decode"] * 1e-3, mean["patch"] * 1e-3
    hbm, mfma = HBM_PEAK_GBPS * 1e9, MFMA_PEAK_TFLOPS[wl.dtype] * 1e12
    roof = alg["reuse_decode"][0] / hbm + alg["patch_act"][0] / hbm + alg["patch_gemm"][1] / mfma
    block = {
        "workload": wl.name,
        "value_GBps": round(kv / (cons_ms * 1e-3) / 1e9, 2),
        "consumer_ms": stats(consumer),
        "tokens_per_s": round(wl.n_tokens / (cons_ms * 1e-3), 1),
        "ms_per_step": round(ms_per_step, 4),
        "whole_step_GBps": round(kv / (ms_per_step * 1e-3) / 1e9, 2),
        "phase_ms": {k: stats(v) for k, v in phase.items()},
        "rooflines": rooflines,
        "decode_readings": {
            "reuse_hbm_frac": round(alg["reuse_decode"][0] / t_r / hbm, 4),
            "patch_mfma_frac": round(alg["patch"][1] / t_p / mfma, 4) if t_p > 0 else None,
            "roofline_time_frac": round(roof / (cons_ms * 1e-3), 4),
            "literal_hbm_frac": round((alg["reuse_decode"][0] + alg["patch"][0])
                                      / (cons_ms * 1e-3) / hbm, 4),
        },
        "fold_ms_once": round(fold_ms, 4),
        "kv_bytes": kv,
        "shape": {"n_layers": wl.n_layers, "d_model": wl.d_model, "n_kv_heads": wl.n_kv_heads,
                  "head_dim": wl.head_dim, "n_tokens": wl.n_tokens, "n_requests": wl.n_seqs,
                  "ranks": sorted(set(wl.ranks)), "ranks_v": sorted(set(wl.rank_v)),
                  "patch_layers": list(wl.patch_layers), "basis_width": wl.w,
                  "aligner_hidden": wl.hidden_width, "rope_theta": wl.rope_theta,
                  "dtype": wl.dtype},
    }
    if wl.n_seqs > 1:  # every request's tokens over the consumer time of the packed batch
        lens = [int(wl.cu_seqlens[b + 1] - wl.cu_seqlens[b]) for b in range(wl.n_seqs)]
        per = sorted(n / (cons_ms * 1e-3) for n in lens)
        block["tokens_per_s_per_request"] = {"min": round(per[0], 1),
                                             "median": round(pct(per, 50), 1),
                                             "max": round(per[-1], 1)}
    return block, codec


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="llama3_8b_bf16")
    ap.add_argument("--no-configs", action="store_true",
                    help="measure only --workload (skip the per-config blocks)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-receive", action="store_true",
                    help="skip the receipt timing (its decode launches share the step's kernel "
                         "and grid, so kernel traces of the step leave it out)")
    ap.add_argument("--fit-workload", default="fit_llama3_8b_head_shared_bf16",
                    help="calibration shape of the offline fit timing (e.g. fit_w1024_bf16)")
    ap.add_argument("--no-fit", action="store_true",
                    help="skip the offline fit timing (it runs after the step's timing)")
    ap.add_argument("--no-aligner", action="store_true",
                    help="skip the unfolded aligner timing (scd_patch_align)")
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

    known = {w.name: w for w in (*W.CONFIGS, *W.MODEL_SCALE_EXTRA, *W.TEST_WORKLOADS)}
    wl = known[args.workload]
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    scd.load_library()
    stream = torch.cuda.current_stream()
    print(f"[bench] {wl.name}: building inputs (T={wl.n_tokens}, L={wl.n_layers})",
          file=sys.stderr, flush=True)
    block, codec = measure(wl, dev, args.steps, args.warmup, stream)
    print(f"[bench] {wl.name}: timed steps done", file=sys.stderr, flush=True)
    dominant = max(PHASES, key=lambda k: block["phase_ms"][k]["mean"])
    dom = block["rooflines"][dominant]
    out = {
        "metric": "reconstructed KV GB/s & tokens/s (Reuse+Patch decode); % of HBM roofline",
        "value": block["value_GBps"],
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": block["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic (seeded, model-shaped; no weights or datasets)",
        "config": {"workload": wl.name, **block["shape"]},
        "tokens_per_s": block["tokens_per_s"],
        "consumer_ms": block["consumer_ms"],
        "whole_step_GBps": block["whole_step_GBps"],
        "phase_ms": block["phase_ms"],
        "roofline": {k: dom[k] for k in ("bound", "achieved", "peak", "unit", "frac", "traffic")},
        "roofline_kernel": dom["kernel"],
        "rooflines": block["rooflines"],
        "decode_readings": block["decode_readings"],
        "fold_ms_once": block["fold_ms_once"],
        "source_digest": source_digest(),
    }
    copy_gbps = copy_ceiling(dev)
    out["decode_readings"]["copy_ceiling_GBps"] = round(copy_gbps, 1)
    out["decode_readings"]["reuse_frac_of_copy_ceiling"] = round(
        block["rooflines"]["reuse_decode"]["achieved"] / copy_gbps, 4)

    # The aligner without the fold (scd_patch_align, the unfolded chain's first half), beside.
    if any(wl.is_patch) and not args.no_aligner:
        print("[bench] timing the unfolded aligner", file=sys.stderr, flush=True)
        out["aligner_unfolded"] = time_aligner(wl, dev, args.steps, args.warmup, stream)

    # The consumer's receipt from host memory (PCIe-inclusive), beside the step.
    if not args.no_receive:
        print("[bench] timing the streamed receipt", file=sys.stderr, flush=True)
        out["receive"] = time_receive(wl, dev, args.steps, args.warmup, stream, codec.model,
                                      codec.batch, codec.rope, codec.inp, codec.z_k, codec.z_v,
                                      codec.z_h, codec.k_cache, codec.v_cache)

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
        out["cpu_baseline"] = cpu_baseline(wl, codec.inp, codec.aligner)
    del codec
    torch.cuda.synchronize()
    torch.cuda.empty_cache()

    # The offline Reuse fit (Section 4.3.1), at the head-shared calibration shape, beside the step.
    if not args.no_fit:
        print("[bench] timing the offline fit", file=sys.stderr, flush=True)
        out["fit"] = time_fit(dev, args.steps, args.warmup, stream, args.fit_workload)
        torch.cuda.empty_cache()

    # Every model-shaped workload in the same run (the same step and readings; a CPU baseline with
    # a smaller budget each).
    if not args.no_configs:
        out["configs"] = {}
        for other in W.CONFIGS:
            if other.name == wl.name:
                continue
            print(f"[bench] {other.name}: building inputs (T={other.n_tokens}, "
                  f"L={other.n_layers})", file=sys.stderr, flush=True)
            blk, cdc = measure(other, dev, args.steps, args.warmup, stream)
            if not args.no_cpu_baseline:
                print(f"[bench] {other.name}: CPU oracle baseline", file=sys.stderr, flush=True)
                blk["cpu_baseline"] = cpu_baseline(other, cdc.inp, cdc.aligner, budget_s=8.0,
                                                   max_tokens=2048)
            out["configs"][other.name] = blk
            del cdc
            torch.cuda.synchronize()
            torch.cuda.empty_cache()
            print(f"[bench] {other.name}: {blk['value_GBps']} GB/s", file=sys.stderr, flush=True)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
