"""Shared helpers of the GPU parity tests: build a workload's inputs, run the HIP path through the
C ABI, run the oracle on the same stored inputs (whole tensors or sampled rows) and compare."""
from __future__ import annotations

import numpy as np
import torch

import paper_2606_07684_amd as scd
from oracle import scd_oracle as O
from synth import workloads as W

TOL = {"f32": 1e-5, "bf16": 2e-2}


Inputs = W.Inputs
alloc_caches = W.alloc_caches
alloc_codes = W.alloc_codes


def model_of(wl: W.Workload) -> scd.Model:
    return scd.Model(n_layers=wl.n_layers, d_model=wl.d_model, n_kv_heads=wl.n_kv_heads,
                     head_dim=wl.head_dim, rope_theta=wl.rope_theta, dtype=wl.dtype,
                     is_patch=wl.is_patch, rank_k=wl.ranks, rank_v=wl.rank_v, rank_h=wl.ranks,
                     basis_width=wl.w)


def batch_of(wl: W.Workload, device) -> scd.Batch:
    cu = W.cu_seqlens(wl, device) if wl.n_seqs > 1 or wl.pos0 is not None else None
    return scd.Batch(n_tokens=wl.n_tokens, cu_seqlens=cu, pos0=W.pos0(wl, device))


def host_positions(wl: W.Workload) -> np.ndarray:
    return O.positions(wl.cu_seqlens, wl.pos0)


def f64(t):
    return None if t is None else t.detach().to("cpu", torch.float64).numpy()


def max_abs_rel(got, want) -> float:
    """max |G - O| / max |O| over one tensor (both fp64)."""
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    assert got.shape == want.shape, (got.shape, want.shape)
    if not np.all(np.isfinite(got)):
        return float("inf")
    den = np.max(np.abs(want))
    return float(np.max(np.abs(got - want)) / (den if den > 0 else 1.0))


def run_gpu(wl: W.Workload, inp: Inputs, rope, which=("decode", "patch", "encode"), fill=None):
    """Run the requested entry points; return dict of outputs (device tensors)."""
    dev = torch.device("cuda")
    model = model_of(wl)
    batch = batch_of(wl, dev)
    out = {}
    if "decode" in which or "patch" in which:
        kc, vc = alloc_caches(wl, dev, fill)
        out["k_cache"], out["v_cache"] = kc, vc
        if "decode" in which:
            scd.scd_reuse_decode(model, batch, rope, inp.z_k, inp.z_v, inp.w_dec_k, inp.w_dec_v,
                                 inp.mu_k, inp.mu_v, kc, vc)
        if "patch" in which:
            scd.scd_patch_kv(model, batch, rope, inp.h_hat, inp.w_k, inp.w_v, inp.b_k, inp.b_v,
                             kc, vc)
    if "encode" in which:
        z_k, z_v, z_h = alloc_codes(wl, dev)
        scd.scd_encode(model, batch, rope, inp.k_in, inp.v_in, inp.h_in, inp.w_enc_k,
                       inp.w_enc_v, inp.w_enc_h, inp.mu_k, inp.mu_v, z_k, z_v, z_h)
        out["z_k"], out["z_v"], out["z_h"] = z_k, z_v, z_h
    torch.cuda.synchronize()
    return out


def sample_tokens(wl: W.Workload, n_random=96, seed=0) -> np.ndarray:
    """Token rows the oracle checks one by one at full size: random rows plus every request's
    first and last token and the rows around 128-row tile edges."""
    T = wl.n_tokens
    rng = np.random.default_rng(seed)
    cu = wl.cu_seqlens
    rows = set(rng.integers(0, T, n_random).tolist())
    for b in range(wl.n_seqs):
        if cu[b + 1] > cu[b]:
            rows.update([int(cu[b]), int(cu[b + 1]) - 1])
    for edge in (127, 128, 255, 256, T - 129, T - 128, T - 1):
        if 0 <= edge < T:
            rows.add(int(edge))
    return np.array(sorted(rows), dtype=np.int64)


def code_rows(wl: W.Workload, tokens: np.ndarray) -> np.ndarray:
    return (tokens[:, None] * wl.g + np.arange(wl.g)[None, :]).reshape(-1)


def take(t: torch.Tensor, rows) -> np.ndarray:
    idx = torch.as_tensor(rows, device=t.device)
    return f64(t.index_select(0, idx))


def compare_all(wl: W.Workload, inp: Inputs, out: dict, tokens=None):
    """Oracle on the same stored inputs; returns {(name, layer): err}.  ``tokens`` restricts the
    comparison to those token rows (full tensors when None)."""
    pos = host_positions(wl)
    H, dh, th, D = wl.n_kv_heads, wl.head_dim, wl.rope_theta, wl.kv_width
    if tokens is None:
        tokens = np.arange(wl.n_tokens)
    crow = code_rows(wl, tokens)
    p = pos[tokens]
    errs = {}
    for l in inp.R:
        if "k_cache" in out and inp.z_k[l] is not None:
            ok = O.decode_k(take(inp.z_k[l], crow), f64(inp.w_dec_k[l]), f64(inp.mu_k[l]), p, H,
                            dh, th)
            ov = O.decode_v(take(inp.z_v[l], crow), f64(inp.w_dec_v[l]), f64(inp.mu_v[l]), D)
            errs[("k_cache", l)] = max_abs_rel(take(out["k_cache"][l], tokens), ok)
            errs[("v_cache", l)] = max_abs_rel(take(out["v_cache"][l], tokens), ov)
        if "z_k" in out:
            zk = O.encode_k(take(inp.k_in[l], tokens), p, f64(inp.w_enc_k[l]), f64(inp.mu_k[l]),
                            H, dh, th)
            zv = O.encode_v(take(inp.v_in[l], tokens), f64(inp.w_enc_v[l]), f64(inp.mu_v[l]))
            errs[("z_k", l)] = max_abs_rel(take(out["z_k"][l], crow), zk)
            errs[("z_v", l)] = max_abs_rel(take(out["z_v"][l], crow), zv)
    for l in inp.P:
        if "k_cache" in out and inp.h_hat[l] is not None:
            hh = take(inp.h_hat[l], tokens)
            ok = O.patch_k(hh, f64(inp.w_k[l]), f64(inp.b_k[l]), p, H, dh, th)
            ov = O.patch_v(hh, f64(inp.w_v[l]), f64(inp.b_v[l]))
            errs[("k_cache", l)] = max_abs_rel(take(out["k_cache"][l], tokens), ok)
            errs[("v_cache", l)] = max_abs_rel(take(out["v_cache"][l], tokens), ov)
        if "z_h" in out:
            zh = O.encode_h(take(inp.h_in[l], tokens), f64(inp.w_enc_h[l]))
            errs[("z_h", l)] = max_abs_rel(take(out["z_h"][l], tokens), zh)
    return errs


def assert_within(errs: dict, tol: float, label: str):
    bad = {k: v for k, v in errs.items() if not (v <= tol)}
    worst = max(errs.items(), key=lambda kv: kv[1]) if errs else None
    print(f"[{label}] {len(errs)} tensors, worst {worst}", flush=True)
    assert not bad, f"{label}: tensors above tolerance {tol}: {sorted(bad.items())[:8]}"
