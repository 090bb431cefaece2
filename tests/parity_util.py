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


def max_abs_rel_cols(got, want) -> float:
    """max over columns j of max_i |G - O|[i, j] / max_i |O|[i, j]: the code tensors' metric.  A
    code column carries one direction of the basis, and with a decaying spectrum the columns'
    scales differ by orders of magnitude, so each column is held to the tolerance on its own
    scale (a per-tensor scale would let the small columns be wrong)."""
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    assert got.shape == want.shape, (got.shape, want.shape)
    if not np.all(np.isfinite(got)):
        return float("inf")
    if got.size == 0:
        return 0.0
    num = np.max(np.abs(got - want), axis=0)
    den = np.max(np.abs(want), axis=0)
    return float(np.max(num / np.where(den > 0, den, 1.0)))


class ErrAccum:
    """Streams the two metrics over chunks of rows: per-tensor max |G - O| / max |O| (caches) and
    the per-column form (codes), keyed by (name, layer)."""

    def __init__(self):
        self.num, self.den, self.cols = {}, {}, set()

    def add(self, key, got, want, per_column=False):
        got = np.asarray(got, np.float64)
        want = np.asarray(want, np.float64)
        assert got.shape == want.shape, (got.shape, want.shape)
        if got.size == 0:
            return
        axis = 0 if per_column else None
        d = np.max(np.abs(got - want), axis=axis)
        if not np.all(np.isfinite(got)):
            d = np.full_like(np.asarray(d, np.float64), np.inf)
        o = np.max(np.abs(want), axis=axis)
        if per_column:
            self.cols.add(key)
        self.num[key] = np.maximum(self.num.get(key, 0.0), d)
        self.den[key] = np.maximum(self.den.get(key, 0.0), o)

    def errors(self) -> dict:
        out = {}
        for k, n in self.num.items():
            dd = np.asarray(self.den[k], np.float64)
            out[k] = float(np.max(np.asarray(n) / np.where(dd > 0, dd, 1.0)))
        return out


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
            errs[("z_k", l)] = max_abs_rel_cols(take(out["z_k"][l], crow), zk)
            errs[("z_v", l)] = max_abs_rel_cols(take(out["z_v"][l], crow), zv)
    for l in inp.P:
        if "k_cache" in out and inp.h_hat[l] is not None:
            hh = take(inp.h_hat[l], tokens)
            ok = O.patch_k(hh, f64(inp.w_k[l]), f64(inp.b_k[l]), p, H, dh, th)
            ov = O.patch_v(hh, f64(inp.w_v[l]), f64(inp.b_v[l]))
            errs[("k_cache", l)] = max_abs_rel(take(out["k_cache"][l], tokens), ok)
            errs[("v_cache", l)] = max_abs_rel(take(out["v_cache"][l], tokens), ov)
        if "z_h" in out:
            zh = O.encode_h(take(inp.h_in[l], tokens), f64(inp.w_enc_h[l]))
            errs[("z_h", l)] = max_abs_rel_cols(take(out["z_h"][l], tokens), zh)
    return errs


def compare_full_chunked(wl: W.Workload, inp: Inputs, out: dict, chunk: int = 8192,
                         label: str = "") -> dict:
    """compare_all over every token of a full-size workload, layer by layer in chunks of token rows
    (the fp64 oracle's working set stays a few hundred MiB); same keys and metrics."""
    pos = host_positions(wl)
    H, dh, th, D, g = wl.n_kv_heads, wl.head_dim, wl.rope_theta, wl.kv_width, wl.g
    acc = ErrAccum()
    for l in range(wl.n_layers):
        print(f"[{label}] layer {l} ({'patch' if wl.is_patch[l] else 'reuse'})", flush=True)
        wdk = f64(inp.w_dec_k[l]) if l in inp.R else None
        wdv = f64(inp.w_dec_v[l]) if l in inp.R else None
        wek = f64(inp.w_enc_k[l]) if l in inp.R else None
        wev = f64(inp.w_enc_v[l]) if l in inp.R else None
        mk = f64(inp.mu_k[l]) if l in inp.R else None
        mv = f64(inp.mu_v[l]) if l in inp.R else None
        wk = f64(inp.w_k[l]) if l in inp.P and inp.w_k[l] is not None else None
        wv = f64(inp.w_v[l]) if l in inp.P and inp.w_v[l] is not None else None
        weh = f64(inp.w_enc_h[l]) if l in inp.P and inp.w_enc_h[l] is not None else None
        for t0 in range(0, wl.n_tokens, chunk):
            t1 = min(t0 + chunk, wl.n_tokens)
            p = pos[t0:t1]
            sl = slice(t0, t1)
            cs = slice(t0 * g, t1 * g)
            if l in inp.R:
                if "k_cache" in out and inp.z_k[l] is not None:
                    ok = O.decode_k(f64(inp.z_k[l][cs]), wdk, mk, p, H, dh, th)
                    ov = O.decode_v(f64(inp.z_v[l][cs]), wdv, mv, D)
                    acc.add(("k_cache", l), f64(out["k_cache"][l][sl]), ok)
                    acc.add(("v_cache", l), f64(out["v_cache"][l][sl]), ov)
                if "z_k" in out:
                    zk = O.encode_k(f64(inp.k_in[l][sl]), p, wek, mk, H, dh, th)
                    zv = O.encode_v(f64(inp.v_in[l][sl]), wev, mv)
                    acc.add(("z_k", l), f64(out["z_k"][l][cs]), zk, per_column=True)
                    acc.add(("z_v", l), f64(out["z_v"][l][cs]), zv, per_column=True)
            else:
                if "k_cache" in out and inp.h_hat[l] is not None:
                    hh = f64(inp.h_hat[l][sl])
                    ok = O.patch_k(hh, wk, f64(inp.b_k[l]), p, H, dh, th)
                    ov = O.patch_v(hh, wv, f64(inp.b_v[l]))
                    acc.add(("k_cache", l), f64(out["k_cache"][l][sl]), ok)
                    acc.add(("v_cache", l), f64(out["v_cache"][l][sl]), ov)
                if "z_h" in out:
                    zh = O.encode_h(f64(inp.h_in[l][sl]), weh)
                    acc.add(("z_h", l), f64(out["z_h"][l][sl]), zh, per_column=True)
    return acc.errors()


def assert_within(errs: dict, tol: float, label: str):
    bad = {k: v for k, v in errs.items() if not (v <= tol)}
    worst = max(errs.items(), key=lambda kv: kv[1]) if errs else None
    print(f"[{label}] {len(errs)} tensors, worst {worst}", flush=True)
    assert not bad, f"{label}: tensors above tolerance {tol}: {sorted(bad.items())[:8]}"


class PatchFromCodes:
    """Stored inputs of every Patch layer, the GPU fold and the GPU Patch from codes."""

    def __init__(self, wl, fill=float("nan"), shared_act=True):
        dev = torch.device("cuda")
        self.wl = wl
        L, T, h, D = wl.n_layers, wl.n_tokens, wl.hidden_width, wl.kv_width
        dt = wl.torch_dtype
        self.z_h, self.w1, self.b1, self.w2, self.b2 = ([None] * L for _ in range(5))
        self.w_k, self.w_v, self.b_k, self.b_v = ([None] * L for _ in range(4))
        self.fk, self.fv, self.ck, self.cv = ([None] * L for _ in range(4))
        for l in wl.patch_layers:
            self.z_h[l] = W.patch_codes(wl, l, dev)
            self.w1[l], self.b1[l], self.w2[l], self.b2[l] = W.aligner_weights(wl, l, dev)
            self.w_k[l], self.w_v[l] = W.proj_weights(wl, l, dev)
            self.b_k[l], self.b_v[l] = W.proj_bias(wl, l, dev)
            self.fk[l] = torch.full((D, h), fill, dtype=dt, device=dev)
            self.fv[l] = torch.full((D, h), fill, dtype=dt, device=dev)
            self.ck[l] = torch.full((D,), fill, dtype=dt, device=dev)
            self.cv[l] = torch.full((D,), fill, dtype=dt, device=dev)
        self.model = model_of(wl)
        self.batch = batch_of(wl, dev)
        scd.scd_patch_fold(self.model, h, self.w2, self.b2, self.w_k, self.w_v, self.b_k,
                           self.b_v, self.fk, self.fv, self.ck, self.cv)
        self.rope = scd.scd_rope_table(self.model, wl.max_position)
        shared = torch.empty((T, h), dtype=dt, device=dev)
        self.act = [(shared if shared_act else torch.empty((T, h), dtype=dt, device=dev))
                    if l in wl.patch_layers else None for l in range(L)]
        self.kc, self.vc = alloc_caches(wl, dev, fill)
        scd.scd_patch_kv_from_codes(self.model, self.batch, self.rope, h, self.z_h, self.w1,
                                    self.b1, self.fk, self.fv, self.ck, self.cv, self.act,
                                    self.kc, self.vc)
        torch.cuda.synchronize()

    def fold_errors(self):
        errs = {}
        for l in self.wl.patch_layers:
            for br, w_p, b_p, f, c in (("k", self.w_k, self.b_k, self.fk, self.ck),
                                       ("v", self.w_v, self.b_v, self.fv, self.cv)):
                want_f, want_c = O.fold_aligner(f64(w_p[l]), f64(b_p[l]), f64(self.w2[l]),
                                                f64(self.b2[l]))
                errs[("w_fold_" + br, l)] = max_abs_rel(f64(f[l]), want_f)
                errs[("c_" + br, l)] = max_abs_rel(f64(c[l]), want_c)
        return errs

    def cache_errors(self, tokens):
        wl = self.wl
        pos = host_positions(wl)[tokens]
        errs = {}
        for l in wl.patch_layers:
            h_hat, _ = O.align(take(self.z_h[l], tokens), f64(self.w1[l]), f64(self.b1[l]),
                               f64(self.w2[l]), f64(self.b2[l]))
            want_k = O.patch_k(h_hat, f64(self.w_k[l]), f64(self.b_k[l]), pos, wl.n_kv_heads,
                               wl.head_dim, wl.rope_theta)
            want_v = O.patch_v(h_hat, f64(self.w_v[l]), f64(self.b_v[l]))
            errs[("k_cache", l)] = max_abs_rel(take(self.kc[l], tokens), want_k)
            errs[("v_cache", l)] = max_abs_rel(take(self.vc[l], tokens), want_v)
        return errs
