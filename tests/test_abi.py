"""C ABI tests that need no GPU: the library loads and exports every declared symbol, every
validation path returns its status before any launch, and the host-only entry points (routing and
payload accounting) agree bit for bit with the oracle."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2606_07684_amd as scd
from oracle import scd_oracle as O
from synth import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "scd.h")

OK, NULL, SHAPE, SCHED, ALIGN, UNSUP, WS, HIP = range(8)
FAKE = 0x7f0000000000  # a 16-byte aligned address that is never dereferenced


@pytest.fixture(scope="module")
def lib():
    return scd.load_library()


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(scd_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert len(names) >= 11
    for n in names:
        assert hasattr(lib, n), f"libscd.so does not export {n}"
    assert set(names) == set(scd.EXPORTED_SYMBOLS)
    assert scd.scd_abi_version() == 5


def test_status_strings(lib):
    for s in range(8):
        assert lib.scd_status_string(s)
    assert lib.scd_status_string(99) == b"unknown status"


def _model(**kw):
    base = dict(n_layers=3, d_model=256, n_kv_heads=2, head_dim=64, rope_theta=1e4, dtype="bf16",
                is_patch=[0, 1, 0], rank_k=[32, 32, 32], rank_v=[32, 32, 32],
                rank_h=[32, 32, 32])
    base.update(kw)
    return scd.Model(**base)


def _ptrs(L, value=FAKE, skip=()):
    arr = (ctypes.c_void_p * L)()
    for l in range(L):
        if l not in skip:
            arr[l] = value
    return ctypes.cast(arr, ctypes.POINTER(ctypes.c_void_p)), arr


def _decode(lib, model, batch, rope=FAKE, maxp=100, **over):
    L = model.n_layers
    keep = []
    args = {}
    for name in ("z_k", "z_v", "w_dec_k", "w_dec_v", "mu_k", "mu_v", "k_cache", "v_cache"):
        if name in over:
            args[name] = over[name]
        else:
            p, a = _ptrs(L)
            keep.append(a)
            args[name] = p
    st = lib.scd_reuse_decode(ctypes.byref(model._c), ctypes.byref(batch._c), rope, maxp,
                              args["z_k"], args["z_v"], args["w_dec_k"], args["w_dec_v"],
                              args["mu_k"], args["mu_v"], args["k_cache"], args["v_cache"], None)
    return st, lib.scd_last_error().decode()


def _batch(n_tokens=10, n_seqs=1, cu=None):
    b = scd.Batch(n_tokens=n_tokens)
    b._c.n_seqs = n_seqs
    b._c.cu_seqlens = cu
    return b


def test_validation_paths_return_before_launch(lib):
    m = _model()
    b = _batch()
    # model problems
    assert lib.scd_reuse_decode(None, ctypes.byref(b._c), FAKE, 10, *([None] * 8), None) == NULL
    assert _decode(lib, _model(head_dim=80, rope_theta=1e4), b)[0] == UNSUP
    mm = _model()
    mm._c.head_dim = 63
    assert _decode(lib, mm, b)[0] == SHAPE
    assert _decode(lib, _model(basis_width=96), b)[0] == SHAPE
    assert _decode(lib, _model(d_model=250), b)[0] == UNSUP
    mm = _model()
    mm._c.dtype = 7
    assert _decode(lib, mm, b)[0] == SHAPE
    # ranks
    st, msg = _decode(lib, _model(rank_k=[32, 32, 40]), b)
    assert st == SCHED and "rank_k of layer 2" in msg
    assert _decode(lib, _model(rank_v=[256, 32, 32]), b)[0] == SCHED  # > basis width 128
    assert _decode(lib, _model(rank_v=[0, 32, 32]), b)[0] == SCHED
    # patch layer ranks are not the decode's business
    assert _decode(lib, _model(rank_k=[32, 8, 32]), _batch(n_tokens=0))[0] == OK
    # batch problems
    assert _decode(lib, m, _batch(n_seqs=0))[0] == SHAPE
    assert _decode(lib, m, _batch(n_tokens=-1))[0] == SHAPE
    assert _decode(lib, m, _batch(n_seqs=3, cu=None))[0] == NULL
    # pointers
    p, keep = _ptrs(3, skip=(2,))
    st, msg = _decode(lib, m, b, z_k=p)
    assert st == NULL and "z_k[2]" in msg
    p2, keep2 = _ptrs(3, skip=(0,))  # layer 0 missing but ... layer 0 is Reuse: required
    assert _decode(lib, m, b, k_cache=p2)[0] == NULL
    p3, keep3 = _ptrs(3, skip=(1,))  # layer 1 is Patch: entry ignored
    assert _decode(lib, m, _batch(n_tokens=0), z_v=p3)[0] == OK
    p4, keep4 = _ptrs(3, value=FAKE + 2)
    assert _decode(lib, m, b, v_cache=p4)[0] == ALIGN
    # RoPE table
    assert _decode(lib, m, b, rope=None)[0] == WS
    assert _decode(lib, m, b, rope=FAKE + 4)[0] == ALIGN
    assert _decode(lib, m, b, maxp=0)[0] == WS
    assert lib.scd_last_error().decode() != ""


def test_zero_tokens_is_ok_without_launch(lib):
    m = _model()
    assert _decode(lib, m, _batch(n_tokens=0), rope=None)[0] == OK
    assert lib.scd_last_error().decode() == ""
    L = m.n_layers
    p, keep = _ptrs(L)
    st = lib.scd_patch_kv(ctypes.byref(m._c), ctypes.byref(_batch(n_tokens=0)._c), None, 0,
                          p, p, p, None, None, p, p, None)
    assert st == OK
    st = lib.scd_encode(ctypes.byref(m._c), ctypes.byref(_batch(n_tokens=0)._c), None, 0,
                        *([p] * 6), None, None, p, p, p, None)
    assert st == OK


def test_encode_and_patch_validation(lib):
    m = _model()
    b = _batch()
    L = m.n_layers
    p, keep = _ptrs(L)
    q, keepq = _ptrs(L, skip=(1,))
    # encode: Patch layer 1 needs h_in
    st = lib.scd_encode(ctypes.byref(m._c), ctypes.byref(b._c), FAKE, 10, p, p, q, p, p, p,
                        None, None, p, p, p, None)
    assert st == NULL and "h_in[1]" in lib.scd_last_error().decode()
    # encode: rank_h above d_model
    mh = _model(rank_h=[32, 512, 32])
    st = lib.scd_encode(ctypes.byref(mh._c), ctypes.byref(b._c), FAKE, 10, *([p] * 6), None,
                        None, p, p, p, None)
    assert st == SCHED
    # patch: bias entries optional but must be aligned
    r, keepr = _ptrs(L, value=FAKE + 8)
    st = lib.scd_patch_kv(ctypes.byref(m._c), ctypes.byref(b._c), FAKE, 10, p, p, p, r, None, p,
                          p, None)
    assert st == ALIGN
    st = lib.scd_patch_kv(ctypes.byref(m._c), ctypes.byref(b._c), None, 10, p, p, p, None, None,
                          p, p, None)
    assert st == WS
    # positions / rope-table argument checks
    assert lib.scd_positions(ctypes.byref(b._c), None, None) == NULL
    assert lib.scd_rope_table(ctypes.byref(m._c), 0, FAKE, 1 << 20, None) == WS
    need = lib.scd_rope_table_bytes(ctypes.byref(m._c), 100)
    assert need == 100 * 32 * 8
    assert lib.scd_rope_table(ctypes.byref(m._c), 100, FAKE, need - 1, None) == WS


def test_aligner_validation(lib):
    m = _model()  # layer 1 is the Patch layer (rank_h 32, d_model 256)
    b = _batch()
    L = m.n_layers
    p, keep = _ptrs(L)

    def align(model=m, batch=b, hidden=64, z=p, w1=p, b1=None, w2=p, b2=None, act=p, out=p):
        return lib.scd_patch_align(ctypes.byref(model._c), ctypes.byref(batch._c), hidden, z, w1,
                                   b1, w2, b2, act, out, None)

    assert align(hidden=0) == SHAPE
    assert align(hidden=40) == SHAPE
    assert "multiple of 16" in lib.scd_last_error().decode()
    q, keepq = _ptrs(L, skip=(1,))
    assert align(w2=q) == NULL and "w2[1]" in lib.scd_last_error().decode()
    assert align(z=q, batch=_batch(n_tokens=0)) == OK  # no tokens: token buffers may be absent
    r, keepr = _ptrs(L, value=FAKE + 8)
    assert align(b1=r) == ALIGN
    assert align(model=_model(rank_h=[32, 24, 32])) == SCHED
    # act entries must be distinct across Patch layers
    m2 = _model(is_patch=[1, 1, 0])
    assert align(model=m2) == SHAPE and "act[1]" in lib.scd_last_error().decode()
    acts = (ctypes.c_void_p * L)(FAKE, FAKE + 4096, FAKE)
    assert align(model=m2, act=ctypes.cast(acts, ctypes.POINTER(ctypes.c_void_p)),
                 batch=_batch(n_tokens=0)) == OK


@pytest.mark.parametrize("wl", [*W.CONFIGS, *W.MODEL_SCALE_EXTRA, *W.TEST_WORKLOADS],
                         ids=lambda w: w.name)
def test_schedule_and_payload_match_oracle(wl):
    m = scd.Model(n_layers=wl.n_layers, d_model=wl.d_model, n_kv_heads=wl.n_kv_heads,
                  head_dim=wl.head_dim, rope_theta=wl.rope_theta, dtype=wl.dtype,
                  is_patch=wl.is_patch, rank_k=wl.ranks, rank_v=wl.rank_v, rank_h=wl.ranks,
                  basis_width=wl.w)
    reuse, patch = scd.scd_schedule(m)
    assert (reuse, patch) == O.schedule(wl.is_patch)
    total, offs = scd.scd_payload_bytes(m, wl.n_tokens)
    t2, o2 = O.payload_bytes(wl.is_patch, wl.n_tokens, wl.n_kv_heads, wl.head_dim, wl.w,
                             wl.ranks, wl.rank_v, wl.ranks, wl.elem_bytes)
    assert total == t2 and offs == o2


def test_workload_shapes_are_the_stated_ones():
    assert W.BATCHED.n_tokens == 111169 and W.BATCHED.n_seqs == 16
    assert min(W.BATCHED.seq_lens) >= 1024 and max(W.BATCHED.seq_lens) <= 16384
    assert W.LLAMA3_8B.patch_layers == (0, 8, 16, 24)
    assert W.LLAMA3_70B.patch_layers == tuple(range(0, 80, 10))
    assert W.QWEN2_7B.n_tokens == 32768 and W.QWEN2_7B.kv_width == 512
    assert W.TINY_F32.kv_width == 256 and W.TINY_F32.is_patch == (0, 0, 1, 0)


def _wl_model(wl):
    return scd.Model(n_layers=wl.n_layers, d_model=wl.d_model, n_kv_heads=wl.n_kv_heads,
                     head_dim=wl.head_dim, rope_theta=wl.rope_theta, dtype=wl.dtype,
                     is_patch=wl.is_patch, rank_k=wl.ranks, rank_v=wl.rank_v, rank_h=wl.ranks,
                     basis_width=wl.w)


@pytest.mark.parametrize("wl", [*W.CONFIGS, *W.TEST_WORKLOADS], ids=lambda w: w.name)
def test_payload_views_tile_the_packed_buffer(wl):
    """The per-layer views the library hands out start at the oracle's layer offsets, keep K
    before V, and cover the packed buffer exactly once: no gap, no overlap, nothing past the end."""
    import torch
    m = _wl_model(wl)
    T = wl.n_tokens
    total, offs = O.payload_bytes(wl.is_patch, T, wl.n_kv_heads, wl.head_dim, wl.w, wl.ranks,
                                  wl.rank_v, wl.ranks, wl.elem_bytes)
    buf = torch.empty(total + 64, dtype=torch.uint8)
    base = buf.data_ptr()
    assert base % 16 == 0
    z_k, z_v, z_h = scd.scd_payload_views(m, T, buf)
    spans = []
    for l, p in enumerate(wl.is_patch):
        if p:
            assert z_k[l] is None and z_v[l] is None
            assert z_h[l].data_ptr() - base == offs[l]
            assert tuple(z_h[l].shape) == (T, wl.ranks[l])
            spans.append(z_h[l])
        else:
            assert z_h[l] is None
            assert z_k[l].data_ptr() - base == offs[l]
            assert z_v[l].data_ptr() > z_k[l].data_ptr()
            spans += [z_k[l], z_v[l]]
    pos = base
    for t in spans:
        assert t.data_ptr() == pos and t.data_ptr() % 16 == 0
        assert t.dtype == m.torch_dtype and t.is_contiguous()
        pos += t.numel() * t.element_size()
    assert pos == base + total


def test_payload_views_and_streamed_decode_validation(lib):
    m = _model()
    b = _batch()
    L = m.n_layers
    views = [(ctypes.c_void_p * L)() for _ in range(3)]
    vp = [ctypes.cast(v, ctypes.POINTER(ctypes.c_void_p)) for v in views]
    assert lib.scd_payload_views(ctypes.byref(m._c), 10, FAKE, *vp) == OK
    assert views[0][1] is None and views[2][1] == FAKE + 10 * 64 * 2
    assert lib.scd_payload_views(ctypes.byref(m._c), 10, FAKE + 8, *vp) == ALIGN
    assert lib.scd_payload_views(ctypes.byref(m._c), 10, None, *vp) == NULL
    assert lib.scd_payload_views(ctypes.byref(m._c), -1, FAKE, *vp) == SHAPE
    assert lib.scd_payload_views(ctypes.byref(m._c), 10, FAKE, vp[0], None, vp[2]) == NULL
    assert lib.scd_payload_views(ctypes.byref(_model(rank_h=[32, 24, 32])._c), 10, FAKE,
                                 *vp) == SCHED

    def streamed(model=m, batch=b, src=FAKE, dst=FAKE, group=2, **over):
        keep, args = [], []
        for name in ("w_dec_k", "w_dec_v", "mu_k", "mu_v", "k_cache", "v_cache"):
            if name in over:
                args.append(over[name])
            else:
                p, a = _ptrs(model.n_layers)
                keep.append(a)
                args.append(p)
        st = lib.scd_reuse_decode_streamed(ctypes.byref(model._c), ctypes.byref(batch._c), FAKE,
                                           100, src, dst, group, *args, None, None)
        return st, lib.scd_last_error().decode()

    assert streamed(group=0)[0] == SHAPE
    assert streamed(src=None)[0] == NULL
    assert streamed(dst=None)[0] == NULL
    assert streamed(dst=FAKE + 8)[0] == ALIGN
    q, keepq = _ptrs(L, skip=(2,))
    st, msg = streamed(w_dec_v=q)
    assert st == NULL and "w_dec_v[2]" in msg
    assert streamed(model=_model(rank_k=[32, 32, 40]))[0] == SCHED
    # no tokens: an empty payload, nothing to copy or decode, no HIP call
    assert streamed(batch=_batch(n_tokens=0))[0] == OK
    assert streamed(batch=_batch(n_tokens=0), src=None, dst=None)[0] == OK


def _distinct_ptrs(L, k):
    """Per-layer fake addresses, distinct across layers and arguments (never dereferenced)."""
    arr = (ctypes.c_void_p * L)(*[FAKE + (16 * k + l + 1) * 4096 for l in range(L)])
    return ctypes.cast(arr, ctypes.POINTER(ctypes.c_void_p)), arr


def _fit_gram(lib, model, batch, branch=0, rope=FAKE, maxp=100, ws=FAKE, ws_bytes=1 << 40,
              **over):
    L = model.n_layers
    keep, args = [], {}
    for k, name in enumerate(("a_in", "b_in", "gram", "colsum")):
        if name in over:
            args[name] = over[name]
        else:
            p, a = _distinct_ptrs(L, k)
            keep.append(a)
            args[name] = p
    st = lib.scd_fit_gram(ctypes.byref(model._c), ctypes.byref(batch._c), rope, maxp, branch,
                          args["a_in"], args["b_in"], args["gram"], args["colsum"], ws, ws_bytes,
                          None)
    return st, lib.scd_last_error().decode()


def _fit_solve(lib, model, branch=0, n_rows=100, lam=0.1, center=1, ws=FAKE, ws_bytes=1 << 40,
               **over):
    L = model.n_layers
    keep, args = [], {}
    for k, name in enumerate(("gram", "colsum", "w_enc", "w_dec", "mu_enc", "mu_dec")):
        if name in over:
            args[name] = over[name]
        else:
            p, a = _distinct_ptrs(L, k)
            keep.append(a)
            args[name] = p
    st = lib.scd_fit_solve(ctypes.byref(model._c), branch, n_rows, lam, center, args["gram"],
                           args["colsum"], args["w_enc"], args["w_dec"], args["mu_enc"],
                           args["mu_dec"], ws, ws_bytes, None)
    return st, lib.scd_last_error().decode()


def test_fit_validation(lib):
    m = _model()  # w = D = 128, two Reuse layers
    b = _batch()
    # branch, basis width, tokens
    assert _fit_gram(lib, m, b, branch=2)[0] == SHAPE
    assert _fit_gram(lib, _model(n_kv_heads=1, head_dim=32, rank_k=[16] * 3, rank_v=[16] * 3),
                     b)[0] == UNSUP  # w = 32 is not a multiple of 64
    assert _fit_gram(lib, m, _batch(n_tokens=0))[0] == SHAPE
    # pointers, RoPE table (keys only), workspace
    p, keep = _ptrs(3, skip=(2,))
    st, msg = _fit_gram(lib, m, b, b_in=p)
    assert st == NULL and "b_in[2]" in msg
    assert _fit_gram(lib, m, b, rope=None)[0] == WS
    assert _fit_gram(lib, m, b, ws=None)[0] == NULL
    assert _fit_gram(lib, m, b, ws=FAKE + 8)[0] == ALIGN
    st, msg = _fit_gram(lib, m, b, ws_bytes=1024)
    assert st == SHAPE and "workspace" in msg
    # solve
    assert _fit_solve(lib, m, branch=-1)[0] == SHAPE
    assert _fit_solve(lib, m, n_rows=0)[0] == SHAPE
    assert _fit_solve(lib, m, lam=-1.0)[0] == SHAPE
    assert _fit_solve(lib, m, lam=float("nan"))[0] == SHAPE
    assert _fit_solve(lib, m, center=2)[0] == SHAPE
    assert _fit_solve(lib, _model(rank_v=[32, 32, 24]), branch=1)[0] == SCHED
    assert _fit_solve(lib, _model(rank_k=[144, 32, 32]))[0] == SCHED  # > basis width 128
    wide = _model(n_kv_heads=18, head_dim=64, rank_k=[32] * 3, rank_v=[32] * 3)  # w = 1152 > 1024
    assert _fit_solve(lib, wide)[0] == UNSUP
    pm, keepm = _ptrs(3, skip=(0,))
    st, msg = _fit_solve(lib, m, mu_dec=pm)
    assert st == NULL and "mu_dec[0]" in msg
    # one buffer for two layers' outputs: the layers of a launch write concurrently
    same = (ctypes.c_void_p * 3)(FAKE, FAKE + 4096, FAKE)
    st, msg = _fit_gram(lib, m, b, gram=ctypes.cast(same, ctypes.POINTER(ctypes.c_void_p)))
    assert st == SHAPE and "gram[2]" in msg
    st, msg = _fit_solve(lib, m, w_dec=ctypes.cast(same, ctypes.POINTER(ctypes.c_void_p)))
    assert st == SHAPE and "w_dec[2]" in msg
    solve_need = 2 * (4 * 256 * 256 + 8 * 256) * 8  # two Reuse layers, w = 128
    st, msg = _fit_solve(lib, m, ws_bytes=solve_need - 8)
    assert st == SHAPE and "workspace" in msg


def test_fit_workspace_bytes_cover_both_calls(lib):
    # Gram partials: jobs x slices x upper tiles x (128^2 + 128) floats, slices = 1024 // units
    # capped by one per 512 rows; solve: 4 (2w)^2 + 8 (2w) doubles
    # per job.  One Reuse-only model, w = 128 (one 256 x 256 Gram = 3 upper tiles).
    # bf16 with w = 128 takes the whole-Gram kernel: one workgroup per (layer, slice), 512 // jobs
    m = _model(is_patch=[0, 0, 0])
    for T in (1, 100, 511, 512, 5000, 200000):
        units = 3
        ns = max(1, min(512 // units, -(-T // 512)))
        sr = -(-T // ns)
        sr = -(-sr // 64) * 64
        ns = -(-T // sr)
        gram = 3 * ns * 3 * (128 * 128 + 128) * 4
        solve = 3 * (4 * 256 * 256 + 8 * 256) * 8
        assert lib.scd_fit_workspace_bytes(ctypes.byref(m._c), T) == max(gram, solve)
    assert lib.scd_fit_workspace_bytes(ctypes.byref(m._c), 0) == 0


def test_fit_solve_noalloc_validation(lib):
    # The allocation-free solve validates exactly as the workspace solve, before any HIP call
    # (these run without a GPU: every case below fails validation).
    assert lib.scd_fit_solve_noalloc_max_bytes() == 64 << 20

    def call(model, branch=0, n_rows=100, lam=0.1, center=1, **over):
        L = model.n_layers
        keep, args = [], {}
        for k, name in enumerate(("gram", "colsum", "w_enc", "w_dec", "mu_enc", "mu_dec")):
            if name in over:
                args[name] = over[name]
            else:
                p, a = _distinct_ptrs(L, k)
                keep.append(a)
                args[name] = p
        st = lib.scd_fit_solve_noalloc(ctypes.byref(model._c), branch, n_rows, lam, center,
                                       args["gram"], args["colsum"], args["w_enc"],
                                       args["w_dec"], args["mu_enc"], args["mu_dec"], None)
        return st, lib.scd_last_error().decode()

    m = _model()
    assert call(m, branch=2)[0] == SHAPE
    assert call(m, n_rows=0)[0] == SHAPE
    assert call(m, lam=float("inf"))[0] == SHAPE
    assert call(m, center=3)[0] == SHAPE
    assert call(_model(rank_k=[144, 32, 32]))[0] == SCHED
    wide = _model(n_kv_heads=18, head_dim=64, rank_k=[32] * 3, rank_v=[32] * 3)  # w = 1152
    assert call(wide)[0] == UNSUP
    # w = 768: 4 (2w)^2 + 8 (2w) doubles per layer (75.6 MB) exceed the 64 MiB scratch array
    big = _model(n_kv_heads=12, head_dim=64, rank_k=[32] * 3, rank_v=[32] * 3)
    st, msg = call(big)
    assert st == WS and "scratch" in msg
    pm, keepm = _ptrs(3, skip=(2,))
    st, msg = call(m, gram=pm)
    assert st == NULL and "gram[2]" in msg
    same = (ctypes.c_void_p * 3)(FAKE, FAKE + 4096, FAKE)
    st, msg = call(m, w_enc=ctypes.cast(same, ctypes.POINTER(ctypes.c_void_p)))
    assert st == SHAPE and "w_enc[2]" in msg
    # a schedule without Reuse layers has nothing to solve and touches no device state
    assert call(_model(is_patch=[1, 1, 1]))[0] == 0


def test_fold_and_patch_from_codes_validation(lib):
    # Every case fails validation, so nothing touches a device (runs without a GPU).
    m = _model()  # layer 1 is the Patch layer (rank_h 32, d_model 256, D 128)
    b = _batch()
    L = m.n_layers

    def fold(model=m, hidden=64, **over):
        keep, args = [], {}
        for k, name in enumerate(("w2", "b2", "w_k", "w_v", "b_k", "b_v", "fk", "fv", "ck", "cv")):
            if name in over:
                args[name] = over[name]
            elif name in ("b2", "b_k", "b_v"):
                args[name] = None
            else:
                p, a = _distinct_ptrs(L, k)
                keep.append(a)
                args[name] = p
        st = lib.scd_patch_fold(ctypes.byref(model._c), hidden, *args.values(), None)
        return st, lib.scd_last_error().decode()

    assert fold(hidden=8)[0] == SHAPE
    q, keepq = _ptrs(L, skip=(1,))
    st, msg = fold(w_k=q)
    assert st == NULL and "w_k[1]" in msg
    r, keepr = _ptrs(L, value=FAKE + 8)
    assert fold(b2=r)[0] == ALIGN
    same, keeps = _ptrs(L)
    st, msg = fold(fk=same, fv=same)
    assert st == SHAPE and "share" in msg
    m2 = _model(is_patch=[1, 1, 0])
    dup = (ctypes.c_void_p * L)(FAKE, FAKE, FAKE + 4096)
    st, msg = fold(model=m2, ck=ctypes.cast(dup, ctypes.POINTER(ctypes.c_void_p)))
    assert st == SHAPE and "c_k[1]" in msg
    assert fold(model=_model(is_patch=[0, 0, 0]))[0] == OK  # no Patch layer: nothing to fold

    p, keep = _ptrs(L)

    def codes(model=m, batch=b, rope=FAKE, hidden=64, z=p, w1=p, b1=None, fk=p, fv=p, ck=None,
              cv=None, act=p, kc=p, vc=p):
        return lib.scd_patch_kv_from_codes(ctypes.byref(model._c), ctypes.byref(batch._c), rope,
                                           100, hidden, z, w1, b1, fk, fv, ck, cv, act, kc, vc,
                                           None)

    assert codes(hidden=40) == SHAPE
    assert codes(fv=q) == NULL and "w_fold_v[1]" in lib.scd_last_error().decode()
    assert codes(rope=None) == WS
    assert codes(ck=r) == ALIGN
    assert codes(model=_model(rank_h=[32, 24, 32])) == SCHED
    assert codes(z=q, act=q, kc=q, vc=q, batch=_batch(n_tokens=0)) == OK


def test_rope_table_is_checked_against_the_model(lib):
    # The binding refuses a RoPE table built for another head_dim or theta, one smaller than its
    # max_position needs, and one that is not device memory (checked before any call).
    import torch

    m = _model()  # head_dim 64, theta 1e4
    need = int(lib.scd_rope_table_bytes(ctypes.byref(m._c), 100))
    assert need == 100 * 32 * 8
    cpu = scd.RopeTable(torch.empty(need, dtype=torch.uint8), 100, m.head_dim, m.rope_theta)
    with pytest.raises(ValueError, match="CUDA"):
        scd._rope_args(cpu, m)
    other = scd.RopeTable(torch.empty(need, dtype=torch.uint8), 100, 128, m.rope_theta)
    with pytest.raises(ValueError, match="head_dim 128"):
        scd._rope_args(other, m)
    theta = scd.RopeTable(torch.empty(need, dtype=torch.uint8), 100, m.head_dim, 5e5)
    with pytest.raises(ValueError, match="theta"):
        scd._rope_args(theta, m)
    assert scd._rope_args(None, m) == (None, 0)
