"""GPU parity of the HIP path against the fp64 oracle, through the C ABI.

Tolerances (max |G - O| / max |O| per layer and branch): 1e-5 on the fp32 path, 2e-2 on the
bf16 path.  Integer work (positions, routing, slot placement) is compared bit for bit.
"""
import numpy as np
import pytest
import torch

import paper_2606_07684_amd as scd
from oracle import scd_oracle as O
from synth import workloads as W
from tests import parity_util as U

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible MI355X")
    scd.load_library()
    yield
    torch.cuda.synchronize()


def _rope_for(wl):
    return scd.scd_rope_table(U.model_of(wl), wl.max_position)


def test_rope_table_is_fp64_rounded_once():
    wl = W.QWEN2_7B.replace(seq_lens=(40000,))
    tab = _rope_for(wl)
    torch.cuda.synchronize()
    got = tab.buffer.view(torch.float32).view(wl.max_position, wl.head_dim // 2, 2).cpu().numpy()
    a = O.rope_angles(np.arange(wl.max_position), wl.head_dim, wl.rope_theta)
    want_c = np.cos(a).astype(np.float32)
    want_s = np.sin(a).astype(np.float32)
    # fp64 evaluation rounded once: equal to numpy's correctly-rounded value up to one ulp
    ulp_c = np.spacing(np.abs(want_c))
    ulp_s = np.spacing(np.abs(want_s))
    assert np.all(np.abs(got[..., 0] - want_c) <= ulp_c)
    assert np.all(np.abs(got[..., 1] - want_s) <= ulp_s)
    print("rope table exact fraction:", np.mean(got[..., 0] == want_c), flush=True)


def test_rope_table_too_small_is_refused():
    wl = W.SMALL_BF16
    model = U.model_of(wl)
    tab = scd.scd_rope_table(model, 64)
    short = scd.RopeTable(tab.buffer[:-8], 64, tab.head_dim, tab.rope_theta)
    with pytest.raises(ValueError, match="needs"):
        scd._rope_args(short, model)
    assert scd._rope_args(tab, model) == (tab.buffer.data_ptr(), 64)


def test_positions_bit_exact():
    lens = [0, 5, 1, 0, 300, 17, 0]
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    p0 = np.array([3, 0, 9, 1, 1000, 7, 2], dtype=np.int32)
    for use_p0 in (False, True):
        b = scd.Batch(n_tokens=int(cu[-1]), cu_seqlens=torch.from_numpy(cu).cuda(),
                      pos0=torch.from_numpy(p0).cuda() if use_p0 else None)
        got = scd.scd_positions(b).cpu().numpy()
        want = O.positions(cu, p0 if use_p0 else None)
        assert np.array_equal(got.astype(np.int64), want)
    b = scd.Batch(n_tokens=77)
    assert np.array_equal(scd.scd_positions(b).cpu().numpy(), np.arange(77))


@pytest.mark.parametrize("wl", [W.TINY_F32, *W.TEST_WORKLOADS], ids=lambda w: w.name)
def test_full_parity_small(wl):
    print(f"case {wl.name}: T={wl.n_tokens} L={wl.n_layers}", flush=True)
    inp = U.Inputs(wl, "cuda")
    rope = _rope_for(wl)
    out = U.run_gpu(wl, inp, rope)
    errs = U.compare_all(wl, inp, out)
    U.assert_within(errs, U.TOL[wl.dtype], wl.name)


@pytest.mark.parametrize("wl", [W.SMALL_BF16, W.SMALL_HEAD_SHARED], ids=lambda w: w.name)
def test_write_once_and_routing(wl):
    """Every slot of every routed layer is written; Reuse decode leaves Patch layers alone and
    vice versa; rows past the batch are never touched."""
    dev = torch.device("cuda")
    inp = U.Inputs(wl, dev, encode=False)
    rope = _rope_for(wl)
    model, batch = U.model_of(wl), U.batch_of(wl, dev)
    T, D, guard = wl.n_tokens, wl.kv_width, 5
    big_k = [torch.full((T + guard, D), float("nan"), dtype=wl.torch_dtype, device=dev)
             for _ in range(wl.n_layers)]
    big_v = [torch.full((T + guard, D), float("nan"), dtype=wl.torch_dtype, device=dev)
             for _ in range(wl.n_layers)]
    kc = [b[:T] for b in big_k]
    vc = [b[:T] for b in big_v]
    scd.scd_reuse_decode(model, batch, rope, inp.z_k, inp.z_v, inp.w_dec_k, inp.w_dec_v,
                         inp.mu_k, inp.mu_v, kc, vc)
    torch.cuda.synchronize()
    for l in range(wl.n_layers):
        for c in (kc[l], vc[l]):
            n_nan = int(torch.isnan(c).sum())
            if wl.is_patch[l]:
                assert n_nan == T * D, f"reuse decode touched patch layer {l}"
            else:
                assert n_nan == 0, f"reuse decode left {n_nan} slots of layer {l} unwritten"
    scd.scd_patch_kv(model, batch, rope, inp.h_hat, inp.w_k, inp.w_v, inp.b_k, inp.b_v, kc, vc)
    torch.cuda.synchronize()
    for l in range(wl.n_layers):
        for big in (big_k[l], big_v[l]):
            assert int(torch.isnan(big[:T]).sum()) == 0
            assert bool(torch.isnan(big[T:]).all()), f"guard rows of layer {l} were written"


def test_deterministic_bitwise():
    wl = W.SMALL_BF16
    inp = U.Inputs(wl, "cuda")
    rope = _rope_for(wl)
    a = U.run_gpu(wl, inp, rope)
    b = U.run_gpu(wl, inp, rope)
    for key in ("k_cache", "v_cache", "z_k", "z_v", "z_h"):
        for x, y in zip(a[key], b[key]):
            if x is not None:
                assert torch.equal(x.view(torch.int16), y.view(torch.int16))


def test_empty_batch_and_reuse_only():
    wl = W.SMALL_BF16.replace(name="reuse_only", patch_layers=())
    inp = U.Inputs(wl, "cuda")
    rope = _rope_for(wl)
    out = U.run_gpu(wl, inp, rope)
    U.assert_within(U.compare_all(wl, inp, out), U.TOL["bf16"], "reuse_only")
    # zero tokens: a valid no-op; token-sized buffers are empty (NULL data pointers)
    e = wl.replace(name="empty", seq_lens=(0,), patch_layers=(1,))
    inp_e = U.Inputs(e, "cuda")
    out_e = U.run_gpu(e, inp_e, None)
    assert all(c.numel() == 0 for c in out_e["k_cache"])


@pytest.mark.parametrize("wl", [W.LLAMA3_8B, W.BATCHED], ids=lambda w: w.name)
def test_full_size_full_tensors(wl):
    """The Llama-3-8B-shaped and the batched ragged workloads at full size, launched as the
    benchmark launches them, compared with the oracle on every token of every layer (streamed
    layer by layer in chunks of 8192 tokens): caches per tensor, codes per column.  The caches
    start as NaN with guard rows past the batch: every routed slot must be written once by the
    Reuse decode or the Patch and no guard row touched."""
    print(f"case {wl.name}: T={wl.n_tokens} L={wl.n_layers} (full tensors)", flush=True)
    dev = torch.device("cuda")
    inp = U.Inputs(wl, dev)
    rope = _rope_for(wl)
    model, batch = U.model_of(wl), U.batch_of(wl, dev)
    T, D, guard = wl.n_tokens, wl.kv_width, 5
    big_k = [torch.full((T + guard, D), float("nan"), dtype=wl.torch_dtype, device=dev)
             for _ in range(wl.n_layers)]
    big_v = [torch.full((T + guard, D), float("nan"), dtype=wl.torch_dtype, device=dev)
             for _ in range(wl.n_layers)]
    kc = [b[:T] for b in big_k]
    vc = [b[:T] for b in big_v]
    z_k, z_v, z_h = U.alloc_codes(wl, dev)
    scd.scd_encode(model, batch, rope, inp.k_in, inp.v_in, inp.h_in, inp.w_enc_k, inp.w_enc_v,
                   inp.w_enc_h, inp.mu_k, inp.mu_v, z_k, z_v, z_h)
    scd.scd_reuse_decode(model, batch, rope, inp.z_k, inp.z_v, inp.w_dec_k, inp.w_dec_v,
                         inp.mu_k, inp.mu_v, kc, vc)
    scd.scd_patch_kv(model, batch, rope, inp.h_hat, inp.w_k, inp.w_v, inp.b_k, inp.b_v, kc, vc)
    torch.cuda.synchronize()
    for l in range(wl.n_layers):
        for big in (big_k[l], big_v[l]):
            assert int(torch.isnan(big[:T]).sum()) == 0, f"layer {l}: slots left unwritten"
            assert bool(torch.isnan(big[T:]).all()), f"guard rows of layer {l} were written"
    out = {"k_cache": kc, "v_cache": vc, "z_k": z_k, "z_v": z_v, "z_h": z_h}
    errs = U.compare_full_chunked(wl, inp, out, label=wl.name)
    U.assert_within(errs, U.TOL[wl.dtype], wl.name + " full tensors")
    del out, inp, big_k, big_v, kc, vc, z_k, z_v, z_h
    torch.cuda.empty_cache()


@pytest.mark.parametrize("wl", [W.QWEN2_7B, W.LLAMA3_70B, *W.MODEL_SCALE_EXTRA],
                         ids=lambda w: w.name)
def test_full_size_sampled(wl):
    """The other full-size configurations, launched exactly as the benchmark launches them; the
    oracle checks sampled token rows (random rows, request boundaries and tile edges) of every
    layer."""
    print(f"case {wl.name}: T={wl.n_tokens} L={wl.n_layers}", flush=True)
    inp = U.Inputs(wl, "cuda")
    rope = _rope_for(wl)
    out = U.run_gpu(wl, inp, rope)
    toks = U.sample_tokens(wl)
    errs = U.compare_all(wl, inp, out, tokens=toks)
    U.assert_within(errs, U.TOL[wl.dtype], wl.name)
    for key in ("k_cache", "v_cache"):
        for c in out[key]:
            assert bool(torch.isfinite(c).all())
    del out, inp
    torch.cuda.empty_cache()


def test_full_rank_round_trip_reproduces_the_input():
    """r = w with an orthonormal basis (W_enc = Q^T, W_dec = Q) and the same offset on both sides:
    decoding the GPU's own codes returns the producer's K and V (keys through deRoPE then RoPE), up
    to the bf16 roundings of the codes and the output (Section 4.3.2)."""
    wl = W.SMALL_FULL_RANK
    inp = U.Inputs(wl, "cuda")
    rope = _rope_for(wl)
    enc = U.run_gpu(wl, inp, rope, which=("encode",))
    model, batch = U.model_of(wl), U.batch_of(wl, torch.device("cuda"))
    kc, vc = U.alloc_caches(wl, torch.device("cuda"))
    scd.scd_reuse_decode(model, batch, rope, enc["z_k"], enc["z_v"], inp.w_dec_k, inp.w_dec_v,
                         inp.mu_k, inp.mu_v, kc, vc)
    torch.cuda.synchronize()
    worst = 0.0
    for l in inp.R:
        for got, want in ((kc[l], inp.k_in[l]), (vc[l], inp.v_in[l])):
            worst = max(worst, U.max_abs_rel(U.f64(got), U.f64(want)))
    print(f"full-rank round trip, worst max-abs-rel {worst:.2e}", flush=True)
    assert worst <= U.TOL["bf16"]
