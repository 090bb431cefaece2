"""GPU tests of the packed payload (Algorithm 1's transmitted code set in one buffer) and of its
streamed receipt, through the C ABI.

- Encoding straight into the packed buffer gives the same codes, bit for bit, as encoding into
  separate per-layer buffers, and they match the oracle.
- The streamed receipt (copy the payload group by group, decode each group as it lands) leaves
  the caches bit-identical to the one-call decode of the same codes, matches the oracle, delivers
  every byte of the payload (Patch codes included) and does not touch the Patch layers' caches.
"""
import pytest
import torch

import paper_2606_07684_amd as scd
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


def _packed_codes(wl, inp, dev):
    """The workload's codes (Reuse layers from the stored inputs, Patch layers' Z_H from the
    generator) copied into one packed device payload."""
    model = U.model_of(wl)
    total, _ = scd.scd_payload_bytes(model, wl.n_tokens)
    payload = torch.empty(total, dtype=torch.uint8, device=dev)
    z_k, z_v, z_h = scd.scd_payload_views(model, wl.n_tokens, payload)
    for l in inp.R:
        z_k[l].copy_(inp.z_k[l])
        z_v[l].copy_(inp.z_v[l])
    for l in inp.P:
        z_h[l].copy_(W.patch_codes(wl, l, dev))
    return payload


def _bitwise_equal(a, b):
    return torch.equal(a.view(torch.int16 if a.element_size() == 2 else torch.int32),
                       b.view(torch.int16 if b.element_size() == 2 else torch.int32))


@pytest.mark.parametrize("wl", [W.SMALL_BF16, W.SMALL_F32, W.SMALL_MANY_LAYERS],
                         ids=lambda w: w.name)
def test_encode_into_packed_payload(wl):
    print(f"case {wl.name}: T={wl.n_tokens} L={wl.n_layers}", flush=True)
    dev = torch.device("cuda")
    inp = U.Inputs(wl, dev, decode=False, patch=False)
    rope = scd.scd_rope_table(U.model_of(wl), wl.max_position)
    sep = U.run_gpu(wl, inp, rope, which=("encode",))
    model = U.model_of(wl)
    total, _ = scd.scd_payload_bytes(model, wl.n_tokens)
    payload = torch.full((total,), 0xFF, dtype=torch.uint8, device=dev)
    z_k, z_v, z_h = scd.scd_payload_views(model, wl.n_tokens, payload)
    scd.scd_encode(model, U.batch_of(wl, dev), rope, inp.k_in, inp.v_in, inp.h_in, inp.w_enc_k,
                   inp.w_enc_v, inp.w_enc_h, inp.mu_k, inp.mu_v, z_k, z_v, z_h)
    torch.cuda.synchronize()
    for l in inp.R:
        assert _bitwise_equal(z_k[l], sep["z_k"][l]) and _bitwise_equal(z_v[l], sep["z_v"][l])
    for l in inp.P:
        assert _bitwise_equal(z_h[l], sep["z_h"][l])
    errs = U.compare_all(wl, inp, {"z_k": z_k, "z_v": z_v, "z_h": z_h})
    U.assert_within(errs, U.TOL[wl.dtype], "packed encode " + wl.name)


def _receive(wl, inp, rope, payload_dev, group, source):
    dev = payload_dev.device
    if source == "pinned":
        src = torch.empty(payload_dev.numel(), dtype=torch.uint8, pin_memory=True)
        src.copy_(payload_dev)
    else:
        src = payload_dev
    dst = torch.full_like(payload_dev, 0xA5)
    kc, vc = U.alloc_caches(wl, dev, float("nan"))
    copy_stream = torch.cuda.Stream()
    scd.scd_reuse_decode_streamed(U.model_of(wl), U.batch_of(wl, dev), rope, src, dst, group,
                                  inp.w_dec_k, inp.w_dec_v, inp.mu_k, inp.mu_v, kc, vc,
                                  copy_stream=copy_stream)
    torch.cuda.synchronize()
    return dst, kc, vc


@pytest.mark.parametrize("wl,group,source", [
    (W.SMALL_BF16, 1, "pinned"), (W.SMALL_BF16, 2, "device"), (W.SMALL_F32, 1, "pinned"),
    (W.TINY_F32, 3, "device"), (W.SMALL_MANY_LAYERS, 5, "pinned"),
    (W.SMALL_MANY_LAYERS, 72, "device"), (W.SMALL_HEAD_SHARED, 1, "pinned"),
    (W.SMALL_DEGENERATE, 2, "pinned"),
], ids=lambda v: v if isinstance(v, (int, str)) else v.name)
def test_streamed_receipt_matches_one_call_decode(wl, group, source):
    print(f"case {wl.name}: group={group} source={source} T={wl.n_tokens}", flush=True)
    dev = torch.device("cuda")
    inp = U.Inputs(wl, dev, encode=False, patch=False)
    rope = scd.scd_rope_table(U.model_of(wl), wl.max_position)
    payload = _packed_codes(wl, inp, dev)
    direct = U.run_gpu(wl, inp, rope, which=("decode",), fill=float("nan"))
    dst, kc, vc = _receive(wl, inp, rope, payload, group, source)
    assert torch.equal(dst, payload), "payload bytes did not all arrive"
    for l in inp.R:
        assert _bitwise_equal(kc[l], direct["k_cache"][l]), f"k_cache[{l}]"
        assert _bitwise_equal(vc[l], direct["v_cache"][l]), f"v_cache[{l}]"
    for l in inp.P:
        assert bool(torch.isnan(kc[l]).all()) and bool(torch.isnan(vc[l]).all())
    errs = U.compare_all(wl, inp, {"k_cache": kc, "v_cache": vc})
    errs = {k: v for k, v in errs.items() if k[1] in inp.R}
    U.assert_within(errs, U.TOL[wl.dtype], f"streamed {wl.name} group {group}")


def test_streamed_receipt_full_size_from_pinned_host():
    """The receipt at the Llama-3-8B shape from pinned host memory, in the grouping the
    benchmark times; sampled rows against the oracle and every cache against the one-call decode."""
    wl = W.LLAMA3_8B
    print(f"case {wl.name}: T={wl.n_tokens} L={wl.n_layers}", flush=True)
    dev = torch.device("cuda")
    inp = U.Inputs(wl, dev, encode=False, patch=False)
    rope = scd.scd_rope_table(U.model_of(wl), wl.max_position)
    payload = _packed_codes(wl, inp, dev)
    direct = U.run_gpu(wl, inp, rope, which=("decode",))
    dst, kc, vc = _receive(wl, inp, rope, payload, scd.DEFAULT_LAYERS_PER_GROUP, "pinned")
    assert torch.equal(dst, payload)
    for l in inp.R:
        assert _bitwise_equal(kc[l], direct["k_cache"][l]), f"k_cache[{l}]"
        assert _bitwise_equal(vc[l], direct["v_cache"][l]), f"v_cache[{l}]"
    toks = U.sample_tokens(wl)
    errs = U.compare_all(wl, inp, {"k_cache": kc, "v_cache": vc}, tokens=toks)
    errs = {k: v for k, v in errs.items() if k[1] in inp.R}
    U.assert_within(errs, U.TOL[wl.dtype], "streamed " + wl.name)
    del direct, kc, vc, dst, payload, inp
    torch.cuda.empty_cache()


def test_streamed_receipt_empty_batch():
    """Zero tokens: an empty payload, a valid no-op (token-sized buffers have NULL data)."""
    wl = W.SMALL_BF16.replace(name="empty", seq_lens=(0,))
    dev = torch.device("cuda")
    inp = U.Inputs(wl, dev, encode=False, patch=False)
    src = torch.empty(0, dtype=torch.uint8, device=dev)
    dst = torch.empty(0, dtype=torch.uint8, device=dev)
    kc, vc = U.alloc_caches(wl, dev)
    scd.scd_reuse_decode_streamed(U.model_of(wl), U.batch_of(wl, dev), None, src, dst, 1,
                                  inp.w_dec_k, inp.w_dec_v, inp.mu_k, inp.mu_v, kc, vc,
                                  copy_stream=torch.cuda.Stream())
    torch.cuda.synchronize()
    assert all(c.numel() == 0 for c in kc)
