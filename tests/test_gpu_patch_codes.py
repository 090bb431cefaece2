"""GPU parity of the consumer's Patch from the transmitted codes (Section 4.4.2: Eq. aligner then
Eq. kv_from_patch) with the aligner's output layer folded into the projections, through the C ABI.

* scd_patch_fold: w_fold = W_P W2 and c = W_P b2 + b_P against the oracle's fold in fp64.
* scd_patch_kv_from_codes: the regenerated K/V against the oracle's literal chain
  H_hat = SiLU(Z_H W1^T + b1) W2^T + b2, K = RoPE(H_hat W_K^T + b_K), V = H_hat W_V^T + b_V, which
  never folds anything.  The GPU side takes only the GPU's own fold of the same stored weights.
  Caches start as NaN: every Patch slot must be written and no Reuse layer touched.  Either one act
  buffer serves every Patch layer (the call runs the layers one after another) or each layer has
  its own (the call runs them together).

Tolerances as everywhere (max |G - O| / max |O| per layer and tensor): 1e-5 fp32, 2e-2 bf16.
"""
import numpy as np
import pytest
import torch

import paper_2606_07684_amd as scd
from oracle import scd_oracle as O
from synth import workloads as W
from tests import parity_util as U

pytestmark = pytest.mark.gpu

SMALL = [W.SMALL_ALIGN, W.SMALL_ALIGN_RING, W.SMALL_F32, W.SMALL_RING5, W.SMALL_HEAD_SHARED,
         W.SMALL_DEGENERATE, W.SMALL_BF16, W.SMALL_MANY_REQUESTS_ALIGN]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible MI355X")
    scd.load_library()
    yield
    torch.cuda.synchronize()


@pytest.mark.parametrize("shared", [True, False], ids=["shared_act", "act_per_layer"])
@pytest.mark.parametrize("wl", SMALL, ids=lambda w: w.name)
def test_fold_and_patch_from_codes_match_oracle(wl, shared):
    print(f"[patch_codes] {wl.name} shared_act={shared}", flush=True)
    s = U.PatchFromCodes(wl, shared_act=shared)
    U.assert_within(s.fold_errors(), U.TOL[wl.dtype], "fold " + wl.name)
    U.assert_within(s.cache_errors(np.arange(wl.n_tokens)), U.TOL[wl.dtype],
                    "patch from codes " + wl.name)
    # Reuse layers are not touched (still the NaN fill)
    for l in range(wl.n_layers):
        if not wl.is_patch[l]:
            assert torch.isnan(s.kc[l].float()).all() and torch.isnan(s.vc[l].float()).all()


def test_patch_from_codes_full_size_full_tensors():
    # the benchmark's Patch phase at the Llama-3-8B shape (one act buffer per layer), every token
    wl = W.LLAMA3_8B
    print(f"[patch_codes] {wl.name} full tensors", flush=True)
    s = U.PatchFromCodes(wl, shared_act=False)
    U.assert_within(s.fold_errors(), U.TOL[wl.dtype], "fold " + wl.name)
    U.assert_within(s.cache_errors(np.arange(wl.n_tokens)), U.TOL[wl.dtype],
                    "patch from codes " + wl.name)
    for l in range(wl.n_layers):  # Reuse layers untouched
        if not wl.is_patch[l]:
            assert torch.isnan(s.kc[l][:64].float()).all()


@pytest.mark.parametrize("wl", [W.QWEN2_7B, W.BATCHED, W.LLAMA3_70B], ids=lambda w: w.name)
def test_patch_from_codes_full_size_sampled(wl):
    print(f"[patch_codes] {wl.name} sampled", flush=True)
    s = U.PatchFromCodes(wl, fill=0.0, shared_act=False)
    U.assert_within(s.fold_errors(), U.TOL[wl.dtype], "fold " + wl.name)
    U.assert_within(s.cache_errors(U.sample_tokens(wl, n_random=48)), U.TOL[wl.dtype],
                    "patch from codes " + wl.name)
    del s
    torch.cuda.empty_cache()


def test_patch_from_codes_equals_align_then_patch_kv():
    # The folded path against the library's own unfolded path (scd_patch_align, then
    # scd_patch_kv on its H_hat): both approximate the same fp64 chain within the bf16 budget.
    wl = W.SMALL_ALIGN
    dev = torch.device("cuda")
    s = U.PatchFromCodes(wl)
    L, T, h, d = wl.n_layers, wl.n_tokens, wl.hidden_width, wl.d_model
    act = [torch.empty((T, h), dtype=wl.torch_dtype, device=dev) if wl.is_patch[l] else None
           for l in range(L)]
    hh = [torch.empty((T, d), dtype=wl.torch_dtype, device=dev) if wl.is_patch[l] else None
          for l in range(L)]
    scd.scd_patch_align(s.model, s.batch, h, s.z_h, s.w1, s.b1, s.w2, s.b2, act, hh)
    kc, vc = U.alloc_caches(wl, dev, float("nan"))
    scd.scd_patch_kv(s.model, s.batch, s.rope, hh, s.w_k, s.w_v, s.b_k, s.b_v, kc, vc)
    torch.cuda.synchronize()
    errs = {}
    for l in wl.patch_layers:
        errs[("k", l)] = U.max_abs_rel(U.f64(s.kc[l]), U.f64(kc[l]))
        errs[("v", l)] = U.max_abs_rel(U.f64(s.vc[l]), U.f64(vc[l]))
    U.assert_within(errs, 2 * U.TOL[wl.dtype], "folded vs unfolded " + wl.name)
