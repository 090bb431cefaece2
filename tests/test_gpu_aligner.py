"""GPU parity of the Patch aligner (Section 4.4.2, Eq. aligner) against the fp64 oracle, through
the C ABI: act = SiLU(Z_H W1^T + b1), H_hat = act W2^T + b2 for every Patch layer.

Tolerances as for the codec (max |G - O| / max |O| per layer and tensor): 1e-5 on the fp32 path,
2e-2 on the bf16 path, where the hidden activations are rounded to bf16 once before the second
product.
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


def _run(wl, fill=None):
    """Aligner of every Patch layer on the GPU; returns (inputs, act, h_hat) per layer."""
    dev = torch.device("cuda")
    L, T, h, d = wl.n_layers, wl.n_tokens, wl.hidden_width, wl.d_model
    z_h, w1, b1, w2, b2, act, hh = ([None] * L for _ in range(7))
    for l in wl.patch_layers:
        z_h[l] = W.patch_codes(wl, l, dev)
        w1[l], b1[l], w2[l], b2[l] = W.aligner_weights(wl, l, dev)
        act[l] = torch.empty((T, h), dtype=wl.torch_dtype, device=dev)
        hh[l] = torch.empty((T, d), dtype=wl.torch_dtype, device=dev)
        if fill is not None:
            act[l].fill_(fill)
            hh[l].fill_(fill)
    scd.scd_patch_align(U.model_of(wl), U.batch_of(wl, dev), h, z_h, w1, b1, w2, b2, act, hh)
    torch.cuda.synchronize()
    return (z_h, w1, b1, w2, b2), act, hh


def _compare(wl, inp, act, hh, tokens):
    z_h, w1, b1, w2, b2 = inp
    errs = {}
    for l in wl.patch_layers:
        want_h, want_a = O.align(U.take(z_h[l], tokens), U.f64(w1[l]), U.f64(b1[l]), U.f64(w2[l]),
                                 U.f64(b2[l]))
        errs[("act", l)] = U.max_abs_rel(U.take(act[l], tokens), want_a)
        errs[("h_hat", l)] = U.max_abs_rel(U.take(hh[l], tokens), want_h)
    return errs


@pytest.mark.parametrize("wl", [W.SMALL_ALIGN, W.SMALL_BF16, W.SMALL_F32, W.SMALL_ALIGN_RING,
                                W.SMALL_MANY_REQUESTS_ALIGN],
                         ids=lambda w: w.name)
def test_aligner_matches_oracle(wl):
    inp, act, hh = _run(wl, fill=float("nan"))
    errs = _compare(wl, inp, act, hh, np.arange(wl.n_tokens))
    U.assert_within(errs, U.TOL[wl.dtype], "aligner " + wl.name)


def test_aligner_full_size_sampled():
    wl = W.LLAMA3_8B
    inp, act, hh = _run(wl)
    errs = _compare(wl, inp, act, hh, U.sample_tokens(wl, n_random=48))
    U.assert_within(errs, U.TOL[wl.dtype], "aligner " + wl.name)


def test_aligner_rejects_shared_activation_buffer():
    wl = W.SMALL_ALIGN
    dev = torch.device("cuda")
    L, T, h, d = wl.n_layers, wl.n_tokens, wl.hidden_width, wl.d_model
    z_h, w1, b1, w2, b2, act, hh = ([None] * L for _ in range(7))
    shared = torch.empty((T, h), dtype=wl.torch_dtype, device=dev)
    for l in wl.patch_layers:
        z_h[l] = W.patch_codes(wl, l, dev)
        w1[l], b1[l], w2[l], b2[l] = W.aligner_weights(wl, l, dev)
        act[l] = shared
        hh[l] = torch.empty((T, d), dtype=wl.torch_dtype, device=dev)
    with pytest.raises(scd.ScdError) as e:
        scd.scd_patch_align(U.model_of(wl), U.batch_of(wl, dev), h, z_h, w1, b1, w2, b2, act, hh)
    assert e.value.status_name == "SCD_ERR_SHAPE"
