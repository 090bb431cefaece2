"""GPU parity of the offline Reuse fit (Section 4.3.1 "Joint Subspace Learning"; Appendix F.1)
against the fp64 oracle, through the C ABI.

* scd_fit_gram: the joint Gram X^T X and column sums 1^T X of the (de-rotated) paired calibration
  rows, compared whole (max |G - O| / max |O|) at the codec's tolerances: 1e-5 on the fp32 path,
  2e-2 on the bf16 path.  The Gram must also be exactly symmetric and bitwise reproducible (its
  row slices are summed in a fixed order).
* scd_fit_solve: offsets, encoder and decoder against the oracle's SVD + ridge fit, at the same
  tolerances, on workloads whose fit is well conditioned (a shared latent with distinct scales
  well above the noise): values everywhere, keys where every position is 0.  De-rotated keys at
  non-zero positions have no such structure in the synthetic caches (drawn without RoPE), so their
  eigenvectors near the cut are not unique to this precision; for them the unique quantity, the
  end-to-end map W_dec W_enc, is compared instead.
* The fitted translator carried through the codec's own encode and decode on held-out rows.
"""
import numpy as np
import pytest
import torch

import paper_2606_07684_amd as scd
from oracle import scd_oracle as O
from synth import workloads as W
from tests import parity_util as U

pytestmark = pytest.mark.gpu

BRANCHES = {"k": scd.FIT_KEYS, "v": scd.FIT_VALUES}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible MI355X")
    scd.load_library()
    yield
    torch.cuda.synchronize()


def _setup(wl, branch, dev, sample="cal"):
    L = wl.n_layers
    a_in, b_in = [None] * L, [None] * L
    R = [l for l in range(L) if not wl.is_patch[l]]
    for l in R:
        a_in[l], b_in[l] = W.fit_pair(wl, l, branch, dev, sample)
    rope = scd.scd_rope_table(U.model_of(wl), wl.max_position) if branch == "k" else None
    return R, a_in, b_in, rope


def _lam(wl):
    # ridge weight of the order of the noise's energy per direction (0.01 per row)
    return 0.05 * wl.n_tokens * wl.g


@pytest.mark.parametrize("branch", ["k", "v"])
@pytest.mark.parametrize("wl", W.FIT_WORKLOADS, ids=lambda w: w.name)
def test_fit_gram_matches_oracle(wl, branch):
    dev = torch.device("cuda")
    model, batch = U.model_of(wl), U.batch_of(wl, dev)
    R, a_in, b_in, rope = _setup(wl, branch, dev)
    L, n2 = wl.n_layers, 2 * wl.w
    gram = [torch.full((n2, n2), float("nan"), device=dev) if l in R else None for l in range(L)]
    colsum = [torch.full((n2,), float("nan"), device=dev) if l in R else None for l in range(L)]
    ws = torch.empty(scd.scd_fit_workspace_bytes(model, wl.n_tokens), dtype=torch.uint8, device=dev)
    print(f"[fit_gram] {wl.name} branch={branch} rows={wl.n_tokens * wl.g}", flush=True)
    scd.scd_fit_gram(model, batch, rope, BRANCHES[branch], a_in, b_in, gram, colsum, ws)
    torch.cuda.synchronize()
    pos = U.host_positions(wl)
    errs = {}
    for l in R:
        G, s = O.fit_gram(U.f64(a_in[l]), U.f64(b_in[l]), pos, wl.n_kv_heads, wl.head_dim,
                          wl.rope_theta, wl.w, branch == "k")
        g = gram[l].cpu()
        assert torch.equal(g, g.T), "Gram is not exactly symmetric"
        errs[("gram", l)] = U.max_abs_rel(U.f64(g), G)
        errs[("colsum", l)] = U.max_abs_rel(U.f64(colsum[l]), s)
    U.assert_within(errs, U.TOL[wl.dtype], f"fit_gram {wl.name} {branch}")
    # bitwise reproducible
    again = [torch.empty_like(t) if t is not None else None for t in gram]
    again_s = [torch.empty_like(t) if t is not None else None for t in colsum]
    scd.scd_fit_gram(model, batch, rope, BRANCHES[branch], a_in, b_in, again, again_s, ws)
    torch.cuda.synchronize()
    for l in R:
        assert torch.equal(again[l], gram[l]) and torch.equal(again_s[l], colsum[l])


def _oracle_fit(wl, branch, a_in, b_in, l, lam, center=True):
    r = wl.rank(l, branch)
    return O.fit_reuse(U.f64(a_in[l]), U.f64(b_in[l]), U.host_positions(wl), wl.n_kv_heads,
                       wl.head_dim, wl.rope_theta, wl.w, branch == "k", r, lam, center)


def _well_conditioned(wl, branch):
    return branch == "v" or wl is W.FIT_POS0_KEYS


@pytest.mark.parametrize("branch", ["k", "v"])
@pytest.mark.parametrize("wl", [*W.FIT_WORKLOADS, W.FIT_W1024_BF16], ids=lambda w: w.name)
def test_fit_solve_matches_oracle(wl, branch):
    dev = torch.device("cuda")
    model, batch = U.model_of(wl), U.batch_of(wl, dev)
    R, a_in, b_in, rope = _setup(wl, branch, dev)
    lam = _lam(wl)
    print(f"[fit_solve] {wl.name} branch={branch} lambda={lam}", flush=True)
    w_enc, w_dec, mu_enc, mu_dec, _, _ = scd.fit_reuse(model, batch, rope, BRANCHES[branch], a_in,
                                                       b_in, lam, center=True)
    torch.cuda.synchronize()
    errs = {}
    for l in R:
        e_o, d_o, ma_o, mb_o = _oracle_fit(wl, branch, a_in, b_in, l, lam)
        errs[("mu_enc", l)] = U.max_abs_rel(U.f64(mu_enc[l]), ma_o)
        errs[("mu_dec", l)] = U.max_abs_rel(U.f64(mu_dec[l]), mb_o)
        errs[("w_dec w_enc", l)] = U.max_abs_rel(U.f64(w_dec[l]) @ U.f64(w_enc[l]), d_o @ e_o)
        if _well_conditioned(wl, branch):
            errs[("w_enc", l)] = U.max_abs_rel(U.f64(w_enc[l]), e_o)
            errs[("w_dec", l)] = U.max_abs_rel(U.f64(w_dec[l]), d_o)
    U.assert_within(errs, U.TOL[wl.dtype], f"fit_solve {wl.name} {branch}")


def _rotate_complex(x, pos, n_heads, head_dim, theta):
    """RoPE written test-side as multiplication of (x_i + 1j x_{i+d/2}) by exp(1j p theta^(-2i/d))
    (the rotation itself, not the oracle's code)."""
    t, half = x.shape[0], head_dim // 2
    xh = x.reshape(t, n_heads, head_dim)
    z = xh[..., :half] + 1j * xh[..., half:]
    freq = theta ** (-2.0 * np.arange(half) / head_dim)
    zr = z * np.exp(1j * np.outer(np.asarray(pos, np.float64), freq))[:, None, :]
    return np.concatenate([zr.real, zr.imag], axis=-1).reshape(t, n_heads * head_dim)


@pytest.mark.parametrize("wl", [W.FIT_SMALL_BF16, W.FIT_HEAD_SHARED, W.FIT_F32, W.FIT_DH32,
                                W.FIT_W256_BF16, W.FIT_W64_BF16], ids=lambda w: w.name)
def test_fit_keys_from_rotated_caches(wl):
    # Key caches as a model holds them: the shared-latent content rows rotated by each token's
    # position (test-side), stored once in the model's dtype.  The fit de-rotates them back to the
    # low-rank content, so the key encoder and decoder are unique and compared directly.
    dev = torch.device("cuda")
    model, batch = U.model_of(wl), U.batch_of(wl, dev)
    L, lam = wl.n_layers, _lam(wl)
    pos = U.host_positions(wl)
    R = [l for l in range(L) if not wl.is_patch[l]]
    a_in, b_in = [None] * L, [None] * L
    for l in R:
        a_c, b_c = W.fit_pair(wl, l, "k", "cpu")
        rot = lambda x: torch.from_numpy(_rotate_complex(U.f64(x), pos, wl.n_kv_heads,  # noqa
                                                         wl.head_dim, wl.rope_theta))
        a_in[l] = rot(a_c).to(device=dev, dtype=wl.torch_dtype).contiguous()
        b_in[l] = rot(b_c).to(device=dev, dtype=wl.torch_dtype).contiguous()
    rope = scd.scd_rope_table(model, wl.max_position)
    print(f"[fit rotated keys] {wl.name} lambda={lam}", flush=True)
    w_enc, w_dec, mu_enc, mu_dec, _, _ = scd.fit_reuse(model, batch, rope, scd.FIT_KEYS, a_in,
                                                       b_in, lam, center=True)
    torch.cuda.synchronize()
    errs = {}
    for l in R:
        e_o, d_o, ma_o, mb_o = _oracle_fit(wl, "k", a_in, b_in, l, lam)
        errs[("w_enc", l)] = U.max_abs_rel(U.f64(w_enc[l]), e_o)
        errs[("w_dec", l)] = U.max_abs_rel(U.f64(w_dec[l]), d_o)
        errs[("mu_enc", l)] = U.max_abs_rel(U.f64(mu_enc[l]), ma_o)
        errs[("mu_dec", l)] = U.max_abs_rel(U.f64(mu_dec[l]), mb_o)
    U.assert_within(errs, U.TOL[wl.dtype], f"fit rotated keys {wl.name}")


def test_fit_solve_on_exact_gram_fp32():
    # The solve alone: the Gram and column sums computed in fp64 on the host (rounded once to
    # fp32), the fit's outputs in fp32 against the oracle's.
    wl = W.FIT_F32
    dev = torch.device("cuda")
    model = U.model_of(wl)
    R, a_in, b_in, _ = _setup(wl, "v", dev)
    lam = _lam(wl)
    L, n2, w = wl.n_layers, 2 * wl.w, wl.w
    gram, colsum = [None] * L, [None] * L
    w_enc, w_dec, mu_enc, mu_dec = ([None] * L for _ in range(4))
    for l in R:
        A, B = U.f64(a_in[l]).reshape(-1, w), U.f64(b_in[l]).reshape(-1, w)
        X = np.concatenate([A, B], axis=1)
        gram[l] = torch.tensor(X.T @ X, dtype=torch.float32, device=dev)
        colsum[l] = torch.tensor(X.sum(0), dtype=torch.float32, device=dev)
        r = wl.rank(l, "v")
        w_enc[l] = torch.empty((r, w), device=dev)
        w_dec[l] = torch.empty((w, r), device=dev)
        mu_enc[l] = torch.empty((w,), device=dev)
        mu_dec[l] = torch.empty((w,), device=dev)
    ws = torch.empty(scd.scd_fit_workspace_bytes(model, wl.n_tokens), dtype=torch.uint8, device=dev)
    scd.scd_fit_solve(model, scd.FIT_VALUES, wl.n_tokens * wl.g, lam, True, gram, colsum, w_enc,
                      w_dec, mu_enc, mu_dec, ws)
    torch.cuda.synchronize()
    errs = {}
    for l in R:
        e_o, d_o, ma_o, mb_o = _oracle_fit(wl, "v", a_in, b_in, l, lam)
        errs[("w_enc", l)] = U.max_abs_rel(U.f64(w_enc[l]), e_o)
        errs[("w_dec", l)] = U.max_abs_rel(U.f64(w_dec[l]), d_o)
        errs[("mu_enc", l)] = U.max_abs_rel(U.f64(mu_enc[l]), ma_o)
        errs[("mu_dec", l)] = U.max_abs_rel(U.f64(mu_dec[l]), mb_o)
    U.assert_within(errs, U.TOL["f32"], "fit_solve exact Gram f32")


def test_fitted_translator_through_the_codec():
    # Fit keys and values on calibration rows, then carry held-out producer rows through the
    # codec's own encode and Reuse decode with the fitted bases: the result must match the
    # oracle's encode/decode with the oracle's own fit, and land near the held-out consumer rows.
    wl = W.FIT_POS0_KEYS
    dev = torch.device("cuda")
    model, batch = U.model_of(wl), U.batch_of(wl, dev)
    L, lam = wl.n_layers, _lam(wl)
    fits, fits_o, held = {}, {}, {}
    for br in ("k", "v"):
        R, a_in, b_in, rope = _setup(wl, br, dev)
        fits[br] = scd.fit_reuse(model, batch, rope, BRANCHES[br], a_in, b_in, lam, center=True)
        fits_o[br] = {l: _oracle_fit(wl, br, a_in, b_in, l, lam) for l in R}
        held[br] = _setup(wl, br, dev, sample="heldout")[1:3]
    rope = scd.scd_rope_table(model, wl.max_position)
    z_k, z_v, z_h = W.alloc_codes(wl, dev)
    kc, vc = W.alloc_caches(wl, dev)
    none = [None] * L
    scd.scd_encode(model, batch, rope, held["k"][0], held["v"][0], none, fits["k"][0],
                   fits["v"][0], none, fits["k"][2], fits["v"][2], z_k, z_v, z_h)
    scd.scd_reuse_decode(model, batch, rope, z_k, z_v, fits["k"][1], fits["v"][1], fits["k"][3],
                         fits["v"][3], kc, vc)
    torch.cuda.synchronize()
    pos = U.host_positions(wl)
    H, dh, th, D = wl.n_kv_heads, wl.head_dim, wl.rope_theta, wl.kv_width
    errs = {}
    for l in R:
        ek, dk, mak, mbk = fits_o["k"][l]
        ev, dv, mav, mbv = fits_o["v"][l]
        want_k = O.decode_k(O.encode_k(U.f64(held["k"][0][l]), pos, ek, mak, H, dh, th), dk, mbk,
                            pos, H, dh, th)
        want_v = O.decode_v(O.encode_v(U.f64(held["v"][0][l]), ev, mav), dv, mbv, D)
        errs[("k_cache", l)] = U.max_abs_rel(U.f64(kc[l]), want_k)
        errs[("v_cache", l)] = U.max_abs_rel(U.f64(vc[l]), want_v)
        # the translator generalises: held-out consumer rows within the noise level
        assert U.max_abs_rel(want_v, U.f64(held["v"][1][l])) < 0.2
    U.assert_within(errs, U.TOL[wl.dtype], "fitted translator through the codec")


def test_fit_full_size_sampled_layers():
    # The calibration shape bench.py times (65,536 rows of the head-shared basis per layer): the
    # Gram of two layers per branch against the oracle, and the values' fit.
    wl = W.FIT_LLAMA3_8B
    dev = torch.device("cuda")
    model, batch = U.model_of(wl), U.batch_of(wl, dev)
    L, n2, T = wl.n_layers, 2 * wl.w, wl.n_tokens
    layers = [1, L - 1]
    ws = torch.empty(scd.scd_fit_workspace_bytes(model, T), dtype=torch.uint8, device=dev)
    pos = U.host_positions(wl)
    for br in ("k", "v"):
        a_in, b_in = [None] * L, [None] * L
        R = [l for l in range(L) if not wl.is_patch[l]]
        for l in R:
            a_in[l], b_in[l] = W.fit_pair(wl, l, br, dev)
        rope = scd.scd_rope_table(model, wl.max_position) if br == "k" else None
        print(f"[fit full size] branch={br} rows={T * wl.g} layers={len(R)}", flush=True)
        w_enc, w_dec, mu_enc, mu_dec, gram, colsum = scd.fit_reuse(
            model, batch, rope, BRANCHES[br], a_in, b_in, _lam(wl), center=True)
        torch.cuda.synchronize()
        errs = {}
        for l in layers:
            G, s = O.fit_gram(U.f64(a_in[l]), U.f64(b_in[l]), pos, wl.n_kv_heads, wl.head_dim,
                              wl.rope_theta, wl.w, br == "k")
            errs[("gram", l)] = U.max_abs_rel(U.f64(gram[l]), G)
            errs[("colsum", l)] = U.max_abs_rel(U.f64(colsum[l]), s)
            if br == "v":
                e_o, d_o, ma_o, mb_o = _oracle_fit(wl, br, a_in, b_in, l, _lam(wl))
                errs[("w_enc", l)] = U.max_abs_rel(U.f64(w_enc[l]), e_o)
                errs[("w_dec", l)] = U.max_abs_rel(U.f64(w_dec[l]), d_o)
                errs[("mu_enc", l)] = U.max_abs_rel(U.f64(mu_enc[l]), ma_o)
                errs[("mu_dec", l)] = U.max_abs_rel(U.f64(mu_dec[l]), mb_o)
        for l in R:
            assert torch.isfinite(w_enc[l]).all() and torch.isfinite(w_dec[l]).all()
        U.assert_within(errs, U.TOL[wl.dtype], f"fit full size {br}")


def test_fit_solve_contains_non_finite_input():
    # A Gram with NaN (e.g. from NaN in the caches) gives NaN outputs for its own layer only; the
    # eigenvalue ranking stays a permutation, so the solve reads nothing outside its workspace.
    wl = W.FIT_SMALL_BF16
    dev = torch.device("cuda")
    model, batch = U.model_of(wl), U.batch_of(wl, dev)
    R, a_in, b_in, _ = _setup(wl, "v", dev)
    lam = _lam(wl)
    w_enc, w_dec, mu_enc, mu_dec, gram, colsum = scd.fit_reuse(model, batch, None, scd.FIT_VALUES,
                                                               a_in, b_in, lam, center=True)
    ref = [t.clone() if t is not None else None for t in w_dec]
    bad, good = R[0], R[1]
    gram[bad][3, :] = float("nan")
    gram[bad][:, 3] = float("nan")
    ws = torch.empty(scd.scd_fit_workspace_bytes(model, wl.n_tokens), dtype=torch.uint8, device=dev)
    scd.scd_fit_solve(model, scd.FIT_VALUES, wl.n_tokens * wl.g, lam, True, gram, colsum, w_enc,
                      w_dec, mu_enc, mu_dec, ws)
    torch.cuda.synchronize()
    assert torch.isnan(w_dec[bad].float()).any()
    assert torch.equal(w_dec[good], ref[good])


@pytest.mark.parametrize("wl", [W.FIT_SMALL_BF16, W.FIT_F32], ids=lambda w: w.name)
def test_fit_without_centring_and_without_ridge(wl):
    # The paper's formulas exactly: no offsets (center = 0 writes none) and lambda = 0 (the
    # decoder is the consumer half of V_r, the encoder a least-squares fit; A^T A is non-singular
    # here because every row carries noise).
    dev = torch.device("cuda")
    model, batch = U.model_of(wl), U.batch_of(wl, dev)
    R, a_in, b_in, _ = _setup(wl, "v", dev)
    w_enc, w_dec, mu_enc, mu_dec, _, _ = scd.fit_reuse(model, batch, None, scd.FIT_VALUES, a_in,
                                                       b_in, 0.0, center=False)
    torch.cuda.synchronize()
    assert all(m is None for m in mu_enc) and all(m is None for m in mu_dec)
    # Without the ridge term the encoder solves the normal equations of A itself: the fp32
    # rounding of the accumulated Gram (about sqrt(N) u relative) reaches the result amplified by
    # cond(A^T A).  The bar is the codec's tolerance or that first-order bound, whichever is larger.
    errs, bound = {}, U.TOL[wl.dtype]
    for l in R:
        e_o, d_o, ma_o, mb_o = _oracle_fit(wl, "v", a_in, b_in, l, 0.0, center=False)
        assert ma_o is None and mb_o is None
        errs[("w_enc", l)] = U.max_abs_rel(U.f64(w_enc[l]), e_o)
        errs[("w_dec", l)] = U.max_abs_rel(U.f64(w_dec[l]), d_o)
        A = U.f64(a_in[l]).reshape(-1, wl.w)
        bound = max(bound, np.linalg.cond(A.T @ A) * np.sqrt(A.shape[0]) * 2.0 ** -24)
    print(f"[fit no centring, lambda 0] tolerance {bound:.3g}", flush=True)
    U.assert_within(errs, bound, f"fit no centring, lambda 0, {wl.name}")


def _rows_with_spectrum(n_rows, sing, seed):
    """Rows X [n_rows, n] whose Gram X^T X is Q diag(sing^2) Q^T exactly (fp64), Q random orthogonal."""
    g = np.random.default_rng(seed)
    n = len(sing)
    q, _ = np.linalg.qr(g.standard_normal((n, n)))
    u, _ = np.linalg.qr(g.standard_normal((n_rows, n)))
    return (u * np.asarray(sing)[None, :]) @ q.T


@pytest.mark.parametrize("case", ["repeated_top_eigenvalues", "rank_below_r"])
def test_fit_solve_degenerate_spectra(case):
    # Eigenvalues that repeat inside the top r (three clusters of 8, 8 and 16), or a Gram whose rank
    # (16) is below r = 32, so the solve's eigenvalue clusters are exercised.  Individual
    # eigenvectors are then not unique; W_dec W_enc is (a rotation inside a degenerate subspace
    # cancels in it, and null directions give zero latents), so that is compared with the oracle's
    # fit on the rows themselves.
    dev = torch.device("cuda")
    w, r, n_rows, lam = 64, 32, 400, 0.1
    if case == "repeated_top_eigenvalues":
        sing = np.sqrt(np.concatenate([[10.0] * 8, [7.0] * 8, [5.0] * 16,
                                       np.linspace(0.5, 0.05, 2 * w - r)]))
    else:
        sing = np.concatenate([[3.0] * 4, np.linspace(2.0, 1.0, 12), np.zeros(2 * w - 16)])
    X = _rows_with_spectrum(n_rows, sing, 7 if case == "rank_below_r" else 5)
    model = scd.Model(n_layers=1, d_model=64, n_kv_heads=1, head_dim=64, rope_theta=1e4,
                      dtype="f32", is_patch=[0], rank_k=[r], rank_v=[r], rank_h=[32],
                      basis_width=w)
    gram = [torch.tensor(X.T @ X, dtype=torch.float32, device=dev)]
    colsum = [torch.tensor(X.sum(0), dtype=torch.float32, device=dev)]
    w_enc = [torch.empty((r, w), device=dev)]
    w_dec = [torch.empty((w, r), device=dev)]
    ws = torch.empty(scd.scd_fit_workspace_bytes(model, n_rows), dtype=torch.uint8, device=dev)
    print(f"[fit degenerate] {case}", flush=True)
    scd.scd_fit_solve(model, scd.FIT_VALUES, n_rows, lam, False, gram, colsum, w_enc, w_dec,
                      [None], [None], ws)
    torch.cuda.synchronize()
    assert torch.isfinite(w_enc[0]).all() and torch.isfinite(w_dec[0]).all()
    e_o, d_o, _, _ = O.fit_reuse(X[:, :w], X[:, w:], np.zeros(n_rows, dtype=np.int64), 1, 64, 1e4,
                                 w, False, r, lam, center=False)
    err = U.max_abs_rel(U.f64(w_dec[0]) @ U.f64(w_enc[0]), d_o @ e_o)
    print(f"[fit degenerate] {case}: W_dec W_enc max-abs-rel {err:.2e}", flush=True)
    assert err <= U.TOL["f32"]


def test_fitted_bases_at_the_config1_shape_through_the_codec():
    # The configs' own bases (w = D = 1024, rank 128, 8192 tokens): fit keys (caches rotated by
    # position test-side, so the de-rotated content is low rank and the fit unique) and values
    # on calibration rows, compare the fits with the oracle's, then carry held-out producer rows
    # through the codec's encode and Reuse decode with the fitted translators (W_dec != W_enc^T)
    # against the oracle's encode and decode with its own fit.
    wl = W.FIT_CODEC_LLAMA3_8B
    dev = torch.device("cuda")
    model, batch = U.model_of(wl), U.batch_of(wl, dev)
    L, lam, pos = wl.n_layers, _lam(wl), U.host_positions(wl)
    H, dh, th, D = wl.n_kv_heads, wl.head_dim, wl.rope_theta, wl.kv_width
    rot = lambda x: _rotate_complex(U.f64(x), pos, H, dh, th)  # noqa: E731
    dev_t = lambda x: torch.from_numpy(x).to(device=dev, dtype=wl.torch_dtype).contiguous()  # noqa
    cal, held = {}, {}
    for br in ("k", "v"):
        for store, sample in ((cal, "cal"), (held, "heldout")):
            a, b = [None] * L, [None] * L
            for l in range(L):
                a_c, b_c = W.fit_pair(wl, l, br, "cpu", sample)
                a[l] = dev_t(rot(a_c)) if br == "k" else a_c.to(dev)
                b[l] = dev_t(rot(b_c)) if br == "k" else b_c.to(dev)
            store[br] = (a, b)
    rope = scd.scd_rope_table(model, wl.max_position)
    fits, errs = {}, {}
    for br, code in (("k", scd.FIT_KEYS), ("v", scd.FIT_VALUES)):
        print(f"[fit codec w=1024] fitting {br}", flush=True)
        fits[br] = scd.fit_reuse(model, batch, rope if br == "k" else None, code, *cal[br], lam,
                                 center=True)
    torch.cuda.synchronize()
    fits_o = {}
    for br in ("k", "v"):
        for l in range(L):
            e_o, d_o, ma_o, mb_o = _oracle_fit(wl, br, *cal[br], l, lam)
            fits_o[(br, l)] = (e_o, d_o, ma_o, mb_o)
            # At rank 128 the latent's scales are 0.8% apart and 8192 rows move the sample
            # eigenvalues by about 1%, so some neighbours land within the fp32 Gram's rounding of
            # each other and their eigenvectors are not unique; W_dec W_enc is (c19).
            w_enc, w_dec = fits[br][0][l], fits[br][1][l]
            errs[(br, "w_dec w_enc", l)] = U.max_abs_rel(U.f64(w_dec) @ U.f64(w_enc), d_o @ e_o)
            errs[(br, "mu_enc", l)] = U.max_abs_rel(U.f64(fits[br][2][l]), ma_o)
            errs[(br, "mu_dec", l)] = U.max_abs_rel(U.f64(fits[br][3][l]), mb_o)
    z_k, z_v, z_h = W.alloc_codes(wl, dev)
    kc, vc = W.alloc_caches(wl, dev)
    none = [None] * L
    print("[fit codec w=1024] encode and decode with the fitted bases", flush=True)
    scd.scd_encode(model, batch, rope, held["k"][0], held["v"][0], none, fits["k"][0],
                   fits["v"][0], none, fits["k"][2], fits["v"][2], z_k, z_v, z_h)
    scd.scd_reuse_decode(model, batch, rope, z_k, z_v, fits["k"][1], fits["v"][1], fits["k"][3],
                         fits["v"][3], kc, vc)
    torch.cuda.synchronize()
    for l in range(L):
        ek, dk, mak, mbk = fits_o[("k", l)]
        ev, dv, mav, mbv = fits_o[("v", l)]
        want_k = O.decode_k(O.encode_k(U.f64(held["k"][0][l]), pos, ek, mak, H, dh, th), dk, mbk,
                            pos, H, dh, th)
        want_v = O.decode_v(O.encode_v(U.f64(held["v"][0][l]), ev, mav), dv, mbv, D)
        errs[("k_cache", l)] = U.max_abs_rel(U.f64(kc[l]), want_k)
        errs[("v_cache", l)] = U.max_abs_rel(U.f64(vc[l]), want_v)
        # the fitted translator carries held-out producer rows onto the consumer's, within the noise
        assert U.max_abs_rel(want_v, U.f64(held["v"][1][l])) < 0.2
        assert U.max_abs_rel(want_k, U.f64(held["k"][1][l])) < 0.2
        assert not torch.allclose(fits["v"][1][l].float(), fits["v"][0][l].float().T)
    U.assert_within(errs, U.TOL[wl.dtype], "fitted bases at the config-1 shape")
