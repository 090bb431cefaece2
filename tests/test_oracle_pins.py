"""Pins of the fp64 oracle against what the mathematics and the paper fix.

None of these re-type the oracle's formulas: RoPE is checked against complex multiplication,
a matrix exponential, closed-form points and its group properties; the linear maps against
explicit loops, exact round trips, in-subspace recovery and the Eckart-Young tail energy.
"""
import math

import numpy as np
import pytest
import scipy.linalg

from oracle import scd_oracle as O



# ------------------------------------------------------------------------------------------
# Independent RoPE formulations (test-side)
# ------------------------------------------------------------------------------------------
def rope_complex(x, pos, n_heads, head_dim, theta, sign=1.0):
    """RoPE as multiplication of (x_i + 1j x_{i+d/2}) by exp(1j * sign * p * theta^(-2i/d))."""
    t = x.shape[0]
    half = head_dim // 2
    xh = np.asarray(x, np.float64).reshape(t, n_heads, head_dim)
    z = xh[..., :half] + 1j * xh[..., half:]
    freq = np.array([theta ** (-2.0 * i / head_dim) for i in range(half)])
    ph = np.exp(1j * sign * np.outer(np.asarray(pos, np.float64), freq))[:, None, :]
    zr = z * ph
    return np.concatenate([zr.real, zr.imag], axis=-1).reshape(t, n_heads * head_dim)


def rope_expm_head(vec, p, head_dim, theta):
    """RoPE of one head vector as expm(p * G) @ vec with G the skew generator of the rotation."""
    half = head_dim // 2
    g = np.zeros((head_dim, head_dim))
    for i in range(half):
        om = theta ** (-2.0 * i / head_dim)
        g[i + half, i] = om
        g[i, i + half] = -om
    return scipy.linalg.expm(p * g) @ vec


def rand_orthonormal(rng, n, k):
    q, r = np.linalg.qr(rng.standard_normal((n, k)))
    return q * np.sign(np.diag(r))[None, :]


# ------------------------------------------------------------------------------------------
# a0 routing and payload
# ------------------------------------------------------------------------------------------
def test_schedule_partitions_layers():
    rng = np.random.default_rng(0)
    for _ in range(20):
        L = int(rng.integers(1, 90))
        flags = rng.integers(0, 2, L)
        reuse, patch = O.schedule(flags)
        assert sorted(reuse + patch) == list(range(L))
        assert not set(reuse) & set(patch)
        assert all(flags[l] for l in patch) and not any(flags[l] for l in reuse)
        assert reuse == sorted(reuse) and patch == sorted(patch)


def test_schedule_reuse_only_and_patch_every_8th():
    # "Reuse-only" is the empty Patch set (Section 6.1 baselines).
    reuse, patch = O.schedule([0] * 32)
    assert reuse == list(range(32)) and patch == []
    reuse, patch = O.schedule([1 if l % 8 == 0 else 0 for l in range(32)])
    assert patch == [0, 8, 16, 24] and len(reuse) == 28


def test_payload_closed_form_and_offsets():
    L, T, H, dh = 6, 37, 4, 16
    D = H * dh
    flags = [1, 0, 0, 1, 0, 0]
    rk = [8, 16, 24, 32, 8, 16]
    rv = [16, 16, 8, 8, 8, 32]
    rh = [40, 8, 8, 24, 8, 8]
    for w in (D, dh):
        g = D // w
        total, offs = O.payload_bytes(flags, T, H, dh, w, rk, rv, rh, 2)
        expect = 0
        for l in range(L):
            n = T * rh[l] if flags[l] else T * g * (rk[l] + rv[l])
            assert offs[l + 1] - offs[l] == 2 * n
            expect += 2 * n
        assert total == expect == offs[-1] and offs[0] == 0


def test_payload_full_rank_identity_equals_raw_kv():
    # With r = w (no compression) and no Patch layers the code set is exactly the raw cache.
    L, T, H, dh = 5, 11, 2, 8
    D = H * dh
    for w in (D, dh):
        total, _ = O.payload_bytes([0] * L, T, H, dh, w, [w] * L, [w] * L, [1] * L, 2)
        assert total == 2 * L * T * D * 2


def test_payload_is_linear_in_tokens_and_rank():
    # O(T r) transmission (Section 4.5).
    base, _ = O.payload_bytes([0, 1], 100, 8, 128, 1024, [64, 64], [64, 64], [64, 64], 2)
    twice_t, _ = O.payload_bytes([0, 1], 200, 8, 128, 1024, [64, 64], [64, 64], [64, 64], 2)
    twice_r, _ = O.payload_bytes([0, 1], 100, 8, 128, 1024, [128] * 2, [128] * 2, [128] * 2, 2)
    assert twice_t == 2 * base and twice_r == 2 * base


def test_payload_equals_the_encoded_code_set():
    # Algorithm 1 transmits exactly the producer's codes: {Z_K, Z_V} of every Reuse layer and Z_H
    # of every Patch layer, in layer order, K before V.  Encode a tiny model with the oracle and
    # lay its actual outputs end to end: their byte sizes must be the payload's offsets, for the
    # full-width basis and the head-shared one, with Patch layers and ranks that differ by layer
    # and branch.
    rng = np.random.default_rng(7)
    T, H, dh, d, theta = 13, 2, 8, 24, 1e4
    D = H * dh
    flags = [0, 1, 0, 0, 1]
    pos = np.arange(T)
    for w in (D, dh):
        g = D // w
        rk = [int(v) for v in rng.integers(1, w + 1, len(flags))]
        rv = [int(v) for v in rng.integers(1, w + 1, len(flags))]
        rh = [int(v) for v in rng.integers(1, d + 1, len(flags))]
        L = len(flags)
        k_a = [rng.standard_normal((T, D)) for _ in range(L)]
        v_a = [rng.standard_normal((T, D)) for _ in range(L)]
        h_a = [rng.standard_normal((T, d)) for _ in range(L)]
        e_k = [rng.standard_normal((rk[l], w)) for l in range(L)]
        e_v = [rng.standard_normal((rv[l], w)) for l in range(L)]
        e_h = [rng.standard_normal((rh[l], d)) for l in range(L)]
        z_k, z_v, z_h = O.encode_all(flags, pos, H, dh, theta, k_a, v_a, h_a, e_k, e_v, e_h)
        sent = []
        for l in range(L):
            sent += [z_h[l]] if flags[l] else [z_k[l], z_v[l]]
        assert all(z is not None for z in sent), "a routed branch produced no code"
        for eb in (2, 4):
            total, offs = O.payload_bytes(flags, T, H, dh, w, rk, rv, rh, eb)
            ends = np.cumsum([0] + [z.size * eb for z in sent])
            per_layer = [0]
            i = 0
            for l in range(L):
                i += 1 if flags[l] else 2
                per_layer.append(int(ends[i]))
            assert offs == per_layer and total == int(ends[-1])
            assert all(z.shape[0] == (T if flags[l] else T * g)
                       for l, z in zip([l for l in range(L) for _ in range(1 if flags[l] else 2)],
                                       sent))


# ------------------------------------------------------------------------------------------
# a1 positions
# ------------------------------------------------------------------------------------------
def test_positions_match_brute_force():
    rng = np.random.default_rng(1)
    for _ in range(10):
        lens = rng.integers(0, 40, int(rng.integers(1, 8)))
        cu = np.concatenate([[0], np.cumsum(lens)])
        p0 = rng.integers(0, 1000, len(lens))
        for use_p0 in (False, True):
            got = O.positions(cu, p0 if use_p0 else None)
            want = []
            for b, n in enumerate(lens):
                for k in range(n):
                    want.append(k + (int(p0[b]) if use_p0 else 0))
            assert got.tolist() == want


# ------------------------------------------------------------------------------------------
# RoPE
# ------------------------------------------------------------------------------------------
def test_rope_closed_form_points():
    # theta = 1e4, d_h = 4: frequencies 1 and 0.01 rad per position.
    e = np.eye(4)
    out = O.rope(e[[0]], [1], 1, 4, 1e4)[0]
    np.testing.assert_allclose(out, [math.cos(1), 0, math.sin(1), 0], atol=1e-15)
    out = O.rope(e[[1]], [3], 1, 4, 1e4)[0]
    np.testing.assert_allclose(out, [0, math.cos(0.03), 0, math.sin(0.03)], atol=1e-15)
    out = O.rope(e[[2]], [2], 1, 4, 1e4)[0]
    np.testing.assert_allclose(out, [-math.sin(2), 0, math.cos(2), 0], atol=1e-15)
    # d_h = 2 is a plain 2-D rotation by p radians.
    out = O.rope(np.array([[0.3, -0.7]]), [5], 1, 2, 123.0)[0]
    c, s = math.cos(5), math.sin(5)
    np.testing.assert_allclose(out, [0.3 * c + 0.7 * s, -0.7 * c + 0.3 * s], atol=1e-15)


def test_rope_matches_complex_and_expm():
    rng = np.random.default_rng(2)
    H, dh, theta = 3, 16, 5e5
    x = rng.standard_normal((7, H * dh))
    pos = rng.integers(0, 40000, 7)
    np.testing.assert_allclose(O.rope(x, pos, H, dh, theta), rope_complex(x, pos, H, dh, theta),
                               atol=1e-12)
    np.testing.assert_allclose(O.rope(x, pos, H, dh, theta, inverse=True),
                               rope_complex(x, pos, H, dh, theta, sign=-1.0), atol=1e-12)
    y = O.rope(x, pos, H, dh, theta)
    for t in range(2):
        for h in range(H):
            np.testing.assert_allclose(y[t, h * dh:(h + 1) * dh],
                                       rope_expm_head(x[t, h * dh:(h + 1) * dh], pos[t], dh,
                                                      theta), atol=1e-9)


def test_rope_group_properties():
    rng = np.random.default_rng(3)
    H, dh, theta = 2, 32, 1e4
    x = rng.standard_normal((9, H * dh))
    pos = rng.integers(0, 5000, 9)
    y = O.rope(x, pos, H, dh, theta)
    # norm of every (u, v) pair is preserved
    half = dh // 2
    xp = x.reshape(9, H, dh)
    yp = y.reshape(9, H, dh)
    np.testing.assert_allclose(xp[..., :half] ** 2 + xp[..., half:] ** 2,
                               yp[..., :half] ** 2 + yp[..., half:] ** 2, rtol=1e-12)
    # deRoPE o RoPE = id, RoPE at position 0 = id
    np.testing.assert_allclose(O.rope(y, pos, H, dh, theta, inverse=True), x, atol=1e-12)
    np.testing.assert_allclose(O.rope(x, np.zeros(9, int), H, dh, theta), x, atol=0)
    # relative position: <RoPE_m q, RoPE_n k> = <RoPE_{m-n} q, k>
    q = rng.standard_normal((1, dh))
    k = rng.standard_normal((1, dh))
    for m, n in [(7, 3), (1000, 999), (4, 4), (30000, 12)]:
        lhs = float((O.rope(q, [m], 1, dh, theta) @ O.rope(k, [n], 1, dh, theta).T)[0, 0])
        rhs = float((O.rope(q, [m - n], 1, dh, theta) @ k.T)[0, 0])
        assert abs(lhs - rhs) < 1e-9 * (1 + abs(rhs))


def test_rope_composes_additively():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((5, 64))
    a = rng.integers(0, 3000, 5)
    b = rng.integers(0, 3000, 5)
    two = O.rope(O.rope(x, a, 2, 32, 1e6), b, 2, 32, 1e6)
    np.testing.assert_allclose(two, O.rope(x, a + b, 2, 32, 1e6), atol=1e-11)


# ------------------------------------------------------------------------------------------
# Linear maps: brute force on tiny inputs
# ------------------------------------------------------------------------------------------
def _loop_matmul_t(x, w):
    """x[n, k] @ w[m, k]^T with explicit loops."""
    n, k = x.shape
    m = w.shape[0]
    out = np.zeros((n, m))
    for i in range(n):
        for j in range(m):
            s = 0.0
            for q in range(k):
                s += float(x[i, q]) * float(w[j, q])
            out[i, j] = s
    return out


@pytest.mark.parametrize("w_is_head", [False, True])
def test_encode_decode_brute_force(w_is_head):
    rng = np.random.default_rng(5)
    H, dh, theta = 2, 4, 1e4
    D = H * dh
    w = dh if w_is_head else D
    g = D // w
    T, r = 5, 3
    pos = np.array([0, 1, 2, 0, 7])
    k = rng.standard_normal((T, D))
    v = rng.standard_normal((T, D))
    e = rng.standard_normal((r, w))
    f = rng.standard_normal((w, r))
    mu_e = rng.standard_normal(w)
    mu_d = rng.standard_normal(w)
    # encode K: deRoPE by the complex formulation, then row loop
    kc = rope_complex(k, pos, H, dh, theta, sign=-1.0)
    rows = []
    for t in range(T):
        for j in range(g):
            rows.append(kc[t, j * w:(j + 1) * w] - mu_e)
    want_zk = _loop_matmul_t(np.array(rows), e)
    np.testing.assert_allclose(O.encode_k(k, pos, e, mu_e, H, dh, theta), want_zk, atol=1e-12)
    rows = [v[t, j * w:(j + 1) * w] - mu_e for t in range(T) for j in range(g)]
    np.testing.assert_allclose(O.encode_v(v, e, mu_e), _loop_matmul_t(np.array(rows), e),
                               atol=1e-12)
    # decode: row loop, un-reshape, then RoPE via complex formulation
    z = rng.standard_normal((T * g, r))
    y = _loop_matmul_t(z, f) + mu_d[None, :]
    tok = np.zeros((T, D))
    for t in range(T):
        for j in range(g):
            tok[t, j * w:(j + 1) * w] = y[t * g + j]
    np.testing.assert_allclose(O.decode_v(z, f, mu_d, D), tok, atol=1e-12)
    np.testing.assert_allclose(O.decode_k(z, f, mu_d, pos, H, dh, theta),
                               rope_complex(tok, pos, H, dh, theta), atol=1e-12)


def test_patch_brute_force_and_encode_h():
    rng = np.random.default_rng(6)
    H, dh, d, T, theta = 2, 4, 5, 4, 1e4
    D = H * dh
    pos = np.array([3, 0, 1, 2])
    hh = rng.standard_normal((T, d))
    wk = rng.standard_normal((D, d))
    wv = rng.standard_normal((D, d))
    bk = rng.standard_normal(D)
    bv = rng.standard_normal(D)
    np.testing.assert_allclose(O.patch_v(hh, wv, bv), _loop_matmul_t(hh, wv) + bv, atol=1e-12)
    np.testing.assert_allclose(O.patch_k(hh, wk, bk, pos, H, dh, theta),
                               rope_complex(_loop_matmul_t(hh, wk) + bk, pos, H, dh, theta),
                               atol=1e-12)
    eh = rng.standard_normal((3, d))
    np.testing.assert_allclose(O.encode_h(hh, eh), _loop_matmul_t(hh, eh), atol=1e-12)


# ------------------------------------------------------------------------------------------
# Linear maps: exact structural results
# ------------------------------------------------------------------------------------------
@pytest.mark.parametrize("w_is_head", [False, True])
def test_full_rank_orthonormal_round_trip(w_is_head):
    rng = np.random.default_rng(7)
    H, dh, theta = 4, 16, 5e5
    D = H * dh
    w = dh if w_is_head else D
    cu = [0, 13, 14, 40]
    pos = O.positions(cu, [0, 5, 100])
    T = cu[-1]
    q = rand_orthonormal(rng, w, w)
    mu = rng.standard_normal(w)
    k = rng.standard_normal((T, D))
    v = rng.standard_normal((T, D))
    zk = O.encode_k(k, pos, q.T, mu, H, dh, theta)
    zv = O.encode_v(v, q.T, mu)
    np.testing.assert_allclose(O.decode_k(zk, q, mu, pos, H, dh, theta), k, atol=1e-12)
    np.testing.assert_allclose(O.decode_v(zv, q, mu, D), v, atol=1e-12)


def test_in_subspace_recovery():
    rng = np.random.default_rng(8)
    H, dh, theta, r = 2, 32, 1e4, 12
    D = H * dh
    T = 50
    pos = np.arange(T) * 37
    q = rand_orthonormal(rng, D, r)
    mu = rng.standard_normal(D)
    c = rng.standard_normal((T, r))
    content = mu[None, :] + c @ q.T
    k_a = rope_complex(content, pos, H, dh, theta)
    np.testing.assert_allclose(O.encode_k(k_a, pos, q.T, mu, H, dh, theta), c, atol=1e-12)
    np.testing.assert_allclose(O.decode_k(c, q, mu, pos, H, dh, theta), k_a, atol=1e-12)
    np.testing.assert_allclose(O.encode_v(content, q.T, mu), c, atol=1e-12)
    np.testing.assert_allclose(O.decode_v(c, q, mu, D), content, atol=1e-12)


def test_invertible_nonorthogonal_pair_is_identity():
    rng = np.random.default_rng(9)
    H, dh, theta = 1, 8, 1e4
    e = rng.standard_normal((8, 8)) + 3 * np.eye(8)
    f = np.linalg.inv(e)
    x = rng.standard_normal((6, 8))
    pos = np.arange(6)
    z = O.encode_k(x, pos, e, None, H, dh, theta)
    np.testing.assert_allclose(O.decode_k(z, f, None, pos, H, dh, theta), x, atol=1e-10)
    np.testing.assert_allclose(O.decode_v(O.encode_v(x, e, None), f, None, 8), x, atol=1e-10)


def test_zero_code_gives_offset():
    rng = np.random.default_rng(10)
    H, dh, theta = 2, 8, 1e4
    D = H * dh
    mu = rng.standard_normal(D)
    pos = np.array([0, 4, 9])
    z = np.zeros((3, 5))
    f = rng.standard_normal((D, 5))
    np.testing.assert_allclose(O.decode_v(z, f, mu, D), np.tile(mu, (3, 1)), atol=0)
    np.testing.assert_allclose(O.decode_k(z, f, mu, pos, H, dh, theta),
                               rope_complex(np.tile(mu, (3, 1)), pos, H, dh, theta), atol=1e-14)


@pytest.mark.parametrize("branch", ["k", "v"])
def test_eckart_young_tail_energy(branch):
    # Truncated SVD is the best rank-r approximation (Appendix F.1, Eckart-Young-Mirsky): with an
    # exact synthetic SVD X - mu = U diag(s) B^T and the top-r right singular vectors as basis,
    # the squared reconstruction error is the sum of the discarded squared singular values.
    rng = np.random.default_rng(11)
    H, dh, theta, r = 2, 16, 5e5, 9
    D = H * dh
    T = 80
    u = rand_orthonormal(rng, T, D)
    b = rand_orthonormal(rng, D, D)
    s = np.sort(rng.uniform(0.1, 5.0, D))[::-1]
    mu = rng.standard_normal(D)
    content = mu[None, :] + (u * s[None, :]) @ b.T
    pos = np.arange(T) + 11
    qb = b[:, :r]
    if branch == "k":
        x = rope_complex(content, pos, H, dh, theta)
        xr = O.decode_k(O.encode_k(x, pos, qb.T, mu, H, dh, theta), qb, mu, pos, H, dh, theta)
    else:
        x = content
        xr = O.decode_v(O.encode_v(x, qb.T, mu), qb, mu, D)
    err = np.sum((x - xr) ** 2)
    np.testing.assert_allclose(err, np.sum(s[r:] ** 2), rtol=1e-10)
    # and any other rank-r orthonormal basis does no better
    qo = rand_orthonormal(rng, D, r)
    if branch == "v":
        xo = O.decode_v(O.encode_v(x, qo.T, mu), qo, mu, D)
        assert np.sum((x - xo) ** 2) >= err


def test_patch_identity_and_bias_only():
    rng = np.random.default_rng(12)
    H, dh, theta = 2, 8, 1e4
    D = H * dh
    T = 6
    pos = np.array([0, 1, 2, 3, 100, 5000])
    hh = rng.standard_normal((T, D))
    eye = np.eye(D)
    np.testing.assert_allclose(O.patch_v(hh, eye, None), hh, atol=0)
    np.testing.assert_allclose(O.patch_k(hh, eye, None, pos, H, dh, theta),
                               rope_complex(hh, pos, H, dh, theta), atol=1e-14)
    b = rng.standard_normal(D)
    zero = np.zeros((D, 7))
    h7 = rng.standard_normal((T, 7))
    np.testing.assert_allclose(O.patch_v(h7, zero, b), np.tile(b, (T, 1)), atol=0)
    np.testing.assert_allclose(O.patch_k(h7, zero, b, pos, H, dh, theta),
                               rope_complex(np.tile(b, (T, 1)), pos, H, dh, theta), atol=1e-14)


def test_whole_model_routing_and_assembly():
    rng = np.random.default_rng(13)
    L, H, dh, d, theta = 5, 2, 8, 12, 1e4
    D = H * dh
    flags = [0, 1, 0, 0, 1]
    T = 9
    pos = np.arange(T)
    r = 4
    z = [rng.standard_normal((T, r)) for _ in range(L)]
    f = [rng.standard_normal((D, r)) for _ in range(L)]
    hh = [rng.standard_normal((T, d)) for _ in range(L)]
    wk = [rng.standard_normal((D, d)) for _ in range(L)]
    rk, rv = O.reuse_decode_all(flags, pos, H, dh, theta, z, z, f, f)
    pk, pv = O.patch_all(flags, pos, H, dh, theta, hh, wk, wk)
    ck, cv = O.assemble(flags, (rk, rv), (pk, pv))
    for l in range(L):
        assert ck[l] is not None and cv[l] is not None  # every layer filled: T_fill = 0
        if flags[l]:
            assert rk[l] is None and pk[l] is not None
            np.testing.assert_allclose(cv[l], hh[l] @ wk[l].T)
        else:
            assert pk[l] is None and rk[l] is not None
            np.testing.assert_allclose(cv[l], z[l] @ f[l].T)


# ------------------------------------------------------------------------------------------
# Patch aligner (Section 4.4.2, Eq. aligner): H_hat = W2 SiLU(W1 z + b1) + b2 (the MLP reading)
# ------------------------------------------------------------------------------------------
def test_silu_closed_forms():
    # sigmoid(1) = 1 / (1 + 1/e); SiLU(x) = x (1 + tanh(x / 2)) / 2 (an independent formulation)
    # (well conditioned for |x| <= 8; 1 + tanh(x/2) cancels further out)
    xs = np.array([-7.5, -3.5, -1.0, -1e-3, 0.0, 1e-3, 0.5, 1.0, 2.0, 7.25])
    want = np.array([x * (1.0 + math.tanh(x / 2.0)) / 2.0 for x in xs])
    np.testing.assert_allclose(O.silu(xs), want, rtol=1e-13, atol=1e-300)
    # far out: SiLU(x) = x e^x (1 - e^x + ...) for x -> -inf and x - x e^-x (1 - ...) for x -> inf
    for x in (-30.0, -45.0):
        assert abs(O.silu(np.array([x]))[0] - x * math.exp(x)) <= 1e-12 * abs(x * math.exp(x))
    for x in (30.0, 45.0):
        assert abs(O.silu(np.array([x]))[0] - (x - x * math.exp(-x))) <= 1e-15 * x
    assert abs(O.silu(np.array([1.0]))[0] - 1.0 / (1.0 + math.exp(-1.0))) < 1e-15
    # SiLU(x) - SiLU(-x) = x; the derivative at 0 is 1/2; no overflow far out
    x = np.linspace(-40.0, 40.0, 161)
    np.testing.assert_allclose(O.silu(x) - O.silu(-x), x, atol=1e-12)
    h = 1e-6
    assert abs((O.silu(np.array([h]))[0] - O.silu(np.array([-h]))[0]) / (2 * h) - 0.5) < 1e-9
    far = O.silu(np.array([-800.0, 800.0]))
    assert np.all(np.isfinite(far)) and far[0] == 0.0 and far[1] == 800.0


def test_align_brute_force():
    rng = np.random.default_rng(41)
    t, r, hid, d = 3, 4, 5, 6
    z = rng.standard_normal((t, r))
    w1, b1 = rng.standard_normal((hid, r)), rng.standard_normal(hid)
    w2, b2 = rng.standard_normal((d, hid)), rng.standard_normal(d)
    y, act = O.align(z, w1, b1, w2, b2)
    for i in range(t):
        a = []
        for j in range(hid):
            s = b1[j]
            for k in range(r):
                s += z[i, k] * w1[j, k]
            a.append(s / (1.0 + math.exp(-s)))
            assert abs(act[i, j] - a[j]) < 1e-12
        for c in range(d):
            s = b2[c]
            for j in range(hid):
                s += a[j] * w2[c, j]
            assert abs(y[i, c] - s) < 1e-12
    # absent biases are zero biases
    y0, _ = O.align(z, w1, None, w2, None)
    y1, _ = O.align(z, w1, np.zeros(hid), w2, np.zeros(d))
    np.testing.assert_array_equal(y0, y1)


def test_align_linear_limit_and_zero_output_layer():
    # with W1 = I and a large positive shift SiLU is the identity to within 60 e^-60, so the
    # aligner is the affine map W2 (z + c) + b2
    rng = np.random.default_rng(43)
    t, r, d, c = 7, 8, 5, 60.0
    z = rng.standard_normal((t, r))
    w2, b2 = rng.standard_normal((d, r)), rng.standard_normal(d)
    y, _ = O.align(z, np.eye(r), np.full(r, c), w2, b2)
    np.testing.assert_allclose(y, (z + c) @ w2.T + b2, rtol=1e-12, atol=1e-9)
    # a zero output layer leaves only its bias
    w1 = rng.standard_normal((6, r))
    y, _ = O.align(z, w1, rng.standard_normal(6), np.zeros((d, 6)), b2)
    np.testing.assert_array_equal(y, np.tile(b2, (t, 1)))


def test_fold_brute_force_and_identity_output_layer():
    rng = np.random.default_rng(47)
    D, d, h = 5, 4, 3
    w_p, b_p = rng.standard_normal((D, d)), rng.standard_normal(D)
    w2, b2 = rng.standard_normal((d, h)), rng.standard_normal(d)
    wf, c = O.fold_aligner(w_p, b_p, w2, b2)
    for n in range(D):
        for j in range(h):
            s = 0.0
            for i in range(d):
                s += w_p[n, i] * w2[i, j]
            assert abs(wf[n, j] - s) < 1e-12
        s = b_p[n]
        for i in range(d):
            s += w_p[n, i] * b2[i]
        assert abs(c[n] - s) < 1e-12
    # an identity output layer with no bias leaves the projection as it is
    wf, c = O.fold_aligner(w_p, None, np.eye(d), None)
    np.testing.assert_array_equal(wf, w_p)
    np.testing.assert_array_equal(c, np.zeros(D))


def test_fold_reproduces_the_literal_aligner_then_patch_chain():
    # Eq. aligner -> Eq. kv_from_patch through H_hat, against the same maps with the output layer
    # folded into the projections and applied to the hidden activations directly.
    rng = np.random.default_rng(53)
    t, r, hid, d, H, dh, theta = 9, 6, 10, 12, 2, 8, 1e4
    D = H * dh
    pos = rng.integers(0, 5000, t)
    z = rng.standard_normal((t, r))
    w1, b1 = rng.standard_normal((hid, r)), rng.standard_normal(hid)
    w2, b2 = rng.standard_normal((d, hid)), rng.standard_normal(d)
    w_k, b_k = rng.standard_normal((D, d)), rng.standard_normal(D)
    w_v, b_v = rng.standard_normal((D, d)), rng.standard_normal(D)
    h_hat, act = O.align(z, w1, b1, w2, b2)
    k_ref = O.patch_k(h_hat, w_k, b_k, pos, H, dh, theta)
    v_ref = O.patch_v(h_hat, w_v, b_v)
    fk, ck = O.fold_aligner(w_k, b_k, w2, b2)
    fv, cv = O.fold_aligner(w_v, b_v, w2, b2)
    np.testing.assert_allclose(O.patch_k(act, fk, ck, pos, H, dh, theta), k_ref, rtol=1e-11,
                               atol=1e-11)
    np.testing.assert_allclose(O.patch_v(act, fv, cv), v_ref, rtol=1e-11, atol=1e-11)


# ------------------------------------------------------------------------------------------
# Offline Reuse fit (Section 4.3.1; Appendix F.1)
# ------------------------------------------------------------------------------------------
def _sign_fix_test(v):
    """Test-side sign convention: each column's largest-magnitude entry positive."""
    v = np.array(v, dtype=np.float64)
    for j in range(v.shape[1]):
        i = int(np.argmax(np.abs(v[:, j])))
        if v[i, j] < 0:
            v[:, j] = -v[:, j]
    return v


def _exact_svd_pair(rng, n, w, sig):
    """Joint rows X = U diag(sig) W^T with U [n, 2w] orthonormal and W [2w, 2w] orthogonal."""
    u = rand_orthonormal(rng, n, 2 * w)
    wm = rand_orthonormal(rng, 2 * w, 2 * w)
    x = (u * sig[None, :]) @ wm.T
    return x[:, :w], x[:, w:], wm


def test_fit_gram_brute_force():
    rng = np.random.default_rng(41)
    T, H, dh, th = 7, 2, 4, 100.0
    w = dh  # head-shared: two rows per token
    a = rng.standard_normal((T, H * dh))
    b = rng.standard_normal((T, H * dh))
    pos = np.array([3, 4, 5, 0, 1, 2, 9])
    G, s = O.fit_gram(a, b, pos, H, dh, th, w, derope=True)
    ar = rope_complex(a, pos, H, dh, th, sign=-1.0)
    br = rope_complex(b, pos, H, dh, th, sign=-1.0)
    rows = []
    for t in range(T):
        for h in range(H):
            rows.append(list(ar[t, h * dh:(h + 1) * dh]) + list(br[t, h * dh:(h + 1) * dh]))
    n2 = 2 * w
    G_ref = np.zeros((n2, n2))
    s_ref = np.zeros(n2)
    for row in rows:
        for i in range(n2):
            s_ref[i] += row[i]
            for j in range(n2):
                G_ref[i, j] += row[i] * row[j]
    np.testing.assert_allclose(G, G_ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(s, s_ref, rtol=1e-12, atol=1e-12)


def test_fit_matches_library_svd_and_ridge():
    # The SVD of the joint rows (LAPACK gesvd, not the oracle's call) and scikit-learn's Ridge
    # fix the encoder and decoder: W_enc = Ridge(A -> Z), W_dec = Ridge(Z -> B), Z = X V_r.
    from sklearn.linear_model import Ridge
    rng = np.random.default_rng(42)
    N, w, r, lam = 60, 6, 3, 0.7
    A = rng.standard_normal((N, w)) @ rng.standard_normal((w, w))
    B = A @ rng.standard_normal((w, w)) + 0.1 * rng.standard_normal((N, w))
    w_enc, w_dec, mu_a, mu_b = O.fit_reuse(A, B, None, 1, w, 1e4, w, False, r, lam, center=False)
    assert mu_a is None and mu_b is None
    X = np.concatenate([A, B], axis=1)
    _, _, vt = scipy.linalg.svd(X, full_matrices=False, lapack_driver="gesvd")
    vr = _sign_fix_test(vt[:r].T)
    Z = X @ vr
    enc = Ridge(alpha=lam, fit_intercept=False, solver="svd").fit(A, Z).coef_
    dec = Ridge(alpha=lam, fit_intercept=False, solver="svd").fit(Z, B).coef_
    assert w_enc.shape == (r, w) and w_dec.shape == (w, r)
    np.testing.assert_allclose(w_enc, enc, rtol=1e-9, atol=1e-10)
    np.testing.assert_allclose(w_dec, dec, rtol=1e-9, atol=1e-10)


def test_fit_decoder_closed_form_on_exact_svd():
    # X = U diag(sig) W^T by construction: the decoder is the consumer half of W's first r
    # columns (sign-fixed), shrunk by sig^2 / (sig^2 + lam) under the ridge penalty.
    rng = np.random.default_rng(43)
    N, w, r = 40, 5, 3
    sig = np.array([9.0, 6.0, 4.0, 1.0, 0.5, 0.3, 0.2, 0.1, 0.05, 0.02])
    A, B, wm = _exact_svd_pair(rng, N, w, sig)
    vr = _sign_fix_test(wm[:, :r])
    for lam in (0.0, 3.0):
        _, w_dec, _, _ = O.fit_reuse(A, B, None, 1, w, 1e4, w, False, r, lam, center=False)
        shrink = sig[:r] ** 2 / (sig[:r] ** 2 + lam)
        np.testing.assert_allclose(w_dec, vr[w:, :] * shrink[None, :], rtol=1e-9, atol=1e-11)


def test_fit_exact_rank_pair_translates_new_samples():
    # Producer and consumer rows driven by one rank-r latent (plus offsets): the fitted
    # translator maps fresh producer rows of the same form onto the consumer's exactly
    # (up to the tiny ridge term).
    rng = np.random.default_rng(44)
    N, w, r = 300, 8, 3
    qa = rng.standard_normal((r, w))
    qb = rng.standard_normal((r, w))
    ma, mb = rng.standard_normal(w), rng.standard_normal(w)
    C = rng.standard_normal((N, r))
    A, B = C @ qa + ma, C @ qb + mb
    w_enc, w_dec, mu_a, mu_b = O.fit_reuse(A, B, None, 1, w, 1e4, w, False, r, 1e-9)
    np.testing.assert_allclose(mu_a, ma + C.mean(0) @ qa, rtol=1e-12, atol=1e-12)
    C2 = rng.standard_normal((50, r))
    A2, B2 = C2 @ qa + ma, C2 @ qb + mb
    z = O.encode_v(A2, w_enc, mu_a)
    np.testing.assert_allclose(O.decode_v(z, w_dec, mu_b, w), B2, rtol=1e-6, atol=1e-6)


def test_fit_self_pair_full_rank_is_identity():
    rng = np.random.default_rng(45)
    N, w = 80, 6
    A = rng.standard_normal((N, w)) @ rng.standard_normal((w, w)) + 2.0
    w_enc, w_dec, mu_a, mu_b = O.fit_reuse(A, A, None, 1, w, 1e4, w, False, w, 0.0)
    np.testing.assert_allclose(w_dec @ w_enc, np.eye(w), rtol=1e-9, atol=1e-9)
    np.testing.assert_allclose(mu_a, mu_b, rtol=0, atol=0)


def test_fit_centering_is_translation_invariant():
    rng = np.random.default_rng(46)
    N, w, r, lam = 70, 6, 4, 0.5
    A = rng.standard_normal((N, w)) * np.arange(1, w + 1)
    B = A @ rng.standard_normal((w, w)) + 0.2 * rng.standard_normal((N, w))
    ca, cb = 5.0 * rng.standard_normal(w), -3.0 * rng.standard_normal(w)
    e0, d0, ma0, mb0 = O.fit_reuse(A, B, None, 1, w, 1e4, w, False, r, lam)
    e1, d1, ma1, mb1 = O.fit_reuse(A + ca, B + cb, None, 1, w, 1e4, w, False, r, lam)
    np.testing.assert_allclose(e1, e0, rtol=1e-8, atol=1e-9)
    np.testing.assert_allclose(d1, d0, rtol=1e-8, atol=1e-9)
    np.testing.assert_allclose(ma1, ma0 + ca, rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(mb1, mb0 + cb, rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(ma0, A.mean(0), rtol=1e-12, atol=1e-12)


def test_fit_keys_are_fitted_in_content_space():
    # Keys are fitted after deRoPE: rotating the content by each token's position (complex
    # multiplication, test side) and fitting with deRoPE gives the content's own fit.
    rng = np.random.default_rng(47)
    T, H, dh, th, r = 50, 2, 8, 500.0, 4
    w = dh
    ca = rng.standard_normal((T, H * dh))
    cb = ca @ np.kron(np.eye(H), rng.standard_normal((dh, dh))) + 0.1 * rng.standard_normal((T, H * dh))
    pos = np.arange(T) * 3 + 1
    ka = rope_complex(ca, pos, H, dh, th)
    kb = rope_complex(cb, pos, H, dh, th)
    fk = O.fit_reuse(ka, kb, pos, H, dh, th, w, True, r, 0.1)
    fc = O.fit_reuse(ca, cb, None, H, dh, th, w, False, r, 0.1)
    for got, want in zip(fk, fc):
        np.testing.assert_allclose(got, want, rtol=1e-8, atol=1e-9)


def test_fit_sign_convention():
    # At lambda = 0 the decoder is the consumer half of V_r, whose full columns have their
    # largest-magnitude entry positive (LAPACK gesvd and a test-side sign rule).
    rng = np.random.default_rng(48)
    N, w, r = 50, 5, 3
    A = rng.standard_normal((N, w))
    B = 3.0 * rng.standard_normal((N, w))
    _, w_dec, _, _ = O.fit_reuse(A, B, None, 1, w, 1e4, w, False, r, 0.0, center=False)
    X = np.concatenate([A, B], axis=1)
    _, _, vt = scipy.linalg.svd(X, full_matrices=False, lapack_driver="gesvd")
    np.testing.assert_allclose(w_dec, _sign_fix_test(vt[:r].T)[w:], rtol=1e-9, atol=1e-11)
