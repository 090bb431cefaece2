"""Plain fp64 CPU oracle of the SCD KV-state codec.

TEST INFRASTRUCTURE ONLY. Nothing on the product path (the HIP library, its C ABI and the
Python binding in ``paper_2606_07684_amd``) imports, calls or links this module; only the
tests, the smoke check and the benchmark's CPU-baseline leg do.  It shares no code with the
GPU path.

Every function follows the paper's definitions, written out in float64 numpy with a library
matmul as the only primitive: no blocking, fusion or reordering beyond the definition.
Inputs may be any real dtype; they are upcast to float64 exactly before any arithmetic.

Conventions (readings of points the paper leaves open; each one is listed in the design notes):

* Layers are 0-based; a layer is Patch when ``is_patch[l]`` is true, Reuse otherwise
  (Section 4.1 "Notation and Preliminaries": L_reuse is the complement of L_patch).
* RoPE uses rotate-half pairing within each head: element ``i`` pairs with ``i + d_h/2``,
  frequency ``omega_i = theta ** (-2 i / d_h)``, angle ``p * omega_i`` (the RoFormer rotation;
  the paper names RoPE/deRoPE as forward and inverse operations in Section 4.1).
* A basis of width ``w`` acts on rows of ``w`` consecutive channels; a token of ``D = H*d_h``
  channels is ``g = D / w`` rows (``w = D``: one row per token; ``w = d_h``: the paper's
  head-shared basis with batch x heads x tokens flattened into one sample axis, Section 4.1).
* Matrices are stored as ``[out, in]`` (the ``nn.Linear`` layout), so every map is ``x @ W.T``.
  The paper writes ``x W`` with ``W`` of shape ``[in, out]``; the two are the same map.
* The encoder subtracts an optional offset ``mu_enc`` before projecting and the decoder adds an
  optional ``mu_dec`` after; ``None`` means zero and gives the paper's equations exactly.
* Patch may add an optional projection bias before RoPE (``None`` means none, as in the paper).

parity pinned: every function here is checked by the ``-m "not gpu"`` tests against closed
forms, invariants and independent formulations (see tests/test_oracle_pins.py).
"""
from __future__ import annotations

import numpy as np

F64 = np.float64


def _f64(x):
    return None if x is None else np.asarray(x, dtype=F64)


# --------------------------------------------------------------------------------------------
# a0: routing table (Section 4.1; Section 4.5 "Online Procedure": fixed sets, constant-time
# membership checks; Algorithm 1 takes L_patch and L_reuse as fixed inputs).
# --------------------------------------------------------------------------------------------
def schedule(is_patch):
    """Split layer indices into (reuse, patch) lists.

    L_patch is the set of layers flagged in ``is_patch``; L_reuse is its complement
    (Section 4.1).  Both lists are in increasing layer order.
    """
    flags = [bool(v) for v in is_patch]
    reuse = [l for l, p in enumerate(flags) if not p]
    patch = [l for l, p in enumerate(flags) if p]
    return reuse, patch


def payload_bytes(is_patch, n_tokens, n_kv_heads, head_dim, basis_width, rank_k, rank_v,
                  rank_h, elem_bytes):
    """Bytes of the transmitted code set and per-layer offsets into one packed buffer.

    Algorithm 1 transmits {Z_K, Z_V} for every Reuse layer and Z_H for every Patch layer;
    Section 4.5 states this is O(T r).  A Reuse layer sends ``T*g*(r_K + r_V)`` elements
    (``g = D / w`` code rows per token), a Patch layer sends ``T*r_H``.  Layers are laid out
    in layer order, K codes before V codes.  Returns ``(total, offsets[L+1])``.
    """
    d = n_kv_heads * head_dim
    g = d // basis_width
    offs = [0]
    for l, p in enumerate(is_patch):
        if p:
            n = n_tokens * rank_h[l]
        else:
            n = n_tokens * g * (rank_k[l] + rank_v[l])
        offs.append(offs[-1] + n * elem_bytes)
    return offs[-1], offs


# --------------------------------------------------------------------------------------------
# a1: token positions of a packed ragged batch (Appendix F.2: the reconstructed cache is used
# as native history with the framework's own cache positions; each request starts at its own
# first position, zero unless given).
# --------------------------------------------------------------------------------------------
def positions(cu_seqlens, pos0=None):
    """Position of every packed token: ``p(t) = t - cu[b] + pos0[b]`` for ``cu[b] <= t < cu[b+1]``."""
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    n_seqs = len(cu) - 1
    out = np.empty(int(cu[-1]), dtype=np.int64)
    for b in range(n_seqs):
        start = 0 if pos0 is None else int(pos0[b])
        out[cu[b]:cu[b + 1]] = np.arange(cu[b + 1] - cu[b], dtype=np.int64) + start
    return out


# --------------------------------------------------------------------------------------------
# RoPE / deRoPE (Section 4.1: keys use rotary embeddings; deRoPE is the inverse operation;
# Section 4.3.1 removes RoPE before fitting, Eq. (decode_kv) re-applies it after decoding,
# Eq. (kv_from_patch) applies it to regenerated keys).
# --------------------------------------------------------------------------------------------
def rope_angles(pos, head_dim, theta):
    """Angles ``a[t, i] = p(t) * theta**(-2 i / d_h)`` for ``i < d_h / 2``, in fp64."""
    half = head_dim // 2
    i = np.arange(half, dtype=F64)
    omega = np.power(F64(theta), -2.0 * i / F64(head_dim))
    return np.asarray(pos, dtype=F64)[:, None] * omega[None, :]


def rope(x, pos, n_kv_heads, head_dim, theta, inverse=False):
    """Rotate each head of ``x[T, H*d_h]`` by its token's position (``inverse`` = deRoPE).

    Forward: ``u' = u cos a - v sin a``, ``v' = v cos a + u sin a`` for the pair
    ``(u, v) = (x[h, i], x[h, i + d_h/2])``.  deRoPE is the same rotation with ``-a``.
    """
    x = _f64(x)
    t = x.shape[0]
    half = head_dim // 2
    a = rope_angles(pos, head_dim, theta)
    if inverse:
        a = -a
    c = np.cos(a)[:, None, :]
    s = np.sin(a)[:, None, :]
    xh = x.reshape(t, n_kv_heads, head_dim)
    u = xh[:, :, :half]
    v = xh[:, :, half:]
    out = np.empty_like(xh)
    out[:, :, :half] = u * c - v * s
    out[:, :, half:] = v * c + u * s
    return out.reshape(t, n_kv_heads * head_dim)


def to_rows(x, basis_width):
    """View token-major ``[T, D]`` as ``[T*g, w]`` (row ``t*g + j`` = channels ``[j*w, (j+1)*w)``)."""
    x = _f64(x)
    return x.reshape(-1, basis_width)


def from_rows(y, d):
    """Inverse of :func:`to_rows`: ``[T*g, w]`` back to ``[T, D]``."""
    return _f64(y).reshape(-1, d)


# --------------------------------------------------------------------------------------------
# a2-a4: producer encode (Section 4.3.2, Eq. (encode_z_kv); Section 4.4.1 for Z_H;
# Algorithm 1, producer half).
# --------------------------------------------------------------------------------------------
def encode_k(k_a, pos, w_enc, mu_enc, n_kv_heads, head_dim, theta):
    """``Z_K = (rows(deRoPE(K_A)) - mu_enc) @ W_enc^T`` with ``W_enc`` stored ``[r_K, w]``."""
    w = _f64(w_enc).shape[1]
    x = to_rows(rope(k_a, pos, n_kv_heads, head_dim, theta, inverse=True), w)
    if mu_enc is not None:
        x = x - _f64(mu_enc)[None, :]
    return x @ _f64(w_enc).T


def encode_v(v_a, w_enc, mu_enc):
    """``Z_V = (rows(V_A) - mu_enc) @ W_enc^T``; values carry no RoPE."""
    w = _f64(w_enc).shape[1]
    x = to_rows(v_a, w)
    if mu_enc is not None:
        x = x - _f64(mu_enc)[None, :]
    return x @ _f64(w_enc).T


def encode_h(h_a, w_enc_h):
    """``Z_H = H_in,A @ W_enc,H^T`` with ``W_enc,H`` stored ``[r_H, d_model]`` (Section 4.4.1)."""
    return _f64(h_a) @ _f64(w_enc_h).T


# --------------------------------------------------------------------------------------------
# a5-a6: consumer Reuse decode (Section 4.3.2, Eq. (decode_kv) and the RoPE that follows it;
# Algorithm 1, consumer half; Appendix F.2 "Online Reuse").
# --------------------------------------------------------------------------------------------
def decode_k(z_k, w_dec, mu_dec, pos, n_kv_heads, head_dim, theta):
    """``K_B = RoPE(unrows(Z_K @ W_dec^T + mu_dec))`` with ``W_dec`` stored ``[w, r_K]``."""
    y = _f64(z_k) @ _f64(w_dec).T
    if mu_dec is not None:
        y = y + _f64(mu_dec)[None, :]
    d = n_kv_heads * head_dim
    return rope(from_rows(y, d), pos, n_kv_heads, head_dim, theta)


def decode_v(z_v, w_dec, mu_dec, d):
    """``V_B = unrows(Z_V @ W_dec^T + mu_dec)``."""
    y = _f64(z_v) @ _f64(w_dec).T
    if mu_dec is not None:
        y = y + _f64(mu_dec)[None, :]
    return from_rows(y, d)


# --------------------------------------------------------------------------------------------
# Patch aligner (Section 4.4.2, Eq. (aligner)): H_hat = g_theta(Z_H).  The paper calls g_theta
# an MLP and fixes neither depth, width nor activation; the reading taken is two layers with the
# backbone's SiLU between them: H_hat = W2 SiLU(W1 z + b1) + b2, weights stored [out, in].
# --------------------------------------------------------------------------------------------
def silu(x):
    """``SiLU(x) = x * sigmoid(x) = x / (1 + e^-x)``, evaluated so that no term overflows."""
    x = _f64(x)
    # sigmoid(x) = 1 / (1 + e^-x) for x >= 0 and e^x / (1 + e^x) for x < 0 (same value)
    e = np.exp(-np.abs(x))
    sig = np.where(x >= 0, 1.0 / (1.0 + e), e / (1.0 + e))
    return x * sig


def align(z_h, w1, b1, w2, b2):
    """``H_hat = SiLU(Z_H @ W1^T + b1) @ W2^T + b2`` with ``W1 [h, r_H]``, ``W2 [d_model, h]``;
    ``b1``/``b2`` may be ``None``.  Returns ``(H_hat, hidden activations)``."""
    a = _f64(z_h) @ _f64(w1).T
    if b1 is not None:
        a = a + _f64(b1)[None, :]
    a = silu(a)
    y = a @ _f64(w2).T
    if b2 is not None:
        y = y + _f64(b2)[None, :]
    return y, a


# --------------------------------------------------------------------------------------------
# a7: Patch KV regeneration (Section 4.4.2, Eq. (kv_from_patch); Appendix F.2 "Online Patch").
# --------------------------------------------------------------------------------------------
def patch_k(h_hat, w_k, b_k, pos, n_kv_heads, head_dim, theta):
    """``K_B = RoPE(H_hat @ W_K^T + b_K)`` with ``W_K`` stored ``[D, d_model]``."""
    y = _f64(h_hat) @ _f64(w_k).T
    if b_k is not None:
        y = y + _f64(b_k)[None, :]
    return rope(y, pos, n_kv_heads, head_dim, theta)


def patch_v(h_hat, w_v, b_v):
    """``V_B = H_hat @ W_V^T + b_V``."""
    y = _f64(h_hat) @ _f64(w_v).T
    if b_v is not None:
        y = y + _f64(b_v)[None, :]
    return y


# --------------------------------------------------------------------------------------------
# The aligner's output layer folded into a projection.  Eq. (aligner) ends in the affine map
# H_hat = act W2^T + b2 and Eq. (kv_from_patch) applies W_P (P = K, V) to H_hat before any
# nonlinearity, so H_hat W_P^T + b_P = act (W_P W2)^T + (W_P b2 + b_P).
# --------------------------------------------------------------------------------------------
def fold_aligner(w_p, b_p, w2, b2):
    """``(W_P @ W2, W_P @ b2 + b_P)`` with ``W_P [D, d_model]``, ``W2 [d_model, h]``; an absent
    bias counts as zero.  Regenerating a Patch layer from the aligner's hidden activations with
    the folded pair, ``patch_k(act, W_fold, c, ...)``, equals ``patch_k(H_hat, W_P, b_P, ...)``."""
    w_p, w2 = _f64(w_p), _f64(w2)
    w_fold = w_p @ w2
    c = np.zeros(w_p.shape[0], dtype=F64)
    if b2 is not None:
        c = c + w_p @ _f64(b2)
    if b_p is not None:
        c = c + _f64(b_p)
    return w_fold, c


# --------------------------------------------------------------------------------------------
# Whole-model passes in Algorithm 1's order, and a8 cache assembly (Appendix F.2 "Cache
# Assembly": Reuse layers hold reconstructed KV, Patch layers hold regenerated KV).
# --------------------------------------------------------------------------------------------
def encode_all(is_patch, pos, n_kv_heads, head_dim, theta, k_a, v_a, h_a,
               w_enc_k, w_enc_v, w_enc_h, mu_k=None, mu_v=None, layers=None):
    """Producer side: codes for every layer (``None`` where the layer's branch is absent)."""
    reuse, patch = schedule(is_patch)
    L = len(is_patch)
    z_k, z_v, z_h = [None] * L, [None] * L, [None] * L
    for l in reuse:
        if layers is not None and l not in layers:
            continue
        z_k[l] = encode_k(k_a[l], pos, w_enc_k[l], None if mu_k is None else mu_k[l],
                          n_kv_heads, head_dim, theta)
        z_v[l] = encode_v(v_a[l], w_enc_v[l], None if mu_v is None else mu_v[l])
    for l in patch:
        if layers is not None and l not in layers:
            continue
        z_h[l] = encode_h(h_a[l], w_enc_h[l])
    return z_k, z_v, z_h


def reuse_decode_all(is_patch, pos, n_kv_heads, head_dim, theta, z_k, z_v, w_dec_k, w_dec_v,
                     mu_k=None, mu_v=None, layers=None):
    """Consumer Reuse branch for every Reuse layer; Patch layers are left as ``None``."""
    reuse, _ = schedule(is_patch)
    d = n_kv_heads * head_dim
    L = len(is_patch)
    k, v = [None] * L, [None] * L
    for l in reuse:
        if layers is not None and l not in layers:
            continue
        k[l] = decode_k(z_k[l], w_dec_k[l], None if mu_k is None else mu_k[l], pos,
                        n_kv_heads, head_dim, theta)
        v[l] = decode_v(z_v[l], w_dec_v[l], None if mu_v is None else mu_v[l], d)
    return k, v


def patch_all(is_patch, pos, n_kv_heads, head_dim, theta, h_hat, w_k, w_v, b_k=None, b_v=None,
              layers=None):
    """Consumer Patch branch for every Patch layer; Reuse layers are left as ``None``."""
    _, patch = schedule(is_patch)
    L = len(is_patch)
    k, v = [None] * L, [None] * L
    for l in patch:
        if layers is not None and l not in layers:
            continue
        k[l] = patch_k(h_hat[l], w_k[l], None if b_k is None else b_k[l], pos,
                       n_kv_heads, head_dim, theta)
        v[l] = patch_v(h_hat[l], w_v[l], None if b_v is None else b_v[l])
    return k, v


def assemble(is_patch, reuse_kv, patch_kv):
    """Hybrid cache: layer ``l`` takes the Patch result when ``is_patch[l]``, else the Reuse one."""
    rk, rv = reuse_kv
    pk, pv = patch_kv
    out_k, out_v = [], []
    for l, p in enumerate(is_patch):
        out_k.append(pk[l] if p else rk[l])
        out_v.append(pv[l] if p else rv[l])
    return out_k, out_v


# --------------------------------------------------------------------------------------------
# Offline Reuse fit (Section 4.3.1 "Joint Subspace Learning"; Appendix F.1 "Reuse: Layer-wise
# Stack-SVD with Ridge Regression").  For one layer and branch the producer's and consumer's
# calibration tensors of the same prefixes are flattened into rows A, B [N, w] (keys de-rotated
# first), a truncated SVD of the joint matrix X = [A B] finds the shared rank-r latent space, and
# ridge regressions fit the producer encoder (A -> Z) and the consumer decoder (Z -> B).
# Readings taken where the paper is open:
#   * latents Z = X V_r (= U_r S_r): the decoders carry the orthonormal right singular vectors and
#     the codes carry the scale;
#   * the decoder is a ridge fit as well, with the same lambda (lambda = 0 gives the SVD factor);
#   * optional centring: A and B lose their column means first; the means become the encoder's
#     and decoder's offsets (the codec subtracts the encoder offset and adds the decoder offset);
#   * each singular vector's sign is fixed so that its entry of largest magnitude is positive
#     (the first such entry on ties).
# --------------------------------------------------------------------------------------------
def fit_rows(x, pos, n_kv_heads, head_dim, theta, basis_width, derope):
    """Calibration rows ``[N, w]`` of one model's cache ``x [T, D]``: de-rotated for keys."""
    if derope:
        x = rope(x, pos, n_kv_heads, head_dim, theta, inverse=True)
    return to_rows(x, basis_width)


def fit_gram(a, b, pos, n_kv_heads, head_dim, theta, basis_width, derope):
    """``G = X^T X`` and ``s = 1^T X`` of the joint rows ``X = [A B]`` (no centring)."""
    x = np.concatenate([fit_rows(a, pos, n_kv_heads, head_dim, theta, basis_width, derope),
                        fit_rows(b, pos, n_kv_heads, head_dim, theta, basis_width, derope)], axis=1)
    return x.T @ x, x.sum(axis=0)


def sign_fix(v):
    """Flip each column of ``v`` so that its entry of largest magnitude is positive."""
    v = _f64(v).copy()
    idx = np.argmax(np.abs(v), axis=0)
    sgn = np.sign(v[idx, np.arange(v.shape[1])])
    sgn[sgn == 0] = 1.0
    return v * sgn[None, :]


def fit_reuse(a, b, pos, n_kv_heads, head_dim, theta, basis_width, derope, rank, lam,
              center=True):
    """Fit one layer's Reuse translator from paired caches ``a`` (producer) and ``b`` (consumer).

    Steps in the paper's order: de-rotate keys; flatten to rows A, B; (centre); truncated SVD of
    X = [A B] keeping ``rank`` right singular vectors V_r; latents Z = X V_r; ridge encoder
    ``E = argmin ||A E - Z||^2 + lam ||E||^2`` and ridge decoder
    ``F = argmin ||Z F - B||^2 + lam ||F||^2``.  Returned in the codec's storage:
    ``(W_enc [r, w] = E^T, W_dec [w, r] = F^T, mu_enc [w], mu_dec [w])`` (offsets None unless
    ``center``).
    """
    A = fit_rows(a, pos, n_kv_heads, head_dim, theta, basis_width, derope)
    B = fit_rows(b, pos, n_kv_heads, head_dim, theta, basis_width, derope)
    mu_a = mu_b = None
    if center:
        mu_a, mu_b = A.mean(axis=0), B.mean(axis=0)
        A, B = A - mu_a[None, :], B - mu_b[None, :]
    X = np.concatenate([A, B], axis=1)
    _, _, vt = np.linalg.svd(X, full_matrices=False)
    vr = sign_fix(vt[:rank].T)
    Z = X @ vr
    w = A.shape[1]
    E = np.linalg.solve(A.T @ A + lam * np.eye(w), A.T @ Z)
    F = np.linalg.solve(Z.T @ Z + lam * np.eye(rank), Z.T @ B)
    return E.T, F.T, mu_a, mu_b
