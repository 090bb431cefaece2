"""Plant plausible mistakes in the oracle (on the CPU) and check the pins catch every one.

Each mutation replaces one oracle function with a subtly wrong variant; at least one pin of
test_oracle_pins must then fail.  This is what makes the pins evidence for the oracle.
"""
import numpy as np
import pytest

from oracle import scd_oracle as O
import tests.test_oracle_pins as P

F64 = np.float64
_rope = O.rope
_positions = O.positions
_encode_k = O.encode_k
_encode_v = O.encode_v
_decode_k = O.decode_k
_decode_v = O.decode_v
_patch_k = O.patch_k
_align = O.align
_silu = O.silu
_fit_rows = O.fit_rows
_sign_fix = O.sign_fix
_payload_bytes = O.payload_bytes
_fold = O.fold_aligner


def payload_patch_term_g(is_patch, n_tokens, n, dh, w, rk, rv, rh, eb):
    # counts a Patch layer's code as g rows per token, like a Reuse layer's
    g = n * dh // w
    offs = [0]
    for l, p in enumerate(is_patch):
        m = n_tokens * g * rh[l] if p else n_tokens * g * (rk[l] + rv[l])
        offs.append(offs[-1] + m * eb)
    return offs[-1], offs


def payload_v_only(is_patch, n_tokens, n, dh, w, rk, rv, rh, eb):
    # forgets the key codes of Reuse layers
    return _payload_bytes(is_patch, n_tokens, n, dh, w, [0] * len(rk), rv, rh, eb)


def payload_patch_as_reuse(is_patch, n_tokens, n, dh, w, rk, rv, rh, eb):
    # sends K/V codes for Patch layers too
    return _payload_bytes([0] * len(is_patch), n_tokens, n, dh, w, rk, rv, rh, eb)


def fold_proj_bias_sign(w_p, b_p, w2, b2):
    # subtracts the projection bias instead of adding it
    return _fold(w_p, None if b_p is None else -np.asarray(b_p, F64), w2, b2)


def fold_bias_dropped(w_p, b_p, w2, b2):
    return _fold(w_p, b_p, w2, None)


def fold_proj_bias_dropped(w_p, b_p, w2, b2):
    return _fold(w_p, None, w2, b2)


def rope_wrong_sign(x, pos, n, dh, theta, inverse=False):
    return _rope(x, pos, n, dh, theta, inverse=not inverse)


def rope_wrong_freq(x, pos, n, dh, theta, inverse=False):
    return _rope(x, pos, n, dh, theta ** 0.5, inverse=inverse)


def rope_interleaved(x, pos, n, dh, theta, inverse=False):
    # pairs (2i, 2i+1) instead of (i, i + d/2)
    t = x.shape[0]
    xh = np.asarray(x, F64).reshape(t, n, dh)
    perm = np.concatenate([np.arange(0, dh, 2), np.arange(1, dh, 2)])
    y = _rope(xh[..., perm].reshape(t, n * dh), pos, n, dh, theta, inverse).reshape(t, n, dh)
    out = np.empty_like(y)
    out[..., perm] = y
    return out.reshape(t, n * dh)


def rope_head_mixed(x, pos, n, dh, theta, inverse=False):
    # pairs across the whole row instead of within each head
    return _rope(x, pos, 1, n * dh, theta, inverse).reshape(x.shape)


def positions_off_by_one(cu, pos0=None):
    return _positions(cu, pos0) + 1


def positions_global(cu, pos0=None):
    # forgets to restart every request at its own first position
    return np.arange(int(np.asarray(cu)[-1]), dtype=np.int64)


def encode_k_no_derope(k_a, pos, w_enc, mu_enc, n, dh, theta):
    x = O.to_rows(k_a, np.asarray(w_enc).shape[1])
    if mu_enc is not None:
        x = x - np.asarray(mu_enc, F64)[None, :]
    return x @ np.asarray(w_enc, F64).T


def encode_v_mu_sign(v_a, w_enc, mu_enc):
    return _encode_v(v_a, w_enc, None if mu_enc is None else -np.asarray(mu_enc, F64))


def encode_v_mu_dropped(v_a, w_enc, mu_enc):
    return _encode_v(v_a, w_enc, None)


def decode_v_transposed(z, w_dec, mu_dec, d):
    y = np.asarray(z, F64) @ np.asarray(w_dec, F64)
    if mu_dec is not None:
        y = y + np.asarray(mu_dec, F64)[None, :]
    return O.from_rows(y, d)


def decode_k_rope_before_mu(z, w_dec, mu_dec, pos, n, dh, theta):
    y = O.from_rows(np.asarray(z, F64) @ np.asarray(w_dec, F64).T, n * dh)
    y = _rope(y, pos, n, dh, theta)
    if mu_dec is not None:
        y = y + np.tile(np.asarray(mu_dec, F64), (n * dh) // len(mu_dec))[None, :]
    return y


def decode_k_no_rope(z, w_dec, mu_dec, pos, n, dh, theta):
    return _decode_v(z, w_dec, mu_dec, n * dh)


def patch_k_no_bias(h, w, b, pos, n, dh, theta):
    return _patch_k(h, w, None, pos, n, dh, theta)


def patch_k_bias_after_rope(h, w, b, pos, n, dh, theta):
    y = _patch_k(h, w, None, pos, n, dh, theta)
    return y if b is None else y + np.asarray(b, F64)[None, :]


def align_w1_transposed(z, w1, b1, w2, b2):
    # contracts z with W1 rather than W1^T (only square-compatible shapes survive)
    return _align(z, np.asarray(w1, F64).T, b1, w2, b2)


def align_silu_after_output(z, w1, b1, w2, b2):
    a = np.asarray(z, F64) @ np.asarray(w1, F64).T
    if b1 is not None:
        a = a + np.asarray(b1, F64)[None, :]
    y = a @ np.asarray(w2, F64).T
    if b2 is not None:
        y = y + np.asarray(b2, F64)[None, :]
    return O.silu(y), a


def align_hidden_bias_dropped(z, w1, b1, w2, b2):
    return _align(z, w1, None, w2, b2)


def silu_sign_flipped(x):
    x = np.asarray(x, F64)
    return x / (1.0 + np.exp(x))


def fit_rows_no_derope(x, pos, n, dh, theta, w, derope):
    return _fit_rows(x, pos, n, dh, theta, w, False)


def sign_fix_negative(v):
    return -_sign_fix(v)


def _fit_variant(a, b, pos, n, dh, theta, w, derope, rank, lam, center=True, *, subtract=True,
                 scaled=True, dec_ridge=True, enc_from_b=False):
    A = O.fit_rows(a, pos, n, dh, theta, w, derope)
    B = O.fit_rows(b, pos, n, dh, theta, w, derope)
    mu_a = mu_b = None
    if center:
        mu_a, mu_b = A.mean(axis=0), B.mean(axis=0)
        if subtract:
            A, B = A - mu_a[None, :], B - mu_b[None, :]
    X = np.concatenate([A, B], axis=1)
    _, s, vt = np.linalg.svd(X, full_matrices=False)
    vr = O.sign_fix(vt[:rank].T)
    Z = X @ vr if scaled else (X @ vr) / s[None, :rank]
    src = B if enc_from_b else A
    E = np.linalg.solve(src.T @ src + lam * np.eye(src.shape[1]), src.T @ Z)
    F = np.linalg.solve(Z.T @ Z + (lam if dec_ridge else 0.0) * np.eye(rank), Z.T @ B)
    return E.T, F.T, mu_a, mu_b


def fit_not_centred(*a, **k):
    return _fit_variant(*a, **k, subtract=False)


def fit_unscaled_latents(*a, **k):
    return _fit_variant(*a, **k, scaled=False)


def fit_decoder_without_ridge(*a, **k):
    return _fit_variant(*a, **k, dec_ridge=False)


def fit_encoder_on_consumer(*a, **k):
    return _fit_variant(*a, **k, enc_from_b=True)


def _schedule_swapped(is_patch):
    flags = [bool(v) for v in is_patch]
    return [l for l, f in enumerate(flags) if f], [l for l, f in enumerate(flags) if not f]


MUTATIONS = [
    ("rope", rope_wrong_sign),
    ("rope", rope_wrong_freq),
    ("rope", rope_interleaved),
    ("rope", rope_head_mixed),
    ("positions", positions_off_by_one),
    ("positions", positions_global),
    ("encode_k", encode_k_no_derope),
    ("encode_v", encode_v_mu_sign),
    ("encode_v", encode_v_mu_dropped),
    ("decode_v", decode_v_transposed),
    ("decode_k", decode_k_rope_before_mu),
    ("decode_k", decode_k_no_rope),
    ("patch_k", patch_k_no_bias),
    ("patch_k", patch_k_bias_after_rope),
    ("schedule", _schedule_swapped),
    ("align", align_w1_transposed),
    ("align", align_silu_after_output),
    ("align", align_hidden_bias_dropped),
    ("silu", silu_sign_flipped),
    ("fit_rows", fit_rows_no_derope),
    ("sign_fix", sign_fix_negative),
    ("fit_reuse", fit_not_centred),
    ("fit_reuse", fit_unscaled_latents),
    ("fit_reuse", fit_decoder_without_ridge),
    ("fit_reuse", fit_encoder_on_consumer),
    ("payload_bytes", payload_patch_term_g),
    ("payload_bytes", payload_v_only),
    ("payload_bytes", payload_patch_as_reuse),
    ("fold_aligner", fold_proj_bias_sign),
    ("fold_aligner", fold_bias_dropped),
    ("fold_aligner", fold_proj_bias_dropped),
]

PINS = [getattr(P, n) for n in dir(P) if n.startswith("test_")]


def _run_pin(fn):
    import inspect
    params = inspect.signature(fn).parameters
    if "w_is_head" in params:
        for v in (False, True):
            fn(v)
    elif "branch" in params:
        for v in ("k", "v"):
            fn(v)
    else:
        fn()


@pytest.mark.parametrize("name,fn", MUTATIONS, ids=[f.__name__ for _, f in MUTATIONS])
def test_pins_catch_planted_mistake(monkeypatch, name, fn):
    monkeypatch.setattr(O, name, fn)
    caught = []
    for pin in PINS:
        try:
            _run_pin(pin)
        except (AssertionError, ValueError, IndexError):
            caught.append(pin.__name__)
    assert caught, f"no pin caught the planted mistake {fn.__name__}"


def test_unmutated_oracle_passes_every_pin():
    for pin in PINS:
        _run_pin(pin)
