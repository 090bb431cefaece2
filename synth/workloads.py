"""Seeded synthetic workloads shaped like the paper's model pairs.

This module is shared input generation only: it holds none of the codec's arithmetic (no
RoPE, no encode, no decode, no projection).  It draws random tensors, builds orthonormal bases
by QR, RMS-normalises hidden states (the producer and consumer models' own normalisation, which
precedes the codec) and synthesises power-law K/V signals.  Both the oracle and the GPU path
consume the tensors it returns, rounded once to the path's dtype.

Every tensor is drawn from its own generator, seeded from (workload name, layer, tensor name),
so any tensor can be regenerated alone.  Variance notation: ``N(0, s)`` has variance ``s``.
"""
from __future__ import annotations

import dataclasses
import functools
import zlib
from typing import Optional, Sequence, Tuple

import numpy as np
import torch


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    n_layers: int
    d_model: int
    n_kv_heads: int
    head_dim: int
    seq_lens: Tuple[int, ...]
    ranks: Tuple[int, ...]            # per layer: r_K = r_H = ranks[l], r_V too unless ranks_v
    patch_layers: Tuple[int, ...]
    rope_theta: float
    dtype: str                        # "f32" or "bf16"
    basis_width: Optional[int] = None  # None -> D = n_kv_heads * head_dim
    power_law: bool = False           # K/V signal spectrum sigma_i ~ 1/i
    pos0: Optional[Tuple[int, ...]] = None
    with_bias: bool = False           # projection bias on the Patch branch (Qwen2-style)
    with_mu: bool = True
    ranks_v: Optional[Tuple[int, ...]] = None  # per-layer r_V when it differs from r_K
    aligner_hidden: Optional[int] = None  # width of the Patch aligner's hidden layer (None: d_model)

    def rank(self, layer: int, branch: str) -> int:
        """Rank of one layer's branch ('k', 'v' or 'h')."""
        if branch == "v" and self.ranks_v is not None:
            return self.ranks_v[layer]
        return self.ranks[layer]

    @property
    def rank_v(self) -> Tuple[int, ...]:
        return self.ranks_v if self.ranks_v is not None else self.ranks

    @property
    def kv_width(self) -> int:
        return self.n_kv_heads * self.head_dim

    @property
    def w(self) -> int:
        return self.basis_width or self.kv_width

    @property
    def g(self) -> int:
        return self.kv_width // self.w

    @property
    def n_tokens(self) -> int:
        return int(sum(self.seq_lens))

    @property
    def n_seqs(self) -> int:
        return len(self.seq_lens)

    @property
    def is_patch(self) -> Tuple[int, ...]:
        return tuple(1 if l in self.patch_layers else 0 for l in range(self.n_layers))

    @property
    def cu_seqlens(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.seq_lens)]).astype(np.int32)

    @property
    def max_position(self) -> int:
        """One past the largest RoPE position any token of the batch takes."""
        p0 = self.pos0 or (0,) * self.n_seqs
        return int(max(a + n for a, n in zip(p0, self.seq_lens)))

    @property
    def hidden_width(self) -> int:
        return self.aligner_hidden or self.d_model

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


def _ragged_lengths(seed: int, n: int, lo: int, hi: int) -> Tuple[int, ...]:
    """``n`` integers uniform on ``[lo, hi]`` inclusive."""
    return tuple(int(x) for x in np.random.default_rng(seed).integers(lo, hi + 1, n))


# The five model-shaped workloads.
TINY_F32 = Workload("tiny_f32", 4, 512, 4, 64, (512,), (32,) * 4, (2,), 1e4, "f32")
LLAMA3_8B = Workload("llama3_8b_bf16", 32, 4096, 8, 128, (8192,), (128,) * 32,
                     (0, 8, 16, 24), 5e5, "bf16", power_law=True)
QWEN2_7B = Workload("qwen2_7b_bf16", 28, 3584, 4, 128, (32768,), (96,) * 28,
                    (0, 7, 14, 21), 1e6, "bf16", power_law=True)
BATCHED = Workload("batched_ragged_bf16", 32, 4096, 8, 128, _ragged_lengths(3, 16, 1024, 16384),
                   tuple((64, 128, 256)[l % 3] for l in range(32)), (0, 8, 16, 24), 5e5, "bf16",
                   power_law=True)
LLAMA3_70B = Workload("llama3_70b_bf16", 80, 8192, 8, 128, (16384,), (128,) * 80,
                      tuple(range(0, 80, 10)), 5e5, "bf16", power_law=True)

CONFIGS = (TINY_F32, LLAMA3_8B, QWEN2_7B, BATCHED, LLAMA3_70B)

# The paper's head-shared basis (one basis of width d_h for all heads, Section 4.3.1) at the
# Llama-3-8B shape, with different key and value ranks.
LLAMA3_8B_HEAD_SHARED = LLAMA3_8B.replace(name="llama3_8b_head_shared_bf16", basis_width=128,
                                          ranks=(64,) * 32, ranks_v=(32,) * 32)
MODEL_SCALE_EXTRA = (LLAMA3_8B_HEAD_SHARED,)

# Small workloads the oracle finishes in seconds that still span several tiles, ragged tails,
# per-layer ranks, the head-shared basis, biases and non-zero first positions.
SMALL_BF16 = Workload("small_bf16", 5, 384, 2, 128, (300, 77, 650), (64, 128, 32, 256, 96),
                      (1, 4), 5e5, "bf16", power_law=True)
SMALL_HEAD_SHARED = Workload("small_head_shared_bf16", 3, 256, 4, 64, (129, 250), (32, 64, 48),
                             (2,), 1e4, "bf16", basis_width=64, with_bias=True,
                             pos0=(5, 1000), ranks_v=(64, 32, 48))
SMALL_F32 = Workload("small_f32", 3, 320, 2, 64, (97, 200, 31), (16, 48, 32), (0,), 1e4, "f32",
                     with_bias=True)
# d_model = 64: the Patch contraction is shorter than the copy pipeline is deep; one KV head.
SMALL_NARROW = Workload("small_narrow_bf16", 2, 64, 1, 128, (200, 57), (64, 32), (1,), 1e4, "bf16")
# Degenerate batches: empty and single-token requests between others, the smallest rank (16, which
# the bf16 decode hands to the generic kernel) next to 32, the head-shared basis, and start positions
# near the top of a long RoPE table.
SMALL_DEGENERATE = Workload("small_degenerate_bf16", 3, 128, 2, 64, (1, 0, 5, 1, 0, 130),
                            (16, 32, 32), (1,), 1e6, "bf16", basis_width=64,
                            pos0=(30000, 7, 0, 29990, 1, 5), ranks_v=(32, 32, 16))
# Full rank: r = w = 256 (the largest rank a launch takes) on the bf16 kernels.
SMALL_FULL_RANK = Workload("small_full_rank_bf16", 2, 256, 2, 128, (300, 33), (256, 256), (1,),
                           5e5, "bf16")
# More requests than the bf16 decode stages in LDS (256): the generic kernel takes the batch.
SMALL_MANY_REQUESTS = Workload("small_many_requests_bf16", 2, 128, 2, 64, _ragged_lengths(5, 300, 0, 3),
                               (32, 32), (1,), 1e4, "bf16")
# Patch aligner on the bf16 GEMM kernel: ragged token count (two partial 256-row tiles), code ranks
# 64 and 192, hidden width 384 (one and a half 256-column tiles).
SMALL_ALIGN = Workload("small_align_bf16", 3, 512, 2, 128, (300, 77, 650), (64, 128, 192), (0, 2),
                       5e5, "bf16", aligner_hidden=384)
# Many short Reuse layers: more row tiles than the decode's one round of workgroups, so shares run
# across layer boundaries (the basis is restaged mid-share) and every layer ends in a partial tile;
# ranks 128 (512-channel chunks) and 256 (256-channel chunks).
SMALL_MANY_LAYERS = Workload("small_many_layers_bf16", 72, 256, 8, 128, (300, 340),
                             (128,) * 48 + (256,) * 24, (), 5e5, "bf16")
# Offline Reuse fit (paired producer/consumer calibration caches): ragged batch with start positions,
# w = D = 128 (one 256 x 256 Gram of three upper tiles, several row slices with a ragged tail);
# the head-shared basis (w = d_h = 128, g = 4); fp32 with w = 64 (a 128-column Gram that spans the
# producer and consumer halves); d_h = 32; single-token requests (every position 0, so de-rotated
# keys keep the shared latent's low rank and the key fit is well conditioned).
FIT_SMALL_BF16 = Workload("fit_small_bf16", 3, 256, 2, 64, (300, 77, 650), (32, 32, 32), (1,), 1e4,
                          "bf16", pos0=(0, 40, 7), ranks_v=(48, 48, 48))
FIT_HEAD_SHARED = Workload("fit_head_shared_bf16", 2, 256, 4, 128, (129, 250), (16, 16), (), 5e5,
                           "bf16", basis_width=128, ranks_v=(32, 32))
FIT_F32 = Workload("fit_f32", 2, 128, 2, 64, (200, 61), (16, 16), (), 1e4, "f32", basis_width=64,
                   ranks_v=(32, 32))
FIT_DH32 = Workload("fit_dh32_bf16", 2, 128, 4, 32, (333,), (16, 32), (0,), 1e4, "bf16")
FIT_POS0_KEYS = Workload("fit_single_tokens_bf16", 2, 128, 2, 64, (1,) * 700, (32, 32), (), 1e4,
                         "bf16", ranks_v=(16, 16))
# Basis widths other than 128 take the bf16 Gram's tile kernel: w = D = 256 (2w = 512: ten upper
# tiles, three of them diagonal) with a packed batch, and the head-shared w = d_h = 64 (2w = 128: one
# tile spanning both models' columns).
FIT_W256_BF16 = Workload("fit_w256_bf16", 2, 256, 2, 128, (333, 190), (64, 64), (), 5e5, "bf16",
                         pos0=(3, 0), ranks_v=(32, 32))
FIT_W64_BF16 = Workload("fit_w64_bf16", 2, 128, 4, 64, (150, 211), (16, 16), (0,), 1e4, "bf16",
                        basis_width=64, ranks_v=(32, 32))
FIT_WORKLOADS = (FIT_SMALL_BF16, FIT_HEAD_SHARED, FIT_F32, FIT_DH32, FIT_POS0_KEYS, FIT_W256_BF16,
                 FIT_W64_BF16)
# The widest basis the solve takes: w = D = 1024 (8 KV heads of 128, one basis over all heads), a
# 2048 x 2048 Gram over 2,600 calibration rows of one Reuse layer.
FIT_W1024_BF16 = Workload("fit_w1024_bf16", 1, 256, 8, 128, (1400, 1200), (64,), (), 5e5, "bf16",
                          pos0=(0, 9), ranks_v=(64,))
# The model-shaped configurations' own bases: the fit at w = D = 1024 on calibration caches of the
# Llama-3-8B shape (8192 tokens of one request, rank 128), two Reuse layers.
FIT_CODEC_LLAMA3_8B = Workload("fit_codec_llama3_8b_bf16", 2, 4096, 8, 128, (8192,), (128, 128), (),
                               5e5, "bf16")
# Calibration at the Llama-3-8B shape with the head-shared basis: 8192 tokens x 8 heads = 65,536
# rows of 128 channels per layer (the paper calibrates on 100-500 prefixes of ~600 tokens).
FIT_LLAMA3_8B = LLAMA3_8B_HEAD_SHARED.replace(name="fit_llama3_8b_head_shared_bf16")

# Patch contractions of 5 and 7 steps of 64 (d_model 320 and 448), whose bf16 kernel cycles its
# operand tiles through a ring of five LDS slots: the ring wraps exactly at the last step, then
# part-way.  (These widths are not multiples of 128, so the aligner and the H encode take the
# generic kernel here.)
SMALL_RING5 = Workload("small_ring5_bf16", 2, 320, 2, 64, (300, 213), (64, 64), (0,), 1e4, "bf16",
                       with_bias=True)
SMALL_RING7 = Workload("small_ring7_bf16", 2, 448, 2, 64, (257,), (32, 64), (1,), 1e4, "bf16")
# The aligner on the same kernel with a second product of 10 steps (hidden width 640) and a first
# of 3 (rank 192).
SMALL_ALIGN_RING = Workload("small_align_ring_bf16", 2, 256, 2, 64, (300,), (64, 192), (0, 1),
                            1e4, "bf16", aligner_hidden=640)

# More requests than the decode body stages in LDS with a Patch code of rank 64: the aligner's
# first product takes the bf16 GEMM body.
SMALL_MANY_REQUESTS_ALIGN = SMALL_MANY_REQUESTS.replace(name="small_many_requests_align_bf16",
                                                        ranks=(64, 64), aligner_hidden=256)

# Ranks between 128 and 256 that are not 256: the encode's two workgroups per row tile then split
# the codes unevenly (128 + 32, 128 + 96, 128 + 64), for keys (de-rotated), values and H.
SMALL_SPLIT_RANKS = Workload("small_split_ranks_bf16", 3, 384, 2, 128, (300, 77, 250),
                             (160, 224, 192), (1,), 5e5, "bf16", ranks_v=(192, 96, 224))
TEST_WORKLOADS = (SMALL_BF16, SMALL_HEAD_SHARED, SMALL_F32, SMALL_NARROW, SMALL_DEGENERATE,
                  SMALL_FULL_RANK, SMALL_MANY_REQUESTS, SMALL_ALIGN, SMALL_MANY_LAYERS, SMALL_RING5,
                  SMALL_RING7, SMALL_ALIGN_RING, SMALL_SPLIT_RANKS)


# --------------------------------------------------------------------------------------------
# Seeded draws
# --------------------------------------------------------------------------------------------
def _seed(wl: Workload, layer: int, tensor: str) -> int:
    return zlib.crc32(f"{wl.name}/{layer}/{tensor}".encode()) & 0x7FFFFFFF


def _randn(wl, layer, tensor, shape, device) -> torch.Tensor:
    g = torch.Generator(device=device)
    g.manual_seed(_seed(wl, layer, tensor))
    return torch.randn(shape, generator=g, device=device, dtype=torch.float32)


def _rms_normalize(x: torch.Tensor) -> torch.Tensor:
    return x * torch.rsqrt(x.square().mean(dim=-1, keepdim=True) + 1e-6)


def power_law_sigma(w: int) -> np.ndarray:
    """``sigma_i = c / i`` (``i = 1..w``) with ``c`` chosen so the signal's per-element RMS is 1."""
    i = np.arange(1, w + 1, dtype=np.float64)
    c = np.sqrt(w / np.sum(1.0 / i ** 2))
    return c / i


@functools.lru_cache(maxsize=512)
def _full_basis(wl: Workload, layer: int, branch: str) -> np.ndarray:
    """Orthonormal ``[w, w]`` matrix (fp64, CPU); its first ``r`` columns are the layer's basis."""
    g = np.random.default_rng(_seed(wl, layer, "basis_" + branch))
    q, r = np.linalg.qr(g.standard_normal((wl.w, wl.w)))
    return q * np.sign(np.diag(r))[None, :]


def _cast(x: torch.Tensor, wl: Workload, device) -> torch.Tensor:
    return x.to(device=device, dtype=wl.torch_dtype).contiguous()


def basis(wl: Workload, layer: int, branch: str, device="cpu"):
    """Reuse artifacts of one layer and branch: ``(W_enc [r, w], W_dec [w, r])`` with W_dec = Q."""
    r = wl.rank(layer, branch)
    q = torch.from_numpy(_full_basis(wl, layer, branch)[:, :r].copy())
    return _cast(q.T.contiguous(), wl, device), _cast(q, wl, device)


def mu(wl: Workload, layer: int, branch: str, device="cpu"):
    """Offset ``mu ~ N(0, 0.1)`` of width ``w`` (the same for encoder and decoder), or None."""
    if not wl.with_mu:
        return None
    return _cast(_randn(wl, layer, "mu_" + branch, (wl.w,), "cpu") * np.sqrt(0.1), wl, device)


def codes(wl: Workload, layer: int, branch: str, device="cpu") -> torch.Tensor:
    """Reuse codes ``[T*g, r]``: N(0,1), scaled per column by sigma_1..r when the spectrum is a
    power law (the projection of the synthetic signal onto its top-r directions)."""
    r = wl.rank(layer, branch)
    z = _randn(wl, layer, "codes_" + branch, (wl.n_tokens * wl.g, r), device)
    if wl.power_law:
        sig = torch.tensor(power_law_sigma(wl.w)[:r], dtype=torch.float32, device=device)
        z = z * sig[None, :]
    return _cast(z, wl, device)


def kv_input(wl: Workload, layer: int, branch: str, device="cpu") -> torch.Tensor:
    """Producer K or V ``[T, D]``: ``mu + signal + N(0, 0.01)``.

    The signal is rank ``r`` in the layer's basis (``C Q^T``, C ~ N(0,1)) for flat spectra, or
    ``G diag(sigma) B^T`` over the full orthonormal ``B`` (first r columns = Q) for power-law
    spectra.  It is drawn directly in the cache's own layout.
    """
    n = wl.n_tokens * wl.g
    b = torch.from_numpy(_full_basis(wl, layer, branch)).to(device=device, dtype=torch.float32)
    if wl.power_law:
        sig = torch.tensor(power_law_sigma(wl.w), dtype=torch.float32, device=device)
        gmat = _randn(wl, layer, "signal_" + branch, (n, wl.w), device) * sig[None, :]
        x = gmat @ b.T
    else:
        r = wl.rank(layer, branch)
        c = _randn(wl, layer, "signal_" + branch, (n, r), device)
        x = c @ b[:, :r].T
    x = x + _randn(wl, layer, "noise_" + branch, (n, wl.w), device) * 0.1
    m = mu(wl, layer, branch, device)
    if m is not None:
        x = x + m.to(torch.float32)[None, :]
    return _cast(x.reshape(wl.n_tokens, wl.kv_width), wl, device)


def hidden(wl: Workload, layer: int, which: str, device="cpu") -> torch.Tensor:
    """RMS-normalised N(0,1) hidden state ``[T, d_model]`` (``which`` = 'h_in' or 'h_hat')."""
    x = _randn(wl, layer, which, (wl.n_tokens, wl.d_model), device)
    return _cast(_rms_normalize(x), wl, device)


def enc_h(wl: Workload, layer: int, device="cpu") -> torch.Tensor:
    """Patch-layer code projection ``W_enc,H`` stored ``[r_H, d_model]`` (orthonormal rows)."""
    r = wl.ranks[layer]
    g = np.random.default_rng(_seed(wl, layer, "enc_h"))
    q, rr = np.linalg.qr(g.standard_normal((wl.d_model, r)))
    q = q * np.sign(np.diag(rr))[None, :]
    return _cast(torch.from_numpy(q.T.copy()), wl, device)


def proj_weights(wl: Workload, layer: int, device="cpu"):
    """Consumer ``W_K, W_V ~ N(0, 1/d_model)`` stored ``[D, d_model]`` (k_proj/v_proj.weight)."""
    s = 1.0 / np.sqrt(wl.d_model)
    wk = _randn(wl, layer, "w_k", (wl.kv_width, wl.d_model), device) * s
    wv = _randn(wl, layer, "w_v", (wl.kv_width, wl.d_model), device) * s
    return _cast(wk, wl, device), _cast(wv, wl, device)


def proj_bias(wl: Workload, layer: int, device="cpu"):
    """Optional ``b_K, b_V ~ N(0, 0.1)`` of width D, or (None, None)."""
    if not wl.with_bias:
        return None, None
    bk = _randn(wl, layer, "b_k", (wl.kv_width,), "cpu") * np.sqrt(0.1)
    bv = _randn(wl, layer, "b_v", (wl.kv_width,), "cpu") * np.sqrt(0.1)
    return _cast(bk, wl, device), _cast(bv, wl, device)


def aligner_weights(wl: Workload, layer: int, device="cpu"):
    """Patch aligner of one layer, ``(W1 [h, r_H], b1 [h], W2 [d_model, h], b2 [d_model])``:
    ``W1 ~ N(0, 1/r_H)``, ``W2 ~ N(0, 1/h)``, biases ``N(0, 0.01)`` (random initialisation of the
    two-layer MLP; no trained aligner is available)."""
    r, h, d = wl.rank(layer, "h"), wl.hidden_width, wl.d_model
    w1 = _randn(wl, layer, "align_w1", (h, r), device) / np.sqrt(r)
    b1 = _randn(wl, layer, "align_b1", (h,), "cpu") * 0.1
    w2 = _randn(wl, layer, "align_w2", (d, h), device) / np.sqrt(h)
    b2 = _randn(wl, layer, "align_b2", (d,), "cpu") * 0.1
    return _cast(w1, wl, device), _cast(b1, wl, device), _cast(w2, wl, device), _cast(b2, wl, device)


def patch_codes(wl: Workload, layer: int, device="cpu") -> torch.Tensor:
    """Patch-layer codes ``Z_H [T, r_H]`` ~ N(0, 1), the aligner's input."""
    return _cast(_randn(wl, layer, "z_h", (wl.n_tokens, wl.rank(layer, "h")), device), wl, device)


def fit_spectrum(r: int) -> np.ndarray:
    """Scales of the shared latent's r directions: evenly spaced from 2 down to 1."""
    return np.linspace(2.0, 1.0, r)


def fit_pair(wl: Workload, layer: int, branch: str, device="cpu", sample: str = "cal"):
    """Paired calibration caches ``(A, B)`` [T, D] of one layer and branch: the producer's and the
    consumer's cache over the same prefixes, driven by one shared latent.  Per row of w channels:
    ``A = mu_A + C diag(s) Q_A^T + N(0, 0.01)`` and ``B = mu_B + C diag(s) Q_B^T + N(0, 0.01)``
    with ``C ~ N(0, 1)`` [T*g, r] shared, ``s`` from :func:`fit_spectrum`, ``Q_A``, ``Q_B``
    orthonormal [w, r] and offsets ``mu ~ N(0, 0.1)``.  Drawn directly in the cache layout.
    ``sample`` names an independent draw of the latent and the noise over the same bases and
    offsets (e.g. held-out rows of the same model pair)."""
    r = wl.rank(layer, branch)
    n = wl.n_tokens * wl.g
    tag = "" if sample == "cal" else sample + "_"
    c = _randn(wl, layer, f"fit_latent_{tag}{branch}", (n, r), device)
    c = c * torch.tensor(fit_spectrum(r), dtype=torch.float32, device=device)[None, :]
    out = []
    for side in ("a", "b"):
        g = np.random.default_rng(_seed(wl, layer, f"fit_basis_{side}_{branch}"))
        q, rr = np.linalg.qr(g.standard_normal((wl.w, r)))
        q = torch.from_numpy(q * np.sign(np.diag(rr))[None, :]).to(device=device,
                                                                    dtype=torch.float32)
        x = c @ q.T + _randn(wl, layer, f"fit_noise_{tag}{side}_{branch}", (n, wl.w), device) * 0.1
        x = x + _randn(wl, layer, f"fit_mu_{side}_{branch}", (wl.w,), "cpu").to(device) * np.sqrt(0.1)
        out.append(_cast(x.reshape(wl.n_tokens, wl.kv_width), wl, device))
    return out[0], out[1]


def cu_seqlens(wl: Workload, device="cpu") -> torch.Tensor:
    return torch.from_numpy(wl.cu_seqlens).to(device)


def pos0(wl: Workload, device="cpu") -> Optional[torch.Tensor]:
    if wl.pos0 is None:
        return None
    return torch.tensor(wl.pos0, dtype=torch.int32, device=device)


def layer_set(wl: Workload, layers: Optional[Sequence[int]] = None):
    return list(range(wl.n_layers)) if layers is None else list(layers)


# --------------------------------------------------------------------------------------------
# Whole input sets and output buffers
# --------------------------------------------------------------------------------------------
class Inputs:
    """All per-layer inputs of a workload on one device (None where a layer has no such tensor)."""

    def __init__(self, wl: Workload, device, encode=True, decode=True, patch=True):
        L = wl.n_layers
        R = [l for l in range(L) if not wl.is_patch[l]]
        P = [l for l in range(L) if wl.is_patch[l]]
        none = lambda: [None] * L  # noqa: E731
        self.wl = wl
        self.R, self.P = R, P
        self.w_enc_k, self.w_dec_k, self.w_enc_v, self.w_dec_v = none(), none(), none(), none()
        self.mu_k, self.mu_v = none(), none()
        self.z_k, self.z_v, self.k_in, self.v_in = none(), none(), none(), none()
        self.h_in, self.w_enc_h, self.h_hat = none(), none(), none()
        self.w_k, self.w_v, self.b_k, self.b_v = none(), none(), none(), none()
        for l in R:
            self.w_enc_k[l], self.w_dec_k[l] = basis(wl, l, "k", device)
            self.w_enc_v[l], self.w_dec_v[l] = basis(wl, l, "v", device)
            self.mu_k[l] = mu(wl, l, "k", device)
            self.mu_v[l] = mu(wl, l, "v", device)
            if decode:
                self.z_k[l] = codes(wl, l, "k", device)
                self.z_v[l] = codes(wl, l, "v", device)
            if encode:
                self.k_in[l] = kv_input(wl, l, "k", device)
                self.v_in[l] = kv_input(wl, l, "v", device)
        for l in P:
            if encode:
                self.h_in[l] = hidden(wl, l, "h_in", device)
                self.w_enc_h[l] = enc_h(wl, l, device)
            if patch:
                self.h_hat[l] = hidden(wl, l, "h_hat", device)
                self.w_k[l], self.w_v[l] = proj_weights(wl, l, device)
                self.b_k[l], self.b_v[l] = proj_bias(wl, l, device)


def alloc_caches(wl: Workload, device, fill=None):
    """Per-layer K and V caches [T, D]; optionally filled with a sentinel bit pattern."""
    ks, vs = [], []
    for _ in range(wl.n_layers):
        for lst in (ks, vs):
            t = torch.empty((wl.n_tokens, wl.kv_width), dtype=wl.torch_dtype, device=device)
            if fill is not None:
                t.fill_(fill)
            lst.append(t)
    return ks, vs


def alloc_codes(wl: Workload, device):
    L = wl.n_layers
    z_k, z_v, z_h = [None] * L, [None] * L, [None] * L
    for l in range(L):
        if wl.is_patch[l]:
            z_h[l] = torch.empty((wl.n_tokens, wl.ranks[l]), dtype=wl.torch_dtype, device=device)
        else:
            for lst, br in ((z_k, "k"), (z_v, "v")):
                lst[l] = torch.empty((wl.n_tokens * wl.g, wl.rank(l, br)), dtype=wl.torch_dtype,
                                     device=device)
    return z_k, z_v, z_h
