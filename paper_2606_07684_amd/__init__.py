"""MI355X-native SCD KV-state codec: the Python binding of ``libscd.so``.

Argument marshalling only.  Every step of the codec runs in the library's HIP kernels; PyTorch
provides device memory and the stream.  The functions carry the C entry points' names and
meaning (``include/scd.h``):

* :func:`scd_rope_table`   fp64-evaluated RoPE cos/sin table (build once per model)
* :func:`scd_positions`    per-token positions of a packed ragged batch
* :func:`scd_schedule`     Reuse / Patch layer lists (Section 4.1, Algorithm 1)
* :func:`scd_payload_bytes` bytes of the transmitted code set (Section 4.5)
* :func:`scd_encode`       producer encode (Eq. encode_z_kv; Section 4.4.1)
* :func:`scd_reuse_decode` consumer Reuse decode into the KV cache (Eq. decode_kv)
* :func:`scd_patch_kv`     consumer Patch KV regeneration into the KV cache (Eq. kv_from_patch)

If the library is missing the first call raises: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import List, Optional, Sequence

import torch

__all__ = [
    "Model", "Batch", "RopeTable", "ScdError", "lib_path", "load_library",
    "scd_rope_table", "scd_positions", "scd_schedule", "scd_payload_bytes",
    "scd_encode", "scd_reuse_decode", "scd_patch_kv", "scd_abi_version",
    "Prepared", "prepare_encode", "prepare_reuse_decode", "prepare_patch_kv",
    "scd_patch_align", "prepare_patch_align", "scd_payload_views",
    "scd_reuse_decode_streamed", "prepare_reuse_decode_streamed", "PreparedStreamed",
    "DEFAULT_LAYERS_PER_GROUP", "scd_patch_fold", "prepare_patch_fold",
    "scd_patch_kv_from_codes", "prepare_patch_kv_from_codes", "scd_fit_solve_noalloc",
    "prepare_fit_solve_noalloc", "scd_fit_solve_noalloc_max_bytes",
]

_PKG_DIR = os.path.dirname(os.path.abspath(__file__))
_LIB = None

SCD_F32, SCD_BF16 = 0, 1
# Layers per copy of the streamed receipt.  Each group boundary costs the copy stream a few tens
# of microseconds (the event between two copies), and the last group's decode is not overlapped;
# at 32 layers of 8K tokens, 8 layers per group balances the two.
DEFAULT_LAYERS_PER_GROUP = 8
_STATUS_NAMES = {0: "SCD_OK", 1: "SCD_ERR_NULL", 2: "SCD_ERR_SHAPE", 3: "SCD_ERR_SCHEDULE",
                 4: "SCD_ERR_ALIGN", 5: "SCD_ERR_UNSUPPORTED", 6: "SCD_ERR_WORKSPACE",
                 7: "SCD_ERR_HIP"}


class ScdError(RuntimeError):
    def __init__(self, status: int, detail: str):
        self.status = status
        self.status_name = _STATUS_NAMES.get(status, str(status))
        super().__init__(f"{self.status_name}: {detail}")


def lib_path() -> str:
    return os.path.join(_PKG_DIR, "libscd.so")


class _CModel(ctypes.Structure):
    _fields_ = [
        ("n_layers", ctypes.c_int32),
        ("d_model", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("basis_width", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("rope_theta", ctypes.c_double),
        ("is_patch", ctypes.POINTER(ctypes.c_uint8)),
        ("rank_k", ctypes.POINTER(ctypes.c_int32)),
        ("rank_v", ctypes.POINTER(ctypes.c_int32)),
        ("rank_h", ctypes.POINTER(ctypes.c_int32)),
    ]


class _CBatch(ctypes.Structure):
    _fields_ = [
        ("n_seqs", ctypes.c_int32),
        ("n_tokens", ctypes.c_int64),
        ("cu_seqlens", ctypes.c_void_p),
        ("pos0", ctypes.c_void_p),
    ]


_VP = ctypes.c_void_p
_PP = ctypes.POINTER(ctypes.c_void_p)
_SIGS = {
    "scd_abi_version": (ctypes.c_int32, []),
    "scd_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "scd_last_error": (ctypes.c_char_p, []),
    "scd_rope_table_bytes": (ctypes.c_size_t, [ctypes.POINTER(_CModel), ctypes.c_int64]),
    "scd_rope_table": (ctypes.c_int, [ctypes.POINTER(_CModel), ctypes.c_int64, _VP,
                                      ctypes.c_size_t, _VP]),
    "scd_positions": (ctypes.c_int, [ctypes.POINTER(_CBatch), _VP, _VP]),
    "scd_schedule": (ctypes.c_int, [ctypes.POINTER(_CModel), ctypes.POINTER(ctypes.c_int32),
                                    ctypes.POINTER(ctypes.c_int32),
                                    ctypes.POINTER(ctypes.c_int32),
                                    ctypes.POINTER(ctypes.c_int32)]),
    "scd_payload_bytes": (ctypes.c_size_t, [ctypes.POINTER(_CModel), ctypes.c_int64,
                                            ctypes.POINTER(ctypes.c_int64)]),
    "scd_encode": (ctypes.c_int, [ctypes.POINTER(_CModel), ctypes.POINTER(_CBatch), _VP,
                                  ctypes.c_int64] + [_PP] * 11 + [_VP]),
    "scd_reuse_decode": (ctypes.c_int, [ctypes.POINTER(_CModel), ctypes.POINTER(_CBatch), _VP,
                                        ctypes.c_int64] + [_PP] * 8 + [_VP]),
    "scd_patch_kv": (ctypes.c_int, [ctypes.POINTER(_CModel), ctypes.POINTER(_CBatch), _VP,
                                    ctypes.c_int64] + [_PP] * 7 + [_VP]),
    "scd_patch_align": (ctypes.c_int, [ctypes.POINTER(_CModel), ctypes.POINTER(_CBatch),
                                       ctypes.c_int32] + [_PP] * 7 + [_VP]),
    "scd_payload_views": (ctypes.c_int, [ctypes.POINTER(_CModel), ctypes.c_int64, _VP,
                                         _PP, _PP, _PP]),
    "scd_reuse_decode_streamed": (ctypes.c_int, [ctypes.POINTER(_CModel),
                                                 ctypes.POINTER(_CBatch), _VP, ctypes.c_int64,
                                                 _VP, _VP, ctypes.c_int32] + [_PP] * 6
                                  + [_VP, _VP]),
    "scd_fit_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(_CModel), ctypes.c_int64]),
    "scd_fit_gram": (ctypes.c_int, [ctypes.POINTER(_CModel), ctypes.POINTER(_CBatch), _VP,
                                    ctypes.c_int64, ctypes.c_int32] + [_PP] * 4
                     + [_VP, ctypes.c_size_t, _VP]),
    "scd_fit_solve": (ctypes.c_int, [ctypes.POINTER(_CModel), ctypes.c_int32, ctypes.c_int64,
                                     ctypes.c_double, ctypes.c_int32] + [_PP] * 6
                      + [_VP, ctypes.c_size_t, _VP]),
    "scd_patch_fold": (ctypes.c_int, [ctypes.POINTER(_CModel), ctypes.c_int32] + [_PP] * 10
                       + [_VP]),
    "scd_patch_kv_from_codes": (ctypes.c_int, [ctypes.POINTER(_CModel), ctypes.POINTER(_CBatch),
                                               _VP, ctypes.c_int64, ctypes.c_int32] + [_PP] * 10
                                + [_VP]),
    "scd_fit_solve_noalloc_max_bytes": (ctypes.c_size_t, []),
    "scd_fit_solve_noalloc": (ctypes.c_int, [ctypes.POINTER(_CModel), ctypes.c_int32,
                                             ctypes.c_int64, ctypes.c_double, ctypes.c_int32]
                              + [_PP] * 6 + [_VP]),
}
EXPORTED_SYMBOLS = tuple(_SIGS)


def load_library():
    """Load libscd.so (once).  Raises if it has not been built."""
    global _LIB
    if _LIB is None:
        path = lib_path()
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is missing: build it with "
                               "`python -m paper_2606_07684_amd.build` (there is no fallback)")
        lib = ctypes.CDLL(path)
        for name, (res, args) in _SIGS.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _LIB = lib
    return _LIB


def _check(status: int):
    if status != 0:
        raise ScdError(status, load_library().scd_last_error().decode())


def scd_abi_version() -> int:
    return int(load_library().scd_abi_version())


# ------------------------------------------------------------------------------------------------
# Descriptors
# ------------------------------------------------------------------------------------------------
@dataclasses.dataclass
class Model:
    """A producer/consumer model pair as the codec sees it (``scd_model_t``)."""
    n_layers: int
    d_model: int
    n_kv_heads: int
    head_dim: int
    rope_theta: float
    dtype: str                    # "f32" or "bf16"
    is_patch: Sequence[int]
    rank_k: Sequence[int]
    rank_v: Sequence[int]
    rank_h: Sequence[int]
    basis_width: Optional[int] = None  # None -> D = n_kv_heads * head_dim

    def __post_init__(self):
        if self.basis_width is None:
            self.basis_width = self.n_kv_heads * self.head_dim
        if self.dtype not in ("f32", "bf16"):
            raise ValueError("dtype must be 'f32' or 'bf16'")
        L = self.n_layers
        for name in ("is_patch", "rank_k", "rank_v", "rank_h"):
            if len(getattr(self, name)) != L:
                raise ValueError(f"{name} must have n_layers = {L} entries")
        self._keep = (
            (ctypes.c_uint8 * L)(*[1 if v else 0 for v in self.is_patch]),
            (ctypes.c_int32 * L)(*self.rank_k),
            (ctypes.c_int32 * L)(*self.rank_v),
            (ctypes.c_int32 * L)(*self.rank_h),
        )
        self._c = _CModel(L, self.d_model, self.n_kv_heads, self.head_dim, self.basis_width,
                          SCD_BF16 if self.dtype == "bf16" else SCD_F32, float(self.rope_theta),
                          *self._keep)

    @property
    def kv_width(self) -> int:
        return self.n_kv_heads * self.head_dim

    @property
    def g(self) -> int:
        return self.kv_width // self.basis_width

    @property
    def torch_dtype(self):
        return torch.bfloat16 if self.dtype == "bf16" else torch.float32

    @property
    def elem_bytes(self) -> int:
        return 2 if self.dtype == "bf16" else 4


@dataclasses.dataclass
class Batch:
    """A packed ragged batch (``scd_batch_t``): device ``cu_seqlens`` [B+1] int32, optional
    device ``pos0`` [B] int32.  ``cu_seqlens=None`` means one request of ``n_tokens`` tokens."""
    n_tokens: int
    cu_seqlens: Optional[torch.Tensor] = None
    pos0: Optional[torch.Tensor] = None

    def __post_init__(self):
        for name in ("cu_seqlens", "pos0"):
            t = getattr(self, name)
            if t is not None and (t.dtype != torch.int32 or not t.is_contiguous()):
                raise ValueError(f"{name} must be a contiguous int32 tensor")
        n_seqs = 1 if self.cu_seqlens is None else self.cu_seqlens.numel() - 1
        if self.pos0 is not None and self.pos0.numel() != n_seqs:
            raise ValueError("pos0 must have one entry per request")
        self._c = _CBatch(n_seqs, int(self.n_tokens),
                          None if self.cu_seqlens is None else self.cu_seqlens.data_ptr(),
                          None if self.pos0 is None else self.pos0.data_ptr())

    @property
    def n_seqs(self) -> int:
        return self._c.n_seqs


@dataclasses.dataclass
class RopeTable:
    """Device RoPE table filled by :func:`scd_rope_table` for positions ``[0, max_position)`` of a
    model with ``head_dim`` and ``rope_theta``; entry points check it against their model."""
    buffer: torch.Tensor
    max_position: int
    head_dim: int
    rope_theta: float


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _ptr_array(tensors, n_layers: int, name: str, shapes: dict, dtype) -> ctypes.Array:
    """Host array of device pointers for one per-layer argument (None entries -> NULL)."""
    if tensors is None:
        return None
    if len(tensors) != n_layers:
        raise ValueError(f"{name} must have one entry per layer ({n_layers})")
    arr = (ctypes.c_void_p * n_layers)()
    for l, t in enumerate(tensors):
        if t is None:
            continue
        if not isinstance(t, torch.Tensor) or not t.is_cuda:
            raise ValueError(f"{name}[{l}] must be a CUDA tensor")
        if t.dtype != dtype:
            raise ValueError(f"{name}[{l}] has dtype {t.dtype}, expected {dtype}")
        if not t.is_contiguous():
            raise ValueError(f"{name}[{l}] must be contiguous")
        want = shapes.get(l)
        if want is not None and tuple(t.shape) != tuple(want):
            raise ValueError(f"{name}[{l}] has shape {tuple(t.shape)}, expected {tuple(want)}")
        arr[l] = t.data_ptr()
    return arr


def _as_pp(arr):
    return None if arr is None else ctypes.cast(arr, _PP)


# ------------------------------------------------------------------------------------------------
# Entry points
# ------------------------------------------------------------------------------------------------
def scd_rope_table(model: Model, max_position: int, device=None, stream=None) -> RopeTable:
    lib = load_library()
    nbytes = int(lib.scd_rope_table_bytes(ctypes.byref(model._c), int(max_position)))
    if nbytes == 0:
        raise ValueError("invalid model or max_position for a RoPE table")
    device = device or torch.device("cuda", torch.cuda.current_device())
    buf = torch.empty(nbytes, dtype=torch.uint8, device=device)
    _check(lib.scd_rope_table(ctypes.byref(model._c), int(max_position), buf.data_ptr(), nbytes,
                              _stream(stream)))
    return RopeTable(buf, int(max_position), int(model.head_dim), float(model.rope_theta))


def scd_positions(batch: Batch, out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    lib = load_library()
    if out is None:
        dev = batch.cu_seqlens.device if batch.cu_seqlens is not None else torch.device("cuda")
        out = torch.empty(batch.n_tokens, dtype=torch.int32, device=dev)
    if out.dtype != torch.int32 or out.numel() != batch.n_tokens or not out.is_cuda:
        raise ValueError("out must be a CUDA int32 tensor of n_tokens entries")
    _check(lib.scd_positions(ctypes.byref(batch._c), out.data_ptr(), _stream(stream)))
    return out


def scd_schedule(model: Model):
    lib = load_library()
    L = model.n_layers
    reuse = (ctypes.c_int32 * L)()
    patch = (ctypes.c_int32 * L)()
    nr, np_ = ctypes.c_int32(), ctypes.c_int32()
    _check(lib.scd_schedule(ctypes.byref(model._c), reuse, ctypes.byref(nr), patch,
                            ctypes.byref(np_)))
    return list(reuse[:nr.value]), list(patch[:np_.value])


def scd_payload_bytes(model: Model, n_tokens: int):
    lib = load_library()
    offs = (ctypes.c_int64 * (model.n_layers + 1))()
    total = int(lib.scd_payload_bytes(ctypes.byref(model._c), int(n_tokens), offs))
    return total, list(offs)


def _rope_args(rope: Optional[RopeTable], model: "Model"):
    """Device pointer and max_position of a RoPE table built for this model (its head_dim and
    theta) and large enough for its max_position; the library reads max_position * head_dim / 2
    (cos, sin) pairs from it."""
    if rope is None:
        return None, 0
    if rope.head_dim != model.head_dim or rope.rope_theta != model.rope_theta:
        raise ValueError(f"RoPE table was built for head_dim {rope.head_dim}, theta "
                         f"{rope.rope_theta}; the model has {model.head_dim}, {model.rope_theta}")
    buf = rope.buffer
    if not isinstance(buf, torch.Tensor) or not buf.is_cuda or not buf.is_contiguous():
        raise ValueError("RoPE table buffer must be a contiguous CUDA tensor")
    need = int(load_library().scd_rope_table_bytes(ctypes.byref(model._c), int(rope.max_position)))
    if need == 0 or buf.numel() * buf.element_size() < need:
        raise ValueError(f"RoPE table holds {buf.numel() * buf.element_size()} bytes; "
                         f"max_position {rope.max_position} needs {need}")
    return buf.data_ptr(), rope.max_position


class Prepared:
    """An entry-point call with its arguments marshalled once; calling it launches the kernels on
    the given (or current) stream.  The referenced tensors must stay alive and unchanged in shape."""

    def __init__(self, fn, args, keep):
        self._fn, self._args, self._keep = fn, args, keep

    def __call__(self, stream=None) -> None:
        _check(self._fn(*self._args, _stream(stream)))


def prepare_encode(model: Model, batch: Batch, rope: Optional[RopeTable], k_in, v_in, h_in,
                   w_enc_k, w_enc_v, w_enc_h, mu_k, mu_v, z_k, z_v, z_h) -> Prepared:
    lib = load_library()
    L, T, D, w, g, d = (model.n_layers, batch.n_tokens, model.kv_width, model.basis_width,
                        model.g, model.d_model)
    dt = model.torch_dtype
    R = [l for l in range(L) if not model.is_patch[l]]
    P = [l for l in range(L) if model.is_patch[l]]
    args = [
        _ptr_array(k_in, L, "k_in", {l: (T, D) for l in R}, dt),
        _ptr_array(v_in, L, "v_in", {l: (T, D) for l in R}, dt),
        _ptr_array(h_in, L, "h_in", {l: (T, d) for l in P}, dt),
        _ptr_array(w_enc_k, L, "w_enc_k", {l: (model.rank_k[l], w) for l in R}, dt),
        _ptr_array(w_enc_v, L, "w_enc_v", {l: (model.rank_v[l], w) for l in R}, dt),
        _ptr_array(w_enc_h, L, "w_enc_h", {l: (model.rank_h[l], d) for l in P}, dt),
        _ptr_array(mu_k, L, "mu_k", {l: (w,) for l in R}, dt),
        _ptr_array(mu_v, L, "mu_v", {l: (w,) for l in R}, dt),
        _ptr_array(z_k, L, "z_k", {l: (T * g, model.rank_k[l]) for l in R}, dt),
        _ptr_array(z_v, L, "z_v", {l: (T * g, model.rank_v[l]) for l in R}, dt),
        _ptr_array(z_h, L, "z_h", {l: (T, model.rank_h[l]) for l in P}, dt),
    ]
    tab, maxp = _rope_args(rope, model)
    return Prepared(lib.scd_encode, (ctypes.byref(model._c), ctypes.byref(batch._c), tab, maxp,
                                     *[_as_pp(a) for a in args]), (model, batch, rope, args))


def scd_encode(model: Model, batch: Batch, rope: Optional[RopeTable], k_in, v_in, h_in,
               w_enc_k, w_enc_v, w_enc_h, mu_k, mu_v, z_k, z_v, z_h, stream=None) -> None:
    prepare_encode(model, batch, rope, k_in, v_in, h_in, w_enc_k, w_enc_v, w_enc_h, mu_k, mu_v,
                   z_k, z_v, z_h)(stream)


def prepare_reuse_decode(model: Model, batch: Batch, rope: Optional[RopeTable], z_k, z_v,
                         w_dec_k, w_dec_v, mu_k, mu_v, k_cache, v_cache) -> Prepared:
    lib = load_library()
    L, T, D, w, g = model.n_layers, batch.n_tokens, model.kv_width, model.basis_width, model.g
    dt = model.torch_dtype
    R = [l for l in range(L) if not model.is_patch[l]]
    args = [
        _ptr_array(z_k, L, "z_k", {l: (T * g, model.rank_k[l]) for l in R}, dt),
        _ptr_array(z_v, L, "z_v", {l: (T * g, model.rank_v[l]) for l in R}, dt),
        _ptr_array(w_dec_k, L, "w_dec_k", {l: (w, model.rank_k[l]) for l in R}, dt),
        _ptr_array(w_dec_v, L, "w_dec_v", {l: (w, model.rank_v[l]) for l in R}, dt),
        _ptr_array(mu_k, L, "mu_k", {l: (w,) for l in R}, dt),
        _ptr_array(mu_v, L, "mu_v", {l: (w,) for l in R}, dt),
        _ptr_array(k_cache, L, "k_cache", {l: (T, D) for l in R}, dt),
        _ptr_array(v_cache, L, "v_cache", {l: (T, D) for l in R}, dt),
    ]
    tab, maxp = _rope_args(rope, model)
    return Prepared(lib.scd_reuse_decode, (ctypes.byref(model._c), ctypes.byref(batch._c), tab,
                                           maxp, *[_as_pp(a) for a in args]),
                    (model, batch, rope, args))


def scd_reuse_decode(model: Model, batch: Batch, rope: Optional[RopeTable], z_k, z_v,
                     w_dec_k, w_dec_v, mu_k, mu_v, k_cache, v_cache, stream=None) -> None:
    prepare_reuse_decode(model, batch, rope, z_k, z_v, w_dec_k, w_dec_v, mu_k, mu_v, k_cache,
                         v_cache)(stream)


def prepare_patch_kv(model: Model, batch: Batch, rope: Optional[RopeTable], h_hat, w_k, w_v,
                     b_k, b_v, k_cache, v_cache) -> Prepared:
    lib = load_library()
    L, T, D, d = model.n_layers, batch.n_tokens, model.kv_width, model.d_model
    dt = model.torch_dtype
    P = [l for l in range(L) if model.is_patch[l]]
    args = [
        _ptr_array(h_hat, L, "h_hat", {l: (T, d) for l in P}, dt),
        _ptr_array(w_k, L, "w_k", {l: (D, d) for l in P}, dt),
        _ptr_array(w_v, L, "w_v", {l: (D, d) for l in P}, dt),
        _ptr_array(b_k, L, "b_k", {l: (D,) for l in P}, dt),
        _ptr_array(b_v, L, "b_v", {l: (D,) for l in P}, dt),
        _ptr_array(k_cache, L, "k_cache", {l: (T, D) for l in P}, dt),
        _ptr_array(v_cache, L, "v_cache", {l: (T, D) for l in P}, dt),
    ]
    tab, maxp = _rope_args(rope, model)
    return Prepared(lib.scd_patch_kv, (ctypes.byref(model._c), ctypes.byref(batch._c), tab, maxp,
                                       *[_as_pp(a) for a in args]), (model, batch, rope, args))


def scd_patch_kv(model: Model, batch: Batch, rope: Optional[RopeTable], h_hat, w_k, w_v,
                 b_k, b_v, k_cache, v_cache, stream=None) -> None:
    prepare_patch_kv(model, batch, rope, h_hat, w_k, w_v, b_k, b_v, k_cache, v_cache)(stream)


def prepare_patch_align(model: Model, batch: Batch, hidden: int, z_h, w1, b1, w2, b2, act,
                        h_hat) -> Prepared:
    """The Patch aligner (Eq. aligner): act = SiLU(z_h w1^T + b1), h_hat = act w2^T + b2 for every
    Patch layer; act is caller-owned scratch, one distinct [T, hidden] buffer per Patch layer."""
    lib = load_library()
    L, T, d = model.n_layers, batch.n_tokens, model.d_model
    dt = model.torch_dtype
    P = [l for l in range(L) if model.is_patch[l]]
    args = [
        _ptr_array(z_h, L, "z_h", {l: (T, model.rank_h[l]) for l in P}, dt),
        _ptr_array(w1, L, "w1", {l: (hidden, model.rank_h[l]) for l in P}, dt),
        _ptr_array(b1, L, "b1", {l: (hidden,) for l in P}, dt),
        _ptr_array(w2, L, "w2", {l: (d, hidden) for l in P}, dt),
        _ptr_array(b2, L, "b2", {l: (d,) for l in P}, dt),
        _ptr_array(act, L, "act", {l: (T, hidden) for l in P}, dt),
        _ptr_array(h_hat, L, "h_hat", {l: (T, d) for l in P}, dt),
    ]
    return Prepared(lib.scd_patch_align, (ctypes.byref(model._c), ctypes.byref(batch._c),
                                          int(hidden), *[_as_pp(a) for a in args]),
                    (model, batch, args))


def scd_patch_align(model: Model, batch: Batch, hidden: int, z_h, w1, b1, w2, b2, act, h_hat,
                    stream=None) -> None:
    prepare_patch_align(model, batch, hidden, z_h, w1, b1, w2, b2, act, h_hat)(stream)


def prepare_patch_fold(model: Model, hidden: int, w2, b2, w_k, w_v, b_k, b_v, w_fold_k, w_fold_v,
                       c_k, c_v) -> Prepared:
    """Fold the aligner's output layer into the consumer's projections (once per model pair):
    w_fold = W_P w2 [D, hidden] and c = W_P b2 + b_P [D] for P = K, V and every Patch layer."""
    lib = load_library()
    L, D, d = model.n_layers, model.kv_width, model.d_model
    dt = model.torch_dtype
    P = [l for l in range(L) if model.is_patch[l]]
    args = [
        _ptr_array(w2, L, "w2", {l: (d, hidden) for l in P}, dt),
        _ptr_array(b2, L, "b2", {l: (d,) for l in P}, dt),
        _ptr_array(w_k, L, "w_k", {l: (D, d) for l in P}, dt),
        _ptr_array(w_v, L, "w_v", {l: (D, d) for l in P}, dt),
        _ptr_array(b_k, L, "b_k", {l: (D,) for l in P}, dt),
        _ptr_array(b_v, L, "b_v", {l: (D,) for l in P}, dt),
        _ptr_array(w_fold_k, L, "w_fold_k", {l: (D, hidden) for l in P}, dt),
        _ptr_array(w_fold_v, L, "w_fold_v", {l: (D, hidden) for l in P}, dt),
        _ptr_array(c_k, L, "c_k", {l: (D,) for l in P}, dt),
        _ptr_array(c_v, L, "c_v", {l: (D,) for l in P}, dt),
    ]
    return Prepared(lib.scd_patch_fold, (ctypes.byref(model._c), int(hidden),
                                         *[_as_pp(a) for a in args]), (model, args))


def scd_patch_fold(model: Model, hidden: int, w2, b2, w_k, w_v, b_k, b_v, w_fold_k, w_fold_v,
                   c_k, c_v, stream=None) -> None:
    prepare_patch_fold(model, hidden, w2, b2, w_k, w_v, b_k, b_v, w_fold_k, w_fold_v, c_k,
                       c_v)(stream)


def prepare_patch_kv_from_codes(model: Model, batch: Batch, rope: Optional[RopeTable], hidden: int,
                                z_h, w1, b1, w_fold_k, w_fold_v, c_k, c_v, act, k_cache,
                                v_cache) -> Prepared:
    """Patch from the transmitted codes: act = SiLU(z_h w1^T + b1), then
    K = RoPE(act w_fold_k^T + c_k), V = act w_fold_v^T + c_v into the cache, layer by layer
    (act entries may repeat: one [T, hidden] buffer can serve every Patch layer)."""
    lib = load_library()
    L, T, D = model.n_layers, batch.n_tokens, model.kv_width
    dt = model.torch_dtype
    P = [l for l in range(L) if model.is_patch[l]]
    args = [
        _ptr_array(z_h, L, "z_h", {l: (T, model.rank_h[l]) for l in P}, dt),
        _ptr_array(w1, L, "w1", {l: (hidden, model.rank_h[l]) for l in P}, dt),
        _ptr_array(b1, L, "b1", {l: (hidden,) for l in P}, dt),
        _ptr_array(w_fold_k, L, "w_fold_k", {l: (D, hidden) for l in P}, dt),
        _ptr_array(w_fold_v, L, "w_fold_v", {l: (D, hidden) for l in P}, dt),
        _ptr_array(c_k, L, "c_k", {l: (D,) for l in P}, dt),
        _ptr_array(c_v, L, "c_v", {l: (D,) for l in P}, dt),
        _ptr_array(act, L, "act", {l: (T, hidden) for l in P}, dt),
        _ptr_array(k_cache, L, "k_cache", {l: (T, D) for l in P}, dt),
        _ptr_array(v_cache, L, "v_cache", {l: (T, D) for l in P}, dt),
    ]
    tab, maxp = _rope_args(rope, model)
    return Prepared(lib.scd_patch_kv_from_codes,
                    (ctypes.byref(model._c), ctypes.byref(batch._c), tab, maxp, int(hidden),
                     *[_as_pp(a) for a in args]), (model, batch, rope, args))


def scd_patch_kv_from_codes(model: Model, batch: Batch, rope: Optional[RopeTable], hidden: int,
                            z_h, w1, b1, w_fold_k, w_fold_v, c_k, c_v, act, k_cache, v_cache,
                            stream=None) -> None:
    prepare_patch_kv_from_codes(model, batch, rope, hidden, z_h, w1, b1, w_fold_k, w_fold_v, c_k,
                                c_v, act, k_cache, v_cache)(stream)


def _payload_buffer(t, name: str, nbytes: int, need_cuda: bool) -> torch.Tensor:
    if not isinstance(t, torch.Tensor) or t.dtype != torch.uint8 or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous uint8 tensor")
    if need_cuda and not t.is_cuda:
        raise ValueError(f"{name} must be a CUDA tensor")
    if t.numel() < nbytes:
        raise ValueError(f"{name} holds {t.numel()} bytes, the payload needs {nbytes}")
    return t


def scd_payload_views(model: Model, n_tokens: int, payload: torch.Tensor):
    """Per-layer code tensors inside one packed payload buffer (uint8, scd_payload_bytes bytes):
    returns (z_k, z_v, z_h), lists of n_layers entries, None where a layer has no such branch.
    The addresses come from the library; the views only wrap them."""
    lib = load_library()
    L, T, g = model.n_layers, int(n_tokens), model.g
    total, _ = scd_payload_bytes(model, T)
    _payload_buffer(payload, "payload", total, need_cuda=False)
    arrs = [(ctypes.c_void_p * L)() for _ in range(3)]
    _check(lib.scd_payload_views(ctypes.byref(model._c), T, payload.data_ptr(),
                                 *[_as_pp(a) for a in arrs]))
    base, dt, eb = payload.data_ptr(), model.torch_dtype, model.elem_bytes
    shapes = (lambda l: (T * g, model.rank_k[l]), lambda l: (T * g, model.rank_v[l]),
              lambda l: (T, model.rank_h[l]))
    views = []
    for arr, shape in zip(arrs, shapes):
        out = []
        for l in range(L):
            if not arr[l]:
                out.append(None)
                continue
            rows, cols = shape(l)
            off = arr[l] - base
            out.append(payload[off:off + rows * cols * eb].view(dt).view(rows, cols))
        views.append(out)
    return tuple(views)


def prepare_reuse_decode_streamed(model: Model, batch: Batch, rope: Optional[RopeTable],
                                  payload_src: torch.Tensor, payload_dst: torch.Tensor,
                                  layers_per_group: int, w_dec_k, w_dec_v, mu_k, mu_v, k_cache,
                                  v_cache) -> "PreparedStreamed":
    """Receipt of a packed payload: copy it from payload_src (pinned host or device memory) to
    payload_dst (device) in groups of layers_per_group layers on the copy stream, decoding each
    group's Reuse layers on the compute stream as soon as it has landed."""
    lib = load_library()
    L, T, D, w = model.n_layers, batch.n_tokens, model.kv_width, model.basis_width
    dt = model.torch_dtype
    total, _ = scd_payload_bytes(model, T)
    _payload_buffer(payload_src, "payload_src", total, need_cuda=False)
    _payload_buffer(payload_dst, "payload_dst", total, need_cuda=True)
    R = [l for l in range(L) if not model.is_patch[l]]
    args = [
        _ptr_array(w_dec_k, L, "w_dec_k", {l: (w, model.rank_k[l]) for l in R}, dt),
        _ptr_array(w_dec_v, L, "w_dec_v", {l: (w, model.rank_v[l]) for l in R}, dt),
        _ptr_array(mu_k, L, "mu_k", {l: (w,) for l in R}, dt),
        _ptr_array(mu_v, L, "mu_v", {l: (w,) for l in R}, dt),
        _ptr_array(k_cache, L, "k_cache", {l: (T, D) for l in R}, dt),
        _ptr_array(v_cache, L, "v_cache", {l: (T, D) for l in R}, dt),
    ]
    tab, maxp = _rope_args(rope, model)
    return PreparedStreamed(lib.scd_reuse_decode_streamed,
                            (ctypes.byref(model._c), ctypes.byref(batch._c), tab, maxp,
                             payload_src.data_ptr(), payload_dst.data_ptr(),
                             int(layers_per_group), *[_as_pp(a) for a in args]),
                            (model, batch, rope, payload_src, payload_dst, args))


class PreparedStreamed(Prepared):
    """A prepared streamed receipt: called with (copy_stream, stream)."""

    def __call__(self, copy_stream=None, stream=None) -> None:
        _check(self._fn(*self._args, _stream(copy_stream), _stream(stream)))


def scd_reuse_decode_streamed(model: Model, batch: Batch, rope: Optional[RopeTable],
                              payload_src, payload_dst, layers_per_group: int, w_dec_k, w_dec_v,
                              mu_k, mu_v, k_cache, v_cache, copy_stream=None,
                              stream=None) -> None:
    prepare_reuse_decode_streamed(model, batch, rope, payload_src, payload_dst,
                                  layers_per_group, w_dec_k, w_dec_v, mu_k, mu_v, k_cache,
                                  v_cache)(copy_stream, stream)


# ------------------------------------------------------------------------------------------------
# Offline Reuse fit
# ------------------------------------------------------------------------------------------------
FIT_KEYS, FIT_VALUES = 0, 1


def scd_fit_workspace_bytes(model: Model, n_tokens: int) -> int:
    return int(load_library().scd_fit_workspace_bytes(ctypes.byref(model._c), int(n_tokens)))


def _workspace_arg(workspace: torch.Tensor):
    if not isinstance(workspace, torch.Tensor) or not workspace.is_cuda:
        raise ValueError("workspace must be a CUDA tensor")
    if not workspace.is_contiguous():
        raise ValueError("workspace must be contiguous")
    return workspace.data_ptr(), workspace.numel() * workspace.element_size()


def prepare_fit_gram(model: Model, batch: Batch, rope: Optional[RopeTable], branch: int, a_in,
                     b_in, gram, colsum, workspace: torch.Tensor) -> Prepared:
    lib = load_library()
    L, T, D, w = model.n_layers, batch.n_tokens, model.kv_width, model.basis_width
    dt = model.torch_dtype
    R = [l for l in range(L) if not model.is_patch[l]]
    args = [
        _ptr_array(a_in, L, "a_in", {l: (T, D) for l in R}, dt),
        _ptr_array(b_in, L, "b_in", {l: (T, D) for l in R}, dt),
        _ptr_array(gram, L, "gram", {l: (2 * w, 2 * w) for l in R}, torch.float32),
        _ptr_array(colsum, L, "colsum", {l: (2 * w,) for l in R}, torch.float32),
    ]
    ws, nbytes = _workspace_arg(workspace)
    tab, maxp = _rope_args(rope, model)
    return Prepared(lib.scd_fit_gram, (ctypes.byref(model._c), ctypes.byref(batch._c), tab, maxp,
                                       int(branch), *[_as_pp(a) for a in args], ws, nbytes),
                    (model, batch, rope, args, workspace))


def scd_fit_gram(model: Model, batch: Batch, rope: Optional[RopeTable], branch: int, a_in, b_in,
                 gram, colsum, workspace: torch.Tensor, stream=None) -> None:
    prepare_fit_gram(model, batch, rope, branch, a_in, b_in, gram, colsum, workspace)(stream)


def prepare_fit_solve(model: Model, branch: int, n_rows: int, ridge_lambda: float, center: bool,
                      gram, colsum, w_enc, w_dec, mu_enc, mu_dec,
                      workspace: torch.Tensor) -> Prepared:
    lib = load_library()
    L, w = model.n_layers, model.basis_width
    dt = model.torch_dtype
    R = [l for l in range(L) if not model.is_patch[l]]
    ranks = model.rank_k if branch == FIT_KEYS else model.rank_v
    args = [
        _ptr_array(gram, L, "gram", {l: (2 * w, 2 * w) for l in R}, torch.float32),
        _ptr_array(colsum, L, "colsum", {l: (2 * w,) for l in R}, torch.float32),
        _ptr_array(w_enc, L, "w_enc", {l: (ranks[l], w) for l in R}, dt),
        _ptr_array(w_dec, L, "w_dec", {l: (w, ranks[l]) for l in R}, dt),
        _ptr_array(mu_enc, L, "mu_enc", {l: (w,) for l in R}, dt),
        _ptr_array(mu_dec, L, "mu_dec", {l: (w,) for l in R}, dt),
    ]
    ws, nbytes = _workspace_arg(workspace)
    return Prepared(lib.scd_fit_solve, (ctypes.byref(model._c), int(branch), int(n_rows),
                                        float(ridge_lambda), 1 if center else 0,
                                        *[_as_pp(a) for a in args], ws, nbytes),
                    (model, args, workspace))


def scd_fit_solve(model: Model, branch: int, n_rows: int, ridge_lambda: float, center: bool,
                  gram, colsum, w_enc, w_dec, mu_enc, mu_dec, workspace: torch.Tensor,
                  stream=None) -> None:
    prepare_fit_solve(model, branch, n_rows, ridge_lambda, center, gram, colsum, w_enc, w_dec,
                      mu_enc, mu_dec, workspace)(stream)


def scd_fit_solve_noalloc_max_bytes() -> int:
    return int(load_library().scd_fit_solve_noalloc_max_bytes())


def prepare_fit_solve_noalloc(model: Model, branch: int, n_rows: int, ridge_lambda: float,
                              center: bool, gram, colsum, w_enc, w_dec, mu_enc,
                              mu_dec) -> Prepared:
    """scd_fit_solve without a workspace: the library's device-resident scratch array holds the
    solve's matrices (calls that overlap on one GPU race on it)."""
    lib = load_library()
    L, w = model.n_layers, model.basis_width
    dt = model.torch_dtype
    R = [l for l in range(L) if not model.is_patch[l]]
    ranks = model.rank_k if branch == FIT_KEYS else model.rank_v
    args = [
        _ptr_array(gram, L, "gram", {l: (2 * w, 2 * w) for l in R}, torch.float32),
        _ptr_array(colsum, L, "colsum", {l: (2 * w,) for l in R}, torch.float32),
        _ptr_array(w_enc, L, "w_enc", {l: (ranks[l], w) for l in R}, dt),
        _ptr_array(w_dec, L, "w_dec", {l: (w, ranks[l]) for l in R}, dt),
        _ptr_array(mu_enc, L, "mu_enc", {l: (w,) for l in R}, dt),
        _ptr_array(mu_dec, L, "mu_dec", {l: (w,) for l in R}, dt),
    ]
    return Prepared(lib.scd_fit_solve_noalloc, (ctypes.byref(model._c), int(branch), int(n_rows),
                                                float(ridge_lambda), 1 if center else 0,
                                                *[_as_pp(a) for a in args]), (model, args))


def scd_fit_solve_noalloc(model: Model, branch: int, n_rows: int, ridge_lambda: float,
                          center: bool, gram, colsum, w_enc, w_dec, mu_enc, mu_dec,
                          stream=None) -> None:
    prepare_fit_solve_noalloc(model, branch, n_rows, ridge_lambda, center, gram, colsum, w_enc,
                              w_dec, mu_enc, mu_dec)(stream)


def fit_reuse(model: Model, batch: Batch, rope: Optional[RopeTable], branch: int, a_in, b_in,
              ridge_lambda: float, center: bool = True, stream=None):
    """Both fit calls with freshly allocated outputs: returns per-layer lists
    ``(w_enc, w_dec, mu_enc, mu_dec, gram, colsum)`` (None for Patch layers; the offsets are None
    without centring)."""
    L, w = model.n_layers, model.basis_width
    R = [l for l in range(L) if not model.is_patch[l]]
    dev = next(t.device for t in a_in if t is not None)
    dt = model.torch_dtype
    ranks = model.rank_k if branch == FIT_KEYS else model.rank_v
    ws = torch.empty(max(scd_fit_workspace_bytes(model, batch.n_tokens), 16), dtype=torch.uint8,
                     device=dev)
    gram, colsum, w_enc, w_dec, mu_enc, mu_dec = ([None] * L for _ in range(6))
    for l in R:
        gram[l] = torch.empty((2 * w, 2 * w), dtype=torch.float32, device=dev)
        colsum[l] = torch.empty((2 * w,), dtype=torch.float32, device=dev)
        w_enc[l] = torch.empty((ranks[l], w), dtype=dt, device=dev)
        w_dec[l] = torch.empty((w, ranks[l]), dtype=dt, device=dev)
        if center:
            mu_enc[l] = torch.empty((w,), dtype=dt, device=dev)
            mu_dec[l] = torch.empty((w,), dtype=dt, device=dev)
    scd_fit_gram(model, batch, rope, branch, a_in, b_in, gram, colsum, ws, stream)
    scd_fit_solve(model, branch, batch.n_tokens * model.g, ridge_lambda, center, gram, colsum,
                  w_enc, w_dec, mu_enc if center else None, mu_dec if center else None, ws, stream)
    return w_enc, w_dec, mu_enc, mu_dec, gram, colsum

