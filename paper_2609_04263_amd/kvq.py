"""Thin ctypes binding of libkvq.so (the C ABI in include/kvq.h).

Argument marshalling only: torch tensors provide device memory and the HIP
stream; every step of the path runs in the library's HIP kernels.  Importing
this module loads ``libkvq.so`` and raises if it is missing or cannot load
(there is no CPU fallback).  Names follow the C ABI without the ``kvq_``
prefix.
"""
from __future__ import annotations

import ctypes as C
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libkvq.so")

FORMAT_FIELDS = ("k_bits", "v_bits", "k_mode", "v_mode", "k_axis", "v_axis",
                 "k_group", "v_group", "residual", "flush", "rotate", "meta_fp16", "sink")

OK, ERR_ARG, ERR_FORMAT, ERR_CAPACITY, ERR_WORKSPACE, ERR_DEVICE, ERR_SCRATCH = range(7)
SCRATCH_BYTES = 4 << 20  # KVQ_SCRATCH_BYTES


class KvqError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {_lib.kvq_strerror(status).decode()} (status {status})")
        self.status = status


class Format(C.Structure):
    _fields_ = [(name, C.c_int32) for name in FORMAT_FIELDS]

    @classmethod
    def of(cls, fmt) -> "Format":
        if isinstance(fmt, Format):
            return fmt
        return cls(*[int(fmt.get(name, 0)) for name in FORMAT_FIELDS])


def _load() -> C.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                          "(the HIP library is required, there is no fallback)")
    L = C.CDLL(LIB_PATH)
    P, I, S = C.c_void_p, C.c_int, C.c_size_t
    Fp = C.POINTER(Format)
    L.kvq_strerror.argtypes = [I]
    L.kvq_strerror.restype = C.c_char_p
    L.kvq_cache_bytes.argtypes = [Fp, I, I, I, I, C.POINTER(S)]
    L.kvq_cache_init.argtypes = [Fp, I, I, I, I, P, S, C.POINTER(P)]
    L.kvq_cache_section.argtypes = [P, I, C.POINTER(S), C.POINTER(S)]
    L.kvq_cache_reset.argtypes = [P]
    L.kvq_cache_len.argtypes = [P, C.POINTER(I), C.POINTER(I)]
    L.kvq_cache_rewind.argtypes = [P, I]
    L.kvq_cache_restore.argtypes = [P, I]
    L.kvq_cache_destroy.argtypes = [P]
    L.kvq_cache_destroy.restype = None
    L.kvq_project_workspace_bytes.argtypes = [I, I, C.POINTER(S)]
    L.kvq_project_qkv.argtypes = [P, I, I, P, I, I, P, P, I, C.c_float, P, P, P, P, S, P]
    L.kvq_merge_adapter.argtypes = [P, I, I, I, P, P, I, C.c_float, P, P]
    L.kvq_project_append.argtypes = [P, I, I, P, I, I, P, P, I, C.c_float, P, P, I, P, S, P]
    L.kvq_append.argtypes = [P, P, P, I, Fp, P]
    L.kvq_decode_workspace_bytes.argtypes = [P, I, C.POINTER(S)]
    L.kvq_decode_attn.argtypes = [P, P, I, C.c_float, P, P, S, P]
    L.kvq_decode_attn_noalloc.argtypes = [P, P, I, C.c_float, P, P]
    L.kvq_prefill_attn.argtypes = [P, P, I, I, C.c_float, P, P, S, P]
    L.kvq_prefill_workspace_bytes.argtypes = [P, C.POINTER(S)]
    L.kvq_time_launches.argtypes = [P, P]
    for name in ("kvq_cache_bytes", "kvq_cache_init", "kvq_cache_section", "kvq_cache_reset",
                 "kvq_cache_len", "kvq_cache_rewind", "kvq_cache_restore", "kvq_project_workspace_bytes",
                 "kvq_project_qkv", "kvq_project_append", "kvq_merge_adapter", "kvq_append",
                 "kvq_decode_workspace_bytes", "kvq_decode_attn", "kvq_decode_attn_noalloc", "kvq_prefill_attn",
                 "kvq_prefill_workspace_bytes",
                 "kvq_time_launches"):
        getattr(L, name).restype = I
    return L


_lib = _load()
EXPORTED = ("kvq_strerror", "kvq_cache_bytes", "kvq_cache_init", "kvq_cache_section",
            "kvq_cache_reset", "kvq_cache_len", "kvq_cache_rewind", "kvq_cache_restore", "kvq_cache_destroy",
            "kvq_project_workspace_bytes", "kvq_project_qkv", "kvq_project_append", "kvq_merge_adapter", "kvq_append",
            "kvq_decode_workspace_bytes", "kvq_decode_attn", "kvq_decode_attn_noalloc", "kvq_prefill_attn",
            "kvq_prefill_workspace_bytes", "kvq_time_launches")


def lib() -> C.CDLL:
    return _lib


def _check(status: int, what: str) -> None:
    if status != OK:
        raise KvqError(status, what)


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


try:  # raw handle of torch's current stream without building a Stream object
    _raw_stream = torch._C._cuda_getCurrentRawStream
except AttributeError:  # pragma: no cover - older torch
    _raw_stream = None


def _stream(stream) -> int:
    if stream is None:
        if _raw_stream is not None:
            return _raw_stream(torch.cuda.current_device())
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


# ------------------------------------------------------------------ cache

def cache_bytes(fmt, B: int, H_kv: int, D: int, T_max: int) -> int:
    out = C.c_size_t()
    _check(_lib.kvq_cache_bytes(C.byref(Format.of(fmt)), B, H_kv, D, T_max, C.byref(out)), "cache_bytes")
    return out.value


class Cache:
    """A packed cache: caller-owned device storage (a zero-filled uint8 torch
    tensor) plus the library's host handle."""

    def __init__(self, fmt, B: int, H_kv: int, D: int, T_max: int, device="cuda", storage=None):
        self.fmt = Format.of(fmt)
        self.B, self.H, self.D, self.T_max = B, H_kv, D, T_max
        nbytes = cache_bytes(self.fmt, B, H_kv, D, T_max)
        if storage is None:
            storage = torch.zeros(nbytes, dtype=torch.uint8, device=device)
        self.storage = storage
        h = C.c_void_p()
        _check(_lib.kvq_cache_init(C.byref(self.fmt), B, H_kv, D, T_max, C.c_void_p(_ptr(storage)),
                                   storage.numel() * storage.element_size(), C.byref(h)), "cache_init")
        self.handle = h
        self._fmt_ref = C.byref(self.fmt)

    def __del__(self):
        h = getattr(self, "handle", None)
        if h is not None and h.value and _lib is not None:
            _lib.kvq_cache_destroy(h)
            self.handle = None

    def section(self, index: int):
        off, ln = C.c_size_t(), C.c_size_t()
        _check(_lib.kvq_cache_section(self.handle, index, C.byref(off), C.byref(ln)), "cache_section")
        return off.value, ln.value

    def reset(self) -> None:
        _check(_lib.kvq_cache_reset(self.handle), "cache_reset")

    def rewind(self, n: int) -> None:
        _check(_lib.kvq_cache_rewind(self.handle, n), "cache_rewind")

    def restore(self, n: int) -> None:
        """Length n after the storage was restored from a snapshot taken at n."""
        _check(_lib.kvq_cache_restore(self.handle, n), "cache_restore")

    def length(self):
        n, nc = C.c_int(), C.c_int()
        _check(_lib.kvq_cache_len(self.handle, C.byref(n), C.byref(nc)), "cache_len")
        return n.value, nc.value

    @property
    def n(self) -> int:
        return self.length()[0]

    def append(self, K, V, n_new: int | None = None, fmt=None, stream=None) -> None:
        """Append bf16 K, V [B, n_new, H_kv, D] (device tensors)."""
        if n_new is None:
            n_new = K.shape[1] if K.dim() == 4 else 1
        f = self._fmt_ref if fmt is None else C.byref(Format.of(fmt))
        st = _lib.kvq_append(self.handle, K.data_ptr(), V.data_ptr(), n_new, f, _stream(stream))
        if st:
            _check(st, "append")

    def decode_workspace_bytes(self, H_q: int) -> int:
        out = C.c_size_t()
        _check(_lib.kvq_decode_workspace_bytes(self.handle, H_q, C.byref(out)), "decode_workspace_bytes")
        return out.value

    def decode_workspace(self, H_q: int, device="cuda"):
        """A workspace of the required size (reuse it across calls)."""
        return torch.empty(self.decode_workspace_bytes(H_q), dtype=torch.uint8, device=device)

    def decode_attn(self, Q, H_q: int, sm_scale: float, O, workspace, stream=None) -> None:
        """O[B, H_q, D] (fp32) <- attention of bf16 Q[B, H_q, D] over the cache."""
        nbytes = workspace.numel() * workspace.element_size()
        st = _lib.kvq_decode_attn(self.handle, Q.data_ptr(), H_q, sm_scale, O.data_ptr(), workspace.data_ptr(),
                                  nbytes, _stream(stream))
        if st:
            _check(st, "decode_attn")

    def decode_attn_noalloc(self, Q, H_q: int, sm_scale: float, O, stream=None) -> None:
        """As decode_attn, with the split partials in the library's static
        scratch (no workspace, nothing allocated)."""
        st = _lib.kvq_decode_attn_noalloc(self.handle, Q.data_ptr(), H_q, sm_scale, O.data_ptr(), _stream(stream))
        if st:
            _check(st, "decode_attn_noalloc")

    def prefill_workspace_bytes(self) -> int:
        out = C.c_size_t()
        _check(_lib.kvq_prefill_workspace_bytes(self.handle, C.byref(out)), "prefill_workspace_bytes")
        return out.value

    def prefill_workspace(self, device="cuda"):
        """A workspace for prefill_attn at the cache's current length."""
        return torch.empty(self.prefill_workspace_bytes(), dtype=torch.uint8, device=device)

    def prefill_attn(self, Q, C_len: int, H_q: int, sm_scale: float, O, workspace, stream=None) -> None:
        """O[B, C, H_q, D] (fp32) <- causal attention of the newest C_len tokens'
        bf16 queries Q[B, C, H_q, D] over the cache."""
        nbytes = workspace.numel() * workspace.element_size()
        st = _lib.kvq_prefill_attn(self.handle, Q.data_ptr(), C_len, H_q, sm_scale, O.data_ptr(),
                                   workspace.data_ptr(), nbytes, _stream(stream))
        if st:
            _check(st, "prefill_attn")


# ------------------------------------------------------------- projection

def project_workspace_bytes(M: int, rank: int) -> int:
    out = C.c_size_t()
    _check(_lib.kvq_project_workspace_bytes(M, rank, C.byref(out)), "project_workspace_bytes")
    return out.value


def project_qkv(H, W, A, Bm, rank: int, lora_scale: float, d_q: int, d_kv: int, Q, K, V, workspace,
                stream=None) -> None:
    """Q/K/V (bf16) <- H W^T + lora_scale * (H A_p^T) B_p^T per projection."""
    M, d_in = H.shape[0], H.shape[-1]
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = _lib.kvq_project_qkv(_ptr(H), M, d_in, _ptr(W), d_q, d_kv, _ptr(A), _ptr(Bm), rank, lora_scale,
                              _ptr(Q), _ptr(K), _ptr(V), _ptr(workspace), nbytes, _stream(stream))
    if st:
        _check(st, "project_qkv")


def project_append(H, W, A, Bm, rank: int, lora_scale: float, d_q: int, d_kv: int, Q, cache: "Cache",
                   n_new: int, workspace, stream=None) -> None:
    """Q (bf16) as project_qkv; K and V coded straight into `cache` (n_new
    tokens of each sequence, rows of H sequence-major)."""
    M, d_in = H.shape[0], H.shape[-1]
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = _lib.kvq_project_append(_ptr(H), M, d_in, _ptr(W), d_q, d_kv, _ptr(A), _ptr(Bm), rank, lora_scale,
                                 _ptr(Q), cache.handle, n_new, _ptr(workspace), nbytes, _stream(stream))
    if st:
        _check(st, "project_append")


def merge_adapter(W, A, Bm, rank: int, lora_scale: float, d_q: int, d_kv: int, Wout, stream=None) -> None:
    """Wout (bf16) <- W + lora_scale * B_p A_p per projection (dense merge; Wout may be W)."""
    d_in = W.shape[-1]
    st = _lib.kvq_merge_adapter(_ptr(W), d_in, d_q, d_kv, _ptr(A), _ptr(Bm), rank, lora_scale, _ptr(Wout),
                                _stream(stream))
    if st:
        _check(st, "merge_adapter")


def time_launches(start_event, stop_event) -> None:
    """Measurement hook: while set, the library's kernels record the two
    hipEvent_t handles (ints) from their own dispatches (see
    kvq_time_launches); time_launches(None, None) clears it."""
    st = _lib.kvq_time_launches(start_event, stop_event)
    if st:
        _check(st, "time_launches")
