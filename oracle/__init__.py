"""CPU oracle for the packed low-bit KV-cache decode path.

TEST INFRASTRUCTURE ONLY.  This package is the plain, slow reference that
the GPU library is checked against.  Only the test suite, the smoke check
(``__graft_entry__.smoke``) and the CPU-baseline leg of ``bench.py`` may
import it; the product package never does, and it imports nothing from the
product package.  The arithmetic lives in ``kvq_oracle.c`` (plain C, built
with gcc ``-O2 -ffp-contract=off``); this module only marshals numpy arrays.

Paper: "Quality Recovery for Quantized KV Caches via Low-Rank Attention
Adaptation".  Entry points and the passages they follow:

* :func:`project`        -- Sec. 3 Eq. (1)-(2), Sec. 3.4 (explicit adapter).
* :func:`merge_adapter`  -- Sec. 3.4 (dense-merge deployment W + (alpha/r) B A).
* :func:`quant_affine`   -- Sec. 3.1 Eq. (3).
* :func:`quant_sym`      -- Sec. 3.1, symmetric control (a reading).
* :func:`fwht_f32`       -- Sec. 3.1, fixed normalized Hadamard transform.
* :class:`Cache`         -- Sec. 3.1 physical incremental cache (append,
  reconstruction) and Sec. 3.1-3.2 attention over the reconstruction:
  decode (one query per sequence) and chunked prefill (the chunk's queries,
  causal, after the chunk is appended).

A bf16 tensor is passed as a ``uint16`` numpy array of its bit patterns.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "kvq_oracle.c")
_LIB = os.path.join(_HERE, "libkvq_oracle.so")

FORMAT_FIELDS = ("k_bits", "v_bits", "k_mode", "v_mode", "k_axis", "v_axis",
                 "k_group", "v_group", "residual", "flush", "rotate", "meta_fp16", "sink")

N_SECTIONS = 10  # Kc Ks Kz Vc Vs Vz Kr Vr Kq Vq

ERRORS = {0: "ok", 1: "bad argument", 2: "bad format", 3: "capacity exceeded",
          4: "non-finite input", 5: "out of memory"}


class OracleError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {ERRORS.get(status, status)}")
        self.status = status


class _Format(C.Structure):
    _fields_ = [(name, C.c_int) for name in FORMAT_FIELDS]


def build(force: bool = True) -> str:
    """Compile the oracle with gcc into ``oracle/libkvq_oracle.so``."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.run(["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
                        "-Wall", "-Wextra", "-fPIC", "-shared", _SRC, "-o", tmp, "-lm"],
                       check=True)
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib() -> C.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = C.CDLL(_LIB)
        P = C.c_void_p
        L.orc_f32_to_f16.argtypes = [C.c_float]
        L.orc_f32_to_f16.restype = C.c_uint16
        L.orc_f16_to_f32.argtypes = [C.c_uint16]
        L.orc_f16_to_f32.restype = C.c_float
        L.orc_f64_to_bf16.argtypes = [C.c_double]
        L.orc_f64_to_bf16.restype = C.c_uint16
        L.orc_quant_affine.argtypes = [P, C.c_int, C.c_int, P, P, P]
        L.orc_quant_sym.argtypes = [P, C.c_int, C.c_int, P, P]
        L.orc_quant_affine16.argtypes = [P, C.c_int, C.c_int, P, P, P]
        L.orc_quant_sym16.argtypes = [P, C.c_int, C.c_int, P, P]
        L.orc_pack_word.argtypes = [P, C.c_int]
        L.orc_pack_word.restype = C.c_uint32
        L.orc_unpack_word.argtypes = [C.c_uint32, C.c_int, P]
        L.orc_fwht_f32.argtypes = [P, C.c_int]
        L.orc_check_format.argtypes = [C.POINTER(_Format), C.c_int]
        L.orc_layout.argtypes = [C.POINTER(_Format), C.c_int, C.c_int, C.c_int, C.c_int, P, P, P]
        L.orc_num_coded.argtypes = [C.POINTER(_Format), C.c_int]
        L.orc_append.argtypes = [C.POINTER(_Format), C.c_int, C.c_int, C.c_int, C.c_int, P,
                                 C.POINTER(C.c_int), P, P, C.c_int]
        L.orc_dequant.argtypes = [C.POINTER(_Format), C.c_int, C.c_int, C.c_int, C.c_int, P,
                                  C.c_int, P, P]
        L.orc_decode_attn.argtypes = [C.POINTER(_Format), C.c_int, C.c_int, C.c_int, C.c_int, P,
                                      C.c_int, P, C.c_int, C.c_double, P]
        L.orc_prefill_attn.argtypes = [C.POINTER(_Format), C.c_int, C.c_int, C.c_int, C.c_int, P,
                                       C.c_int, C.c_int, P, C.c_int, C.c_double, P]
        L.orc_project.argtypes = [P, C.c_int, C.c_int, P, C.c_int, C.c_int, P, P, C.c_int,
                                  C.c_double, P, P]
        L.orc_merge_adapter.argtypes = [P, C.c_int, C.c_int, C.c_int, P, P, C.c_int, C.c_double, P, P]
        L.orc_set_threads.argtypes = [C.c_int]
        L.orc_set_threads.restype = None
        L.orc_get_threads.restype = C.c_int
        _lib = L
    return _lib


def _ptr(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"], "oracle arrays must be C-contiguous"
    return a.ctypes.data_as(C.c_void_p)


def _fmt(fmt) -> _Format:
    return _Format(*[int(fmt.get(name, 0)) for name in FORMAT_FIELDS])


# ---------------------------------------------------------------- threads

def set_threads(n: int) -> None:
    """OpenMP threads for the loops over independent units (results are the
    same for any count)."""
    lib().orc_set_threads(int(n))


def get_threads() -> int:
    return int(lib().orc_get_threads())


# ---------------------------------------------------------------- scalars

def f32_to_f16(x) -> np.ndarray:
    """binary32 -> binary16 bit patterns, round to nearest even (oracle's own)."""
    x = np.asarray(x, dtype=np.float32)
    L = lib()
    return np.array([L.orc_f32_to_f16(float(v)) for v in x.ravel()], dtype=np.uint16).reshape(x.shape)


def f16_to_f32(h) -> np.ndarray:
    h = np.asarray(h, dtype=np.uint16)
    L = lib()
    return np.array([L.orc_f16_to_f32(int(v)) for v in h.ravel()], dtype=np.float32).reshape(h.shape)


def f64_to_bf16(x) -> np.ndarray:
    x = np.asarray(x, dtype=np.float64)
    L = lib()
    return np.array([L.orc_f64_to_bf16(float(v)) for v in x.ravel()], dtype=np.uint16).reshape(x.shape)


# ----------------------------------------------------------------- coding

def quant_affine(x, bits: int):
    """Eq. (3) on one group: returns (codes uint8, scale float32, offset float32)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    codes = np.zeros(x.size, dtype=np.uint8)
    s = np.zeros(1, dtype=np.float32)
    z = np.zeros(1, dtype=np.float32)
    lib().orc_quant_affine(_ptr(x), x.size, bits, _ptr(codes), _ptr(s), _ptr(z))
    return codes, s[0], z[0]


def quant_sym(x, bits: int):
    """Symmetric control on one group: returns (unsigned codes, scale)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    codes = np.zeros(x.size, dtype=np.uint8)
    s = np.zeros(1, dtype=np.float32)
    lib().orc_quant_sym(_ptr(x), x.size, bits, _ptr(codes), _ptr(s))
    return codes, s[0]


def quant_affine16(x, bits: int):
    """Eq. (3) with fp16 metadata: returns (codes, scale fp16 bits, offset fp16 bits)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    codes = np.zeros(x.size, dtype=np.uint8)
    s = np.zeros(1, dtype=np.uint16)
    z = np.zeros(1, dtype=np.uint16)
    lib().orc_quant_affine16(_ptr(x), x.size, bits, _ptr(codes), _ptr(s), _ptr(z))
    return codes, s[0], z[0]


def quant_sym16(x, bits: int):
    """Symmetric control with an fp16 scale: returns (codes, scale fp16 bits)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    codes = np.zeros(x.size, dtype=np.uint8)
    s = np.zeros(1, dtype=np.uint16)
    lib().orc_quant_sym16(_ptr(x), x.size, bits, _ptr(codes), _ptr(s))
    return codes, s[0]


def pack_word(codes, bits: int) -> int:
    c = np.ascontiguousarray(codes, dtype=np.uint8)
    assert c.size == 32 // bits
    return int(lib().orc_pack_word(_ptr(c), bits))


def unpack_word(word: int, bits: int) -> np.ndarray:
    out = np.zeros(32 // bits, dtype=np.uint8)
    lib().orc_unpack_word(C.c_uint32(word), bits, _ptr(out))
    return out


def fwht_f32(x) -> np.ndarray:
    """Normalized Hadamard transform of the last axis, binary32, fixed stage order."""
    y = np.array(x, dtype=np.float32, copy=True, order="C")
    n = y.shape[-1]
    flat = y.reshape(-1, n)
    for row in flat:
        lib().orc_fwht_f32(_ptr(row), n)
    return flat.reshape(y.shape)


# ------------------------------------------------------------------ cache

def check_format(fmt, D: int) -> int:
    f = _fmt(fmt)
    return int(lib().orc_check_format(C.byref(f), D))


def layout(fmt, B: int, H: int, D: int, T_max: int):
    """(offsets[10], lengths[10], total bytes) of the storage image."""
    f = _fmt(fmt)
    off = np.zeros(N_SECTIONS, dtype=np.uint64)
    ln = np.zeros(N_SECTIONS, dtype=np.uint64)
    tot = np.zeros(1, dtype=np.uint64)
    st = lib().orc_layout(C.byref(f), B, H, D, T_max, _ptr(off), _ptr(ln), _ptr(tot))
    if st:
        raise OracleError(st, "layout")
    return [int(v) for v in off], [int(v) for v in ln], int(tot[0])


def num_coded(fmt, n: int) -> int:
    f = _fmt(fmt)
    return int(lib().orc_num_coded(C.byref(f), n))


class Cache:
    """The oracle's packed cache: a host byte image plus the token count."""

    def __init__(self, fmt, B: int, H: int, D: int, T_max: int):
        self.fmt = dict(fmt)
        self.B, self.H, self.D, self.T_max = B, H, D, T_max
        self._f = _fmt(fmt)
        self.offsets, self.lengths, total = layout(fmt, B, H, D, T_max)
        self.image = np.zeros(total, dtype=np.uint8)
        self.n = 0

    def append(self, K: np.ndarray, V: np.ndarray) -> None:
        """Append bf16 K, V of shape [B, n_new, H, D] (uint16 bit patterns)."""
        K = np.ascontiguousarray(K, dtype=np.uint16)
        V = np.ascontiguousarray(V, dtype=np.uint16)
        assert K.shape == V.shape and K.ndim == 4
        assert K.shape[0] == self.B and K.shape[2] == self.H and K.shape[3] == self.D
        n = C.c_int(self.n)
        st = lib().orc_append(C.byref(self._f), self.B, self.H, self.D, self.T_max, _ptr(self.image),
                              C.byref(n), _ptr(K), _ptr(V), K.shape[1])
        if st:
            raise OracleError(st, "append")
        self.n = n.value

    @property
    def n_coded(self) -> int:
        return num_coded(self.fmt, self.n)

    def dequant(self):
        """Reconstruction (Khat, Vhat), each fp64 [B, H, n, D]."""
        shape = (self.B, self.H, self.n, self.D)
        kh = np.zeros(shape, dtype=np.float64)
        vh = np.zeros(shape, dtype=np.float64)
        st = lib().orc_dequant(C.byref(self._f), self.B, self.H, self.D, self.T_max, _ptr(self.image),
                               self.n, _ptr(kh), _ptr(vh))
        if st:
            raise OracleError(st, "dequant")
        return kh, vh

    def decode_attn(self, Q: np.ndarray, sm_scale: float) -> np.ndarray:
        """Attention of bf16 Q [B, H_q, D] over the cache; fp64 [B, H_q, D]."""
        Q = np.ascontiguousarray(Q, dtype=np.uint16)
        assert Q.ndim == 3 and Q.shape[0] == self.B and Q.shape[2] == self.D
        O = np.zeros(Q.shape, dtype=np.float64)
        st = lib().orc_decode_attn(C.byref(self._f), self.B, self.H, self.D, self.T_max,
                                   _ptr(self.image), self.n, _ptr(Q), Q.shape[1], float(sm_scale),
                                   _ptr(O))
        if st:
            raise OracleError(st, "decode_attn")
        return O

    def prefill_attn(self, Q: np.ndarray, sm_scale: float) -> np.ndarray:
        """Causal attention of the last C appended tokens' bf16 queries
        Q [B, C, H_q, D] over the cache; fp64 [B, C, H_q, D]."""
        Q = np.ascontiguousarray(Q, dtype=np.uint16)
        assert Q.ndim == 4 and Q.shape[0] == self.B and Q.shape[3] == self.D
        O = np.zeros(Q.shape, dtype=np.float64)
        st = lib().orc_prefill_attn(C.byref(self._f), self.B, self.H, self.D, self.T_max,
                                    _ptr(self.image), self.n, Q.shape[1], _ptr(Q), Q.shape[2],
                                    float(sm_scale), _ptr(O))
        if st:
            raise OracleError(st, "prefill_attn")
        return O

    def section(self, i: int) -> np.ndarray:
        """Raw bytes of section i (0..7: Kc, Ks, Kz, Vc, Vs, Vz, Kr, Vr)."""
        return self.image[self.offsets[i]:self.offsets[i] + self.lengths[i]]


# ------------------------------------------------------------- projection

def project(Hm, W, A, Bm, rank: int, scale: float, d_q: int, d_kv: int):
    """Eq. (1)-(2) with explicit adapters.  Returns (Y fp64, Y bf16 bits),
    each [M, d_q + 2 d_kv] with columns Q | K | V."""
    Hm = np.ascontiguousarray(Hm, dtype=np.uint16)
    W = np.ascontiguousarray(W, dtype=np.uint16)
    M, d_in = Hm.shape
    N = d_q + 2 * d_kv
    assert W.shape == (N, d_in)
    if rank > 0:
        A = np.ascontiguousarray(A, dtype=np.uint16)
        Bm = np.ascontiguousarray(Bm, dtype=np.uint16)
        assert A.shape == (3 * rank, d_in) and Bm.shape == (N, rank)
        pa, pb = _ptr(A), _ptr(Bm)
    else:
        pa = pb = None
    Y = np.zeros((M, N), dtype=np.float64)
    Yb = np.zeros((M, N), dtype=np.uint16)
    st = lib().orc_project(_ptr(Hm), M, d_in, _ptr(W), d_q, d_kv, pa, pb, rank, float(scale),
                           _ptr(Y), _ptr(Yb))
    if st:
        raise OracleError(st, "project")
    return Y, Yb


def merge_adapter(W, A, Bm, rank: int, scale: float, d_q: int, d_kv: int):
    """Sec. 3.4 dense merge W' = W + scale * B_p A_p row by row.  Returns
    (W' fp64, W' bf16 bits), each [d_q + 2 d_kv, d_in]."""
    W = np.ascontiguousarray(W, dtype=np.uint16)
    N, d_in = W.shape
    assert N == d_q + 2 * d_kv
    if rank > 0:
        A = np.ascontiguousarray(A, dtype=np.uint16)
        Bm = np.ascontiguousarray(Bm, dtype=np.uint16)
        assert A.shape == (3 * rank, d_in) and Bm.shape == (N, rank)
        pa, pb = _ptr(A), _ptr(Bm)
    else:
        pa = pb = None
    Wd = np.zeros((N, d_in), dtype=np.float64)
    Wb = np.zeros((N, d_in), dtype=np.uint16)
    st = lib().orc_merge_adapter(_ptr(W), d_in, d_q, d_kv, pa, pb, rank, float(scale), _ptr(Wd), _ptr(Wb))
    if st:
        raise OracleError(st, "merge_adapter")
    return Wd, Wb
