"""Oracle for the hybrid weighted sum -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The GPU library never does; the two
share no code.  The arithmetic lives in ``fiona_oracle.c`` (plain C, built with
gcc); this module only marshals NumPy arrays to it.

Functions follow the paper as cited in ``fiona_oracle.c``:
``weighted_sum`` is the per-contribution form of Sec. 4.2, Eq. (routed-example);
the NTT helpers exist to pin the meaning of the element-wise product (PMult,
Sec. 2.2) as multiplication in Z_q[X]/(X^N + 1).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "fiona_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

_u32p = ctypes.POINTER(ctypes.c_uint32)
_u64p = ctypes.POINTER(ctypes.c_uint64)
_i8p = ctypes.POINTER(ctypes.c_int8)


def build() -> str:
    """Compile the oracle with gcc (always; a few seconds)."""
    tmp = _LIB + ".tmp%d" % os.getpid()
    subprocess.run(["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-fPIC", "-shared", "-pthread",
                    _SRC, "-o", tmp], check=True)
    os.replace(tmp, _LIB)
    return _LIB


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        L = ctypes.CDLL(_LIB)
        L.oracle_weighted_sum.restype = ctypes.c_int
        L.oracle_weighted_sum.argtypes = [
            ctypes.c_uint32, _u64p, ctypes.c_uint32, _u64p, _u64p, ctypes.c_uint32,
            _u32p, _u32p, _u32p, _u32p, _u32p, _u32p, _i8p, _u32p, _u64p, _u64p, ctypes.c_int]
        L.oracle_find_psi.restype = ctypes.c_uint64
        L.oracle_find_psi.argtypes = [ctypes.c_uint32, ctypes.c_uint64]
        for name in ("oracle_ntt_naive", "oracle_intt_naive"):
            getattr(L, name).restype = None
            getattr(L, name).argtypes = [_u64p, _u64p, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_uint64]
        for name in ("oracle_ntt_fast", "oracle_intt_fast"):
            getattr(L, name).restype = ctypes.c_int
            getattr(L, name).argtypes = [_u64p, _u64p, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_uint64]
        L.oracle_mul_acc.restype = None
        L.oracle_mul_acc.argtypes = [_u64p, _u64p, _u64p, ctypes.c_uint32, ctypes.c_uint64]
        L.oracle_negacyclic_mul.restype = None
        L.oracle_negacyclic_mul.argtypes = [_u64p, _u64p, _u64p, ctypes.c_uint32, ctypes.c_uint64]
        _lib = L
    return _lib


def _p(a, t):
    return a.ctypes.data_as(t)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def weighted_sum(q_pos, x, pt, pm_off, pm_input, pm_pt, grp_off, grp_mem_off, mem_input, mem_sign,
                 grp_scale, scales, n_threads: int = 1) -> np.ndarray:
    """Per-contribution hybrid weighted sum over flat positions.

    q_pos: uint64 [S] modulus of each position; x: uint64 [n_in][2][S];
    pt: uint64 [n_pt][S]; returns uint64 [n_out][2][S].
    """
    q_pos = _c(q_pos, np.uint64)
    S = q_pos.shape[0]
    x = _c(x, np.uint64).reshape(-1, 2, S)
    pt = _c(pt, np.uint64).reshape(-1, S) if np.size(pt) else np.zeros((0, S), np.uint64)
    pm_off, pm_input, pm_pt = (_c(a, np.uint32) for a in (pm_off, pm_input, pm_pt))
    grp_off, grp_mem_off, mem_input, grp_scale = (_c(a, np.uint32) for a in (grp_off, grp_mem_off, mem_input, grp_scale))
    mem_sign = _c(mem_sign, np.int8)
    scales = _c(scales, np.uint64)
    n_out = pm_off.shape[0] - 1
    if grp_off.shape[0] != n_out + 1:
        raise ValueError("pm_off and grp_off disagree on the number of outputs")
    if pm_input.size and int(pm_input.max()) >= x.shape[0]:
        raise ValueError("raw term input out of range")
    if mem_input.size and int(mem_input.max()) >= x.shape[0]:
        raise ValueError("member input out of range")
    if pm_pt.size and int(pm_pt.max()) >= pt.shape[0]:
        raise ValueError("plaintext index out of range")
    out = np.zeros((n_out, 2, S), dtype=np.uint64)
    # ctypes needs non-null pointers even for empty arrays
    keep = []

    def nz(a, dtype):
        if a.size == 0:
            a = np.zeros(1, dtype=dtype)
        keep.append(a)
        return a

    rc = lib().oracle_weighted_sum(
        S, _p(q_pos, _u64p), x.shape[0], _p(nz(x, np.uint64), _u64p), _p(nz(pt, np.uint64), _u64p), n_out,
        _p(pm_off, _u32p), _p(nz(pm_input, np.uint32), _u32p), _p(nz(pm_pt, np.uint32), _u32p),
        _p(grp_off, _u32p), _p(nz(grp_mem_off, np.uint32), _u32p), _p(nz(mem_input, np.uint32), _u32p),
        _p(nz(mem_sign, np.int8), _i8p), _p(nz(grp_scale, np.uint32), _u32p), _p(nz(scales, np.uint64), _u64p),
        _p(out, _u64p), int(n_threads))
    if rc != 0:
        raise RuntimeError("oracle_weighted_sum failed")
    return out


def weighted_sum_layer(layer, x_full, pt_full, n_threads: int = 1) -> np.ndarray:
    """Whole-layer form: x_full [n_in][2][L][N], pt_full [n_pt][L][N] -> [n_out][2][L][N]."""
    L, N = layer.L, layer.N
    q_pos = np.repeat(np.asarray(layer.moduli, dtype=np.uint64), N)
    out = weighted_sum(q_pos, np.asarray(x_full).reshape(layer.n_in, 2, L * N),
                       np.asarray(pt_full).reshape(-1, L * N), layer.pm_off, layer.pm_input, layer.pm_pt,
                       layer.grp_off, layer.grp_mem_off, layer.mem_input, layer.mem_sign, layer.grp_scale,
                       layer.scales, n_threads)
    return out.reshape(layer.n_out, 2, L, N)


def weighted_sum_sampled(layer, limbs, coeffs, x_s, pt_s, n_threads: int = 1) -> np.ndarray:
    """Sampled-position form: x_s [n_in][2][S], pt_s [n_pt][S] -> [n_out][2][S]."""
    q_pos = np.asarray(layer.moduli, dtype=np.uint64)[np.asarray(limbs)]
    return weighted_sum(q_pos, x_s, pt_s, layer.pm_off, layer.pm_input, layer.pm_pt, layer.grp_off,
                        layer.grp_mem_off, layer.mem_input, layer.mem_sign, layer.grp_scale, layer.scales,
                        n_threads)


def find_psi(N: int, q: int) -> int:
    return int(lib().oracle_find_psi(N, q))


def _transform(fn, a, N, q, psi):
    a = _c(a, np.uint64)
    out = np.zeros(N, dtype=np.uint64)
    rc = getattr(lib(), fn)(_p(a, _u64p), _p(out, _u64p), N, q, psi)
    if rc not in (None, 0):
        raise ValueError(fn + " failed")
    return out


def ntt_naive(a, q, psi):
    return _transform("oracle_ntt_naive", a, len(a), q, psi)


def intt_naive(a, q, psi):
    return _transform("oracle_intt_naive", a, len(a), q, psi)


def ntt(a, q, psi):
    return _transform("oracle_ntt_fast", a, len(a), q, psi)


def intt(a, q, psi):
    return _transform("oracle_intt_fast", a, len(a), q, psi)


def negacyclic_mul(a, b, q):
    a, b = _c(a, np.uint64), _c(b, np.uint64)
    c = np.zeros(len(a), dtype=np.uint64)
    lib().oracle_negacyclic_mul(_p(a, _u64p), _p(b, _u64p), _p(c, _u64p), len(a), q)
    return c


def mul_acc(acc, a, b, q):
    """acc + a * b (mod q), element-wise; acc is updated in place and returned."""
    a, b = _c(a, np.uint64), _c(b, np.uint64)
    assert acc.dtype == np.uint64 and acc.flags.c_contiguous and len(acc) == len(a) == len(b)
    lib().oracle_mul_acc(_p(acc, _u64p), _p(a, _u64p), _p(b, _u64p), len(a), q)
    return acc
