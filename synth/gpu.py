"""Device-side fill of the synthetic inputs (HIP), same values as synth's NumPy generator."""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

from . import TAG_CT, TAG_IN, TAG_PT, Layer

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "csrc", "synth_fill.hip")
LIB_PATH = os.path.join(_HERE, "libfiona_synth.so")
_lib = None


def build() -> str:
    tmp = LIB_PATH + ".tmp%d" % os.getpid()
    cmd = [os.environ.get("HIPCC", "/opt/rocm/bin/hipcc"), "--offload-arch=gfx950", "-O3", "-std=c++17",
           "-fPIC", "-shared", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", _SRC, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + r.stderr)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libfiona_synth.so is not built (run __graft_entry__.build())")
        L = ctypes.CDLL(LIB_PATH)
        L.synth_fill_uniform.restype = ctypes.c_int
        L.synth_fill_uniform.argtypes = [ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint32,
                                         ctypes.c_uint64, ctypes.c_uint64, ctypes.c_void_p, ctypes.c_void_p]
        L.synth_fill_pts.restype = ctypes.c_int
        L.synth_fill_pts.argtypes = [ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint32,
                                     ctypes.c_uint64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint64,
                                     ctypes.c_uint64, ctypes.c_void_p, ctypes.c_void_p]
        _lib = L
    return _lib


def _moduli(layer: Layer):
    return (ctypes.c_uint64 * len(layer.moduli))(*[int(q) for q in layer.moduli])


def _stream():
    import torch
    return torch.cuda.current_stream().cuda_stream


def fill_inputs(layer: Layer, t) -> None:
    """t: device tensor of >= n_in*2*L*N 8-byte elements -> input ciphertexts [n_in][2][L][N]."""
    n = layer.n_in * 2 * layer.L * layer.N
    assert t.is_cuda and t.is_contiguous() and t.element_size() == 8 and t.numel() >= n
    m = _moduli(layer)
    rc = lib().synth_fill_uniform(t.data_ptr(), layer.n_in * 2 * layer.L, layer.L, layer.N, layer.seed, TAG_IN,
                                  ctypes.cast(m, ctypes.c_void_p), _stream())
    if rc != 0:
        raise RuntimeError("synth_fill_uniform failed (%d)" % rc)


def fill_cts(layer: Layer, t, n_ct: int) -> None:
    """t: device tensor of >= n_ct*2*L*N 8-byte elements -> n_ct ciphertexts [n_ct][2][L][N]
    of uniform residues (generator tag TAG_CT)."""
    n = n_ct * 2 * layer.L * layer.N
    assert t.is_cuda and t.is_contiguous() and t.element_size() == 8 and t.numel() >= n
    m = _moduli(layer)
    rc = lib().synth_fill_uniform(t.data_ptr(), n_ct * 2 * layer.L, layer.L, layer.N, layer.seed, TAG_CT,
                                  ctypes.cast(m, ctypes.c_void_p), _stream())
    if rc != 0:
        raise RuntimeError("synth_fill_uniform failed (%d)" % rc)


def fill_rows(t, n_rows: int, moduli, N: int, seed: int, tag: int) -> None:
    """t: device tensor of >= n_rows*N 8-byte elements -> rows of N uniform residues,
    row r modulo moduli[r % len(moduli)], value at flat index r*N + k as in
    synth.uniform_mod_np(seed, tag, r*N + k, q)."""
    assert t.is_cuda and t.is_contiguous() and t.element_size() == 8 and t.numel() >= n_rows * N
    m = (ctypes.c_uint64 * len(moduli))(*[int(q) for q in moduli])
    rc = lib().synth_fill_uniform(t.data_ptr(), n_rows, len(moduli), N, seed, tag, ctypes.cast(m, ctypes.c_void_p),
                                  _stream())
    if rc != 0:
        raise RuntimeError("synth_fill_uniform failed (%d)" % rc)


def fill_pts(layer: Layer, t, pitch: int = 0) -> None:
    """t: device tensor -> this layer's plaintext table, plaintext p at word p * pitch
    (pitch 0 = L*N, packed rows); t needs (n_pt-1)*pitch + L*N 8-byte elements."""
    import torch
    pitch = int(pitch) if pitch else layer.L * layer.N
    assert pitch >= layer.L * layer.N
    n = (layer.n_pt - 1) * pitch + layer.L * layer.N if layer.n_pt else 0
    assert t.is_cuda and t.is_contiguous() and t.element_size() == 8 and t.numel() >= n
    if layer.n_pt == 0:
        return
    glob = torch.from_numpy(np.ascontiguousarray(layer.pt_global.astype(np.int64))).to(t.device)
    const = None
    if layer.pt_const is not None:
        const = torch.from_numpy(np.ascontiguousarray(layer.pt_const.astype(np.int64))).to(t.device)
    m = _moduli(layer)
    rc = lib().synth_fill_pts(t.data_ptr(), layer.n_pt, layer.L, layer.N, pitch, glob.data_ptr(),
                              const.data_ptr() if const is not None else None, layer.seed, TAG_PT,
                              ctypes.cast(m, ctypes.c_void_p), _stream())
    if rc != 0:
        raise RuntimeError("synth_fill_pts failed (%d)" % rc)
    torch.cuda.current_stream().synchronize()   # glob/const are freed on return
