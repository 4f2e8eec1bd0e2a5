"""Python binding of the MI355X hybrid weighted sum (include/fiona.h).

Argument marshalling only: every step of the computation runs in the HIP
kernels of ``libfiona.so``.  PyTorch supplies device memory and streams.  If
the library has not been built, importing works but every call raises.

    ctx  = Ctx(N, L, moduli)
    plan = Plan.from_layer(ctx, layer)          # or Plan(ctx, n_in=..., ...)
    hybrid_linear(plan, in_t, pt_t, sign_t, scale_t, out_t)

Tensors are device tensors of 8-byte elements (uint64 residues, stored in any
8-byte dtype) for in/pt/scale/out and int8 for the signs, laid out as the
header describes: in [n_in][2][L][N], pt n_pt rows of [L][N] at the plan's
pitch (default L*N), out [n_out][2][L][N].
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfiona.so")

FIONA_PLAN_NO_SHARING = 1
FIONA_PLAN_HOST_ONLY = 2
FIONA_PLAN_NO_LDS_SUMS = 4
FIONA_PLAN_NO_PARTIAL_SHARING = 8
FIONA_PLAN_PER_CONTRIBUTION = 16
FIONA_PLAN_NO_OUTPUT_BURSTS = 32
FIONA_PLAN_CHECK_INPUTS = 64

FIONA_ERR_ARG = -1
FIONA_ERR_PRECONDITION = -9
FIONA_ERR_BOUNDS = -10

STATUS = {0: "FIONA_OK", -1: "FIONA_ERR_ARG", -2: "FIONA_ERR_PLAN", -3: "FIONA_ERR_UNSUPPORTED",
          -4: "FIONA_ERR_ALIGN", -5: "FIONA_ERR_ALIAS", -6: "FIONA_ERR_HIP", -7: "FIONA_ERR_NOMEM",
          -8: "FIONA_ERR_NODEVICE", -9: "FIONA_ERR_PRECONDITION", -10: "FIONA_ERR_BOUNDS"}


class FionaError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__("%s: %s (%d)" % (where, STATUS.get(status, "unknown"), status))


class _LayerDesc(ctypes.Structure):
    _fields_ = [("n_in", ctypes.c_uint32), ("n_out", ctypes.c_uint32), ("n_pt", ctypes.c_uint32),
                ("n_scale", ctypes.c_uint32),
                ("pm_off", ctypes.c_void_p), ("pm_input", ctypes.c_void_p), ("pm_pt", ctypes.c_void_p),
                ("grp_off", ctypes.c_void_p), ("grp_mem_off", ctypes.c_void_p),
                ("mem_input", ctypes.c_void_p), ("mem_sign", ctypes.c_void_p), ("grp_scale", ctypes.c_void_p),
                ("flags", ctypes.c_uint32), ("pt_pitch", ctypes.c_uint64)]


class _Stats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_uint64) for n in (
        "ct_terms", "n_pmult", "n_member", "n_member_nonzero", "n_use", "n_sum_distinct", "n_sum_resident",
        "pmult_per_contribution", "pmult_grouped", "addsub_unshared", "addsub_shared", "addsub_partial")] + \
        [(n, ctypes.c_uint32) for n in ("tile", "waves", "lds_bytes", "grid", "split_outputs", "segment_slots",
                                        "n_partial", "partial_levels", "output_rounds",
                                        "output_buffer_rows", "input_passes")]


_lib = None


def lib():
    """The loaded HIP library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libfiona.so is not built (run __graft_entry__.build()); "
                               "there is no fallback path")
        L = ctypes.CDLL(LIB_PATH)
        L.fiona_ctx_create.restype = ctypes.c_int
        L.fiona_ctx_create.argtypes = [ctypes.c_uint32, ctypes.c_uint32, ctypes.c_void_p,
                                       ctypes.POINTER(ctypes.c_void_p)]
        L.fiona_ctx_destroy.restype = None
        L.fiona_ctx_destroy.argtypes = [ctypes.c_void_p]
        L.fiona_plan_create.restype = ctypes.c_int
        L.fiona_plan_create.argtypes = [ctypes.c_void_p, ctypes.POINTER(_LayerDesc),
                                        ctypes.POINTER(ctypes.c_void_p)]
        L.fiona_plan_destroy.restype = None
        L.fiona_plan_destroy.argtypes = [ctypes.c_void_p]
        L.fiona_plan_stats.restype = ctypes.c_int
        L.fiona_plan_stats.argtypes = [ctypes.c_void_p, ctypes.POINTER(_Stats)]
        L.fiona_hybrid_linear.restype = ctypes.c_int
        L.fiona_hybrid_linear.argtypes = [ctypes.c_void_p] * 7
        L.fiona_pt_pitch_hint.restype = ctypes.c_uint64
        L.fiona_pt_pitch_hint.argtypes = [ctypes.c_void_p]
        L.fiona_status_string.restype = ctypes.c_char_p
        L.fiona_status_string.argtypes = [ctypes.c_int]
        _lib = L
    return _lib


def _check(rc: int, where: str):
    if rc != 0:
        raise FionaError(rc, where)


class Ctx:
    """RNS parameters: N coefficients, L limbs with moduli q_l < 2^50."""

    def __init__(self, N: int, L: int, moduli):
        self.N, self.L = int(N), int(L)
        self.moduli = [int(q) for q in moduli]
        arr = (ctypes.c_uint64 * len(self.moduli))(*self.moduli)
        h = ctypes.c_void_p()
        _check(lib().fiona_ctx_create(self.N, self.L, ctypes.cast(arr, ctypes.c_void_p), ctypes.byref(h)),
               "fiona_ctx_create")
        self._h = h

    @property
    def handle(self):
        return self._h

    def pt_pitch_hint(self) -> int:
        """fiona_pt_pitch_hint: a padded plaintext pitch (words) for this context."""
        return int(lib().fiona_pt_pitch_hint(self._h))

    def close(self):
        if getattr(self, "_h", None) and self._h.value:
            lib().fiona_ctx_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _u32(a):
    return np.ascontiguousarray(a, dtype=np.uint32)


class Plan:
    """A compiled layer (fiona_plan_create)."""

    def __init__(self, ctx: Ctx, n_in, n_out, n_pt, n_scale, pm_off, pm_input, pm_pt, grp_off, grp_mem_off,
                 mem_input, mem_sign, grp_scale, flags: int = 0, pt_pitch: int = 0):
        self.ctx = ctx
        keep = [_u32(pm_off), _u32(pm_input), _u32(pm_pt), _u32(grp_off), _u32(grp_mem_off),
                _u32(mem_input), np.ascontiguousarray(mem_sign, dtype=np.int8), _u32(grp_scale)]

        def ptr(a):
            return a.ctypes.data if a.size else None

        d = _LayerDesc(int(n_in), int(n_out), int(n_pt), int(n_scale), *[ptr(a) for a in keep], int(flags),
                       int(pt_pitch))
        h = ctypes.c_void_p()
        _check(lib().fiona_plan_create(ctx.handle, ctypes.byref(d), ctypes.byref(h)), "fiona_plan_create")
        self._h = h
        self.n_in, self.n_out, self.n_pt, self.n_scale = int(n_in), int(n_out), int(n_pt), int(n_scale)
        self.n_member = int(keep[4][-1]) if keep[4].size else 0
        self.pt_pitch = int(pt_pitch) if pt_pitch else ctx.L * ctx.N

    @classmethod
    def from_layer(cls, ctx: Ctx, layer, flags: int = 0, pt_pitch: int = 0) -> "Plan":
        return cls(ctx, layer.n_in, layer.n_out, layer.n_pt, len(layer.scales), layer.pm_off, layer.pm_input,
                   layer.pm_pt, layer.grp_off, layer.grp_mem_off, layer.mem_input, layer.mem_sign,
                   layer.grp_scale, flags, pt_pitch)

    def pt_words(self) -> int:
        """Words the plaintext table spans under this plan's pitch."""
        return (self.n_pt - 1) * self.pt_pitch + self.ctx.L * self.ctx.N if self.n_pt else 0

    @property
    def handle(self):
        return self._h

    def stats(self) -> dict:
        s = _Stats()
        _check(lib().fiona_plan_stats(self._h, ctypes.byref(s)), "fiona_plan_stats")
        return {n: int(getattr(s, n)) for n, _ in _Stats._fields_}

    def close(self):
        if getattr(self, "_h", None) and self._h.value:
            lib().fiona_plan_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _dptr(t, name, elem_size):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("%s must be a device tensor" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if t.element_size() != elem_size:
        raise ValueError("%s must have %d-byte elements" % (name, elem_size))
    return t.data_ptr()


def _call_ptrs(plan: Plan, in_t, pt_t, sign_t, scale_t, out_t):
    """The device pointers of one call, after checking the tensors' sizes."""
    N, L = plan.ctx.N, plan.ctx.L
    sizes = [(in_t, "in_cts", plan.n_in * 2 * L * N), (pt_t, "pt_diags", plan.pt_words()),
             (out_t, "out_cts", plan.n_out * 2 * L * N), (sign_t, "ternary_groups", plan.n_member),
             (scale_t, "scales", plan.n_scale)]
    for t, name, n in sizes:
        if t is not None and t.numel() < n:
            raise ValueError("%s has %d elements, needs %d" % (name, t.numel(), n))
    return (_dptr(in_t, "in_cts", 8), _dptr(pt_t, "pt_diags", 8), _dptr(sign_t, "ternary_groups", 1),
            _dptr(scale_t, "scales", 8), _dptr(out_t, "out_cts", 8))


def hybrid_linear(plan: Plan, in_t, pt_t, sign_t, scale_t, out_t, stream=None) -> None:
    """fiona_hybrid_linear on torch device tensors (queued on ``stream``, default: current)."""
    _check(lib().fiona_hybrid_linear(plan.handle, *_call_ptrs(plan, in_t, pt_t, sign_t, scale_t, out_t),
                                     _stream_handle(stream)), "fiona_hybrid_linear")


class Rescaler:
    """NTT tables and workspace for the rescale epilogue (fiona_rescaler_create)."""

    def __init__(self, ctx: Ctx, max_ct: int, psi=None):
        L = lib()
        L.fiona_rescaler_create.restype = ctypes.c_int
        L.fiona_rescaler_create.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint32,
                                            ctypes.POINTER(ctypes.c_void_p)]
        L.fiona_rescaler_destroy.restype = None
        L.fiona_rescaler_destroy.argtypes = [ctypes.c_void_p]
        L.fiona_rescale.restype = ctypes.c_int
        L.fiona_rescale.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint32, ctypes.c_void_p,
                                    ctypes.c_void_p]
        self.ctx = ctx
        self.max_ct = int(max_ct)
        roots = None
        if psi is not None:
            roots = (ctypes.c_uint64 * ctx.L)(*[int(p) for p in psi])
        h = ctypes.c_void_p()
        _check(L.fiona_rescaler_create(ctx.handle, ctypes.cast(roots, ctypes.c_void_p) if roots else None,
                                       self.max_ct, ctypes.byref(h)), "fiona_rescaler_create")
        self._h = h

    @property
    def handle(self):
        return self._h

    def close(self):
        if getattr(self, "_h", None) and self._h.value:
            lib().fiona_rescaler_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def rescale(rescaler: Rescaler, in_t, n_ct: int, out_t, stream=None) -> None:
    """fiona_rescale on torch device tensors: in [n_ct][2][L][N] -> out [n_ct][2][L-1][N]."""
    import torch

    N, L = rescaler.ctx.N, rescaler.ctx.L
    if in_t.numel() < n_ct * 2 * L * N or out_t.numel() < n_ct * 2 * (L - 1) * N:
        raise ValueError("tensors too small for %d ciphertexts" % n_ct)
    if stream is None:
        stream = torch.cuda.current_stream()
    s = stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)
    _check(lib().fiona_rescale(rescaler.handle, _dptr(in_t, "in_cts", 8), int(n_ct), _dptr(out_t, "out_cts", 8), s),
           "fiona_rescale")


class Rotator:
    """NTT tables of the data moduli and the special prime, and the workspace of
    the hoisted rotations (fiona_rotator_create)."""

    def __init__(self, ctx: Ctx, special_prime: int, max_rot: int, psi=None):
        L = lib()
        L.fiona_rotator_create.restype = ctypes.c_int
        L.fiona_rotator_create.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_void_p, ctypes.c_uint32,
                                           ctypes.POINTER(ctypes.c_void_p)]
        L.fiona_rotator_destroy.restype = None
        L.fiona_rotator_destroy.argtypes = [ctypes.c_void_p]
        L.fiona_rotation_key_words.restype = ctypes.c_uint64
        L.fiona_rotation_key_words.argtypes = [ctypes.c_void_p]
        L.fiona_rotation_key_layout.restype = ctypes.c_int
        L.fiona_rotation_key_layout.argtypes = [ctypes.c_void_p, ctypes.c_uint32, ctypes.c_void_p, ctypes.c_void_p,
                                                ctypes.c_void_p]
        L.fiona_hoisted_rotate.restype = ctypes.c_int
        L.fiona_hoisted_rotate.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint32, ctypes.c_void_p,
                                           ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        self.ctx = ctx
        self.P = int(special_prime)
        self.max_rot = int(max_rot)
        roots = None
        if psi is not None:
            roots = (ctypes.c_uint64 * (ctx.L + 1))(*[int(p) for p in psi])
        h = ctypes.c_void_p()
        _check(L.fiona_rotator_create(ctx.handle, self.P, ctypes.cast(roots, ctypes.c_void_p) if roots else None,
                                      self.max_rot, ctypes.byref(h)), "fiona_rotator_create")
        self._h = h

    @property
    def handle(self):
        return self._h

    def key_words(self) -> int:
        """Words of one rotation key: L * 2 * (L + 1) * N."""
        return int(lib().fiona_rotation_key_words(self._h))

    def close(self):
        if getattr(self, "_h", None) and self._h.value:
            lib().fiona_rotator_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _stream_handle(stream):
    import torch

    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def rotation_key_layout(rotator: Rotator, galois: int, key_t, out_t, stream=None) -> None:
    """fiona_rotation_key_layout: a key [L][2][L+1][N] in natural NTT order -> the library's layout."""
    n = rotator.key_words()
    if key_t.numel() < n or out_t.numel() < n:
        raise ValueError("key tensors need %d words" % n)
    _check(lib().fiona_rotation_key_layout(rotator.handle, int(galois), _dptr(key_t, "key", 8),
                                           _dptr(out_t, "key_out", 8), _stream_handle(stream)),
           "fiona_rotation_key_layout")


def hoisted_rotate(rotator: Rotator, ct_t, galois, keys_t, out_t, stream=None) -> None:
    """fiona_hoisted_rotate: ct [2][L][N] -> out [len(galois)][2][L][N], keys [len(galois)] in the library layout."""
    N, L = rotator.ctx.N, rotator.ctx.L
    n_rot = len(galois)
    if ct_t.numel() < 2 * L * N or out_t.numel() < n_rot * 2 * L * N or keys_t.numel() < n_rot * rotator.key_words():
        raise ValueError("tensors too small for %d rotations" % n_rot)
    g = (ctypes.c_uint32 * max(1, n_rot))(*[int(x) for x in galois])
    _check(lib().fiona_hoisted_rotate(rotator.handle, _dptr(ct_t, "ct", 8), n_rot, ctypes.cast(g, ctypes.c_void_p),
                                      _dptr(keys_t, "keys", 8), _dptr(out_t, "out_cts", 8), _stream_handle(stream)),
           "fiona_hoisted_rotate")


def mac_microbench(blocks: int, chunks: int, sink_t, stream=None) -> int:
    """fiona_mac_microbench: the register-only raw-route arithmetic over
    blocks * 256 threads; returns the plaintext words it multiplies."""
    L = lib()
    L.fiona_mac_microbench.restype = ctypes.c_int
    L.fiona_mac_microbench.argtypes = [ctypes.c_uint32, ctypes.c_uint32, ctypes.c_void_p, ctypes.c_void_p]
    L.fiona_mac_microbench_words.restype = ctypes.c_uint64
    L.fiona_mac_microbench_words.argtypes = [ctypes.c_uint32, ctypes.c_uint32]
    if sink_t.numel() < blocks * 256:
        raise ValueError("sink holds fewer than blocks * 256 words")
    _check(L.fiona_mac_microbench(int(blocks), int(chunks), _dptr(sink_t, "sink", 8), _stream_handle(stream)),
           "fiona_mac_microbench")
    return int(L.fiona_mac_microbench_words(int(blocks), int(chunks)))


def check_ntt_offsets(op: str, N: int, L: int, moduli, capacity: int, n_call: int, out_shrink: int = 0):
    """fiona_check_ntt_offsets: host replay of every memory access of one
    rescale (op "rescale", L moduli) or one rotation call (op "rotate", L data
    moduli then the special prime).  Returns (status, first violation or "")."""
    L_ = lib()
    L_.fiona_check_ntt_offsets.restype = ctypes.c_int
    L_.fiona_check_ntt_offsets.argtypes = [ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_void_p,
                                           ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_char_p,
                                           ctypes.c_size_t]
    mods = (ctypes.c_uint64 * len(moduli))(*[int(q) for q in moduli])
    msg = ctypes.create_string_buffer(512)
    rc = L_.fiona_check_ntt_offsets({"rescale": 0, "rotate": 1}[op], int(N), int(L), ctypes.cast(mods, ctypes.c_void_p),
                                    int(capacity), int(n_call), int(out_shrink), msg, 512)
    return rc, msg.value.decode()


def stream_read(src_t, blocks: int, sink_t, stream=None) -> int:
    """fiona_stream_read over all of src_t (8-byte elements, an even count);
    returns the bytes read."""
    L_ = lib()
    L_.fiona_stream_read.restype = ctypes.c_int
    L_.fiona_stream_read.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint32, ctypes.c_void_p,
                                     ctypes.c_void_p]
    if sink_t.numel() < blocks:
        raise ValueError("sink holds fewer than blocks words")
    _check(L_.fiona_stream_read(_dptr(src_t, "src", 8), src_t.numel(), int(blocks), _dptr(sink_t, "sink", 8),
                                _stream_handle(stream)), "fiona_stream_read")
    return src_t.numel() * 8


def stream_copy(src_t, dst_t, blocks: int, stream=None) -> int:
    """fiona_stream_copy of all of src_t into dst_t; returns the bytes moved (read + written)."""
    L_ = lib()
    L_.fiona_stream_copy.restype = ctypes.c_int
    L_.fiona_stream_copy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint32,
                                     ctypes.c_void_p]
    if dst_t.numel() < src_t.numel():
        raise ValueError("dst is smaller than src")
    _check(L_.fiona_stream_copy(_dptr(src_t, "src", 8), _dptr(dst_t, "dst", 8), src_t.numel(), int(blocks),
                                _stream_handle(stream)), "fiona_stream_copy")
    return 2 * src_t.numel() * 8


def stream_write(dst_t, blocks: int, stream=None) -> int:
    """fiona_stream_write over all of dst_t (8-byte elements, an even count);
    returns the bytes written."""
    L_ = lib()
    L_.fiona_stream_write.restype = ctypes.c_int
    L_.fiona_stream_write.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint32, ctypes.c_void_p]
    _check(L_.fiona_stream_write(_dptr(dst_t, "dst", 8), dst_t.numel(), int(blocks), _stream_handle(stream)),
           "fiona_stream_write")
    return dst_t.numel() * 8


def plan_check_inputs(plan: Plan, signs, scales, x=None, pt=None) -> int:
    """fiona_plan_check_inputs on host arrays (NumPy): signs int8 [n_member],
    scales uint64 [n_scale], x uint64 [n_in][2][L][N] or None, pt uint64 rows at
    the plan's pitch or None.  Returns the status (0, FIONA_ERR_PRECONDITION, ...)."""
    L_ = lib()
    L_.fiona_plan_check_inputs.restype = ctypes.c_int
    L_.fiona_plan_check_inputs.argtypes = [ctypes.c_void_p] * 5
    keep = [np.ascontiguousarray(signs, dtype=np.int8), np.ascontiguousarray(scales, dtype=np.uint64)]
    keep += [None if a is None else np.ascontiguousarray(a, dtype=np.uint64) for a in (x, pt)]
    ptrs = [None if a is None or not a.size else a.ctypes.data for a in keep]
    return int(L_.fiona_plan_check_inputs(plan.handle, *ptrs))


def hybrid_linear_static(plan: Plan, in_t, pt_t, sign_t, scale_t, out_t, stream=None) -> None:
    """fiona_hybrid_linear_static: hybrid_linear with its word blocks in the
    library's static per-device array (allocates nothing)."""
    L_ = lib()
    L_.fiona_hybrid_linear_static.restype = ctypes.c_int
    L_.fiona_hybrid_linear_static.argtypes = [ctypes.c_void_p] * 7
    _check(L_.fiona_hybrid_linear_static(plan.handle, *_call_ptrs(plan, in_t, pt_t, sign_t, scale_t, out_t),
                                         _stream_handle(stream)), "fiona_hybrid_linear_static")
