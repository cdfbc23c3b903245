"""Python binding of libvcattn.so, the MI355X (gfx950) 8-bit VC-Attention forward.

Argument marshalling only: every step of the attention path runs in the library's HIP kernels.
torch is used for device memory and the current stream. The names mirror the C ABI declared in
include/vc_attn.h (vc_attn_group, vc_attn_prep, vc_attn_forward, ...). There is no fallback: if
the shared library is missing, importing the entry points raises.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libvcattn.so")
D = 128

VC_OK = 0
STATUS = {0: "VC_OK", 1: "VC_ERR_NULL", 2: "VC_ERR_SHAPE", 3: "VC_ERR_UNSUPPORTED", 4: "VC_ERR_WORKSPACE",
          5: "VC_ERR_ALIGN", 6: "VC_ERR_HIP", 7: "VC_ERR_INTERNAL"}
P_EXPCAST, P_EXP_THEN_CAST = 0, 1
QK_INT8, QK_FP8, QK_MXFP4 = 0, 1, 2
GROUP_IDENTITY, GROUP_CUBE, GROUP_KMEANS = 0, 1, 2


class VcError(RuntimeError):
    def __init__(self, fn: str, status: int, lib=None):
        msg = f"{fn} returned {STATUS.get(status, status)}"
        if lib is not None:
            msg += f" ({lib.vc_status_str(status).decode()})"
            if status == 6:
                msg += f", hipError {lib.vc_last_hip_error()}"
        super().__init__(msg)
        self.status = status


class Shape(C.Structure):
    _fields_ = [(n, C.c_int32) for n in ("B", "H", "N", "d", "F", "Ht", "Wd")]


class Opts(C.Structure):
    _fields_ = [("qk_fmt", C.c_int32), ("p_mode", C.c_int32), ("rope", C.c_int32), ("hadamard", C.c_int32),
                ("smooth_k", C.c_int32), ("smooth_v", C.c_int32), ("sm_scale", C.c_float), ("beta", C.c_float)]


class GroupOpts(C.Structure):
    _fields_ = [("mode", C.c_int32), ("k", C.c_int32), ("iters", C.c_int32), ("warm_start", C.c_int32),
                ("cube", C.c_int32 * 3)]


class Prepped(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("q", "q_scale", "k", "k_scale", "k_mean", "v", "v_scale", "v_mean",
                                          "q_mx_scale", "k_mx_scale")]


_lib = None


def lib():
    """The loaded shared library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with paper_2609_15810_amd/build.py "
                               "(the HIP library is required; there is no fallback)")
        L = C.CDLL(LIB_PATH)
        L.vc_attn_workspace_size.restype = C.c_size_t
        L.vc_attn_workspace_size.argtypes = [C.POINTER(Shape), C.POINTER(Opts), C.POINTER(GroupOpts)]
        L.vc_status_str.restype = C.c_char_p
        L.vc_status_str.argtypes = [C.c_int]
        L.vc_last_hip_error.restype = C.c_int
        L.vc_rope_tables.restype = C.c_int
        L.vc_rope_tables.argtypes = [C.c_int32, C.c_int32, C.c_int32, C.c_double, C.c_void_p, C.c_void_p]
        L.vc_attn_group.restype = C.c_int
        L.vc_attn_group.argtypes = [C.POINTER(Shape), C.POINTER(GroupOpts), C.c_void_p, C.c_void_p, C.c_void_p,
                                    C.c_void_p, C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]
        L.vc_attn_prep.restype = C.c_int
        L.vc_attn_prep.argtypes = [C.POINTER(Shape), C.POINTER(Opts), C.c_void_p, C.c_void_p, C.c_void_p,
                                   C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.POINTER(Prepped),
                                   C.c_void_p, C.c_size_t, C.c_void_p]
        L.vc_attn_prep_noalloc.restype = C.c_int
        L.vc_attn_prep_noalloc.argtypes = [C.POINTER(Shape), C.POINTER(Opts), C.c_void_p, C.c_void_p, C.c_void_p,
                                           C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.POINTER(Prepped),
                                           C.c_void_p]
        L.vc_attn_forward.restype = C.c_int
        L.vc_attn_forward.argtypes = [C.POINTER(Shape), C.POINTER(Opts), C.POINTER(Prepped), C.c_void_p,
                                      C.c_void_p, C.c_void_p]
        L.vc_attn_forward_codes.restype = C.c_int
        L.vc_attn_forward_codes.argtypes = [C.POINTER(Shape), C.POINTER(Opts), C.POINTER(Prepped), C.c_void_p,
                                            C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]
        L.vc_fp8_score_product.restype = C.c_int
        L.vc_fp8_score_product.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_int32, C.c_void_p]
        L.vc_opts_default.argtypes = [C.POINTER(Opts)]
        L.vc_group_opts_default.argtypes = [C.POINTER(GroupOpts)]
        _lib = L
    return _lib


def _check(fn: str, st: int):
    if st != VC_OK:
        raise VcError(fn, st, lib())


def make_shape(B: int, H: int, grid) -> Shape:
    F, Ht, Wd = grid
    return Shape(B, H, F * Ht * Wd, D, F, Ht, Wd)


def make_opts(p_mode=P_EXPCAST, rope=True, hadamard=True, smooth_k=True, smooth_v=True, sm_scale=0.0,
              beta=-0.35, qk_fmt=QK_INT8) -> Opts:
    o = Opts()
    lib().vc_opts_default(C.byref(o))
    o.qk_fmt = int(qk_fmt)
    o.p_mode, o.rope, o.hadamard = int(p_mode), int(rope), int(hadamard)
    o.smooth_k, o.smooth_v, o.sm_scale, o.beta = int(smooth_k), int(smooth_v), float(sm_scale), float(beta)
    return o


def make_group_opts(mode=GROUP_KMEANS, k=32, iters=8, warm_start=False, cube=(4, 2, 16)) -> GroupOpts:
    g = GroupOpts()
    lib().vc_group_opts_default(C.byref(g))
    g.mode, g.k, g.iters, g.warm_start = int(mode), int(k), int(iters), int(bool(warm_start))
    g.cube[0], g.cube[1], g.cube[2] = (int(c) for c in cube)
    return g


def workspace_size(shape: Shape, opts: Opts | None = None, gopts: GroupOpts | None = None) -> int:
    return int(lib().vc_attn_workspace_size(C.byref(shape), C.byref(opts) if opts is not None else None,
                                            C.byref(gopts) if gopts is not None else None))


def rope_tables_host(F: int, Ht: int, Wd: int, theta: float = 10000.0):
    """vc_rope_tables into host numpy arrays [(F+Ht+Wd), 64] fp32."""
    cos_t = np.empty((F + Ht + Wd, 64), np.float32)
    sin_t = np.empty_like(cos_t)
    _check("vc_rope_tables", lib().vc_rope_tables(F, Ht, Wd, float(theta), cos_t.ctypes.data, sin_t.ctypes.data))
    return cos_t, sin_t


def _ptr(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return C.c_void_p(s.cuda_stream)


@dataclass
class PreppedBuffers:
    """Device buffers of the low-bit operands (layouts documented in include/vc_attn.h)."""
    q: object
    q_scale: object
    k: object
    k_scale: object
    k_mean: object
    v: object
    v_scale: object
    v_mean: object
    q_mx_scale: object = None
    k_mx_scale: object = None

    def as_struct(self) -> Prepped:
        return Prepped(*(None if t is None else t.data_ptr()
                         for t in (self.q, self.q_scale, self.k, self.k_scale, self.k_mean, self.v, self.v_scale,
                                   self.v_mean, self.q_mx_scale, self.k_mx_scale)))


def alloc_prepped(shape: Shape, device="cuda", qk_fmt: int = None) -> PreppedBuffers:
    """Buffers for vc_attn_prep / vc_attn_forward. INT8 and FP8: q, k [B, H, Np, 128] bytes and fp32
    block scales; MXFP4: q, k packed codes [B, H, Np, 64] bytes and E8M0 scale bytes [B, H, Np, 4]."""
    import torch
    B, H, N = shape.B, shape.H, shape.N
    T = (N + 127) // 128
    Np = 128 * T
    e = dict(device=device)
    mx = qk_fmt == QK_MXFP4
    cw = D // 2 if mx else D
    return PreppedBuffers(
        q=torch.empty((B, H, Np, cw), dtype=torch.int8, **e), q_scale=torch.empty((B, H, T), dtype=torch.float32, **e),
        k=torch.empty((B, H, Np, cw), dtype=torch.int8, **e), k_scale=torch.empty((B, H, T), dtype=torch.float32, **e),
        k_mean=torch.empty((B, H, D), dtype=torch.float32, **e),
        v=torch.empty((B, H, Np, D), dtype=torch.uint8, **e), v_scale=torch.empty((B, H, D), dtype=torch.float32, **e),
        v_mean=torch.empty((B, H, T, D), dtype=torch.int16, **e),
        q_mx_scale=torch.empty((B, H, Np, 4), dtype=torch.uint8, **e) if mx else None,
        k_mx_scale=torch.empty((B, H, Np, 4), dtype=torch.uint8, **e) if mx else None)


def vc_attn_group(shape, gopts, V, centroids, labels, perm, inv_perm, ws, stream=None):
    _check("vc_attn_group", lib().vc_attn_group(C.byref(shape), C.byref(gopts), _ptr(V), _ptr(centroids),
                                                _ptr(labels), _ptr(perm), _ptr(inv_perm), _ptr(ws),
                                                ws.numel() * ws.element_size() if ws is not None else 0,
                                                _stream(stream)))


def vc_attn_prep(shape, opts, Q, K, V, perm, q_perm, rope_cos, rope_sin, out: PreppedBuffers, ws, stream=None):
    st = out.as_struct()
    _check("vc_attn_prep", lib().vc_attn_prep(C.byref(shape), C.byref(opts), _ptr(Q), _ptr(K), _ptr(V), _ptr(perm),
                                              _ptr(q_perm), _ptr(rope_cos), _ptr(rope_sin), C.byref(st), _ptr(ws),
                                              ws.numel() * ws.element_size(), _stream(stream)))


def vc_attn_prep_noalloc(shape, opts, Q, K, V, perm, q_perm, rope_cos, rope_sin, out: PreppedBuffers, stream=None):
    st = out.as_struct()
    _check("vc_attn_prep_noalloc", lib().vc_attn_prep_noalloc(C.byref(shape), C.byref(opts), _ptr(Q), _ptr(K), _ptr(V),
                                                              _ptr(perm), _ptr(q_perm), _ptr(rope_cos), _ptr(rope_sin),
                                                              C.byref(st), _stream(stream)))


def vc_attn_forward(shape, opts, inp: PreppedBuffers, q_perm, O, stream=None):
    st = inp.as_struct()
    _check("vc_attn_forward", lib().vc_attn_forward(C.byref(shape), C.byref(opts), C.byref(st), _ptr(q_perm),
                                                    _ptr(O), _stream(stream)))


def vc_attn_forward_codes(shape, opts, inp: PreppedBuffers, q_perm, O, p_codes, stream=None):
    st = inp.as_struct()
    nbytes = p_codes.numel() * p_codes.element_size() if p_codes is not None else 0
    _check("vc_attn_forward_codes", lib().vc_attn_forward_codes(C.byref(shape), C.byref(opts), C.byref(st),
                                                                _ptr(q_perm), _ptr(O), _ptr(p_codes), nbytes,
                                                                _stream(stream)))


def vc_fp8_score_product(a, b, c_in, out, stream=None):
    """a, b: uint8 E4M3 bytes [n, 32, 128]; c_in, out: fp32 [n, 32, 32] (device tensors)."""
    n = a.shape[0]
    _check("vc_fp8_score_product", lib().vc_fp8_score_product(_ptr(a), _ptr(b), _ptr(c_in), _ptr(out), n,
                                                              _stream(stream)))


class Attention:
    """Buffers for one attention shape and the three calls of the path.

    group() computes the permutation (and centroids) from V; prep() produces the low-bit
    operands; forward() writes O. Inputs are bf16 tensors [B, H, N, 128] on the device
    (torch.bfloat16 or int16 bit patterns).
    """

    def __init__(self, B, H, grid, opts: Opts | None = None, gopts: GroupOpts | None = None, device="cuda"):
        import torch
        self.shape = make_shape(B, H, grid)
        self.opts = opts if opts is not None else make_opts()
        self.gopts = gopts if gopts is not None else make_group_opts()
        self.device = device
        ws = workspace_size(self.shape, self.opts, self.gopts)
        if ws == 0:
            raise VcError("vc_attn_workspace_size", 2)
        self.ws = torch.empty(ws, dtype=torch.uint8, device=device)
        N = self.shape.N
        e = dict(device=device, dtype=torch.int32)
        self.perm = torch.empty((B, H, N), **e)
        self.inv_perm = torch.empty((B, H, N), **e)
        self.labels = torch.empty((B, H, N), **e)
        self.centroids = torch.zeros((B, H, max(self.gopts.k, 1), D), dtype=torch.float32, device=device)
        self.prepped = alloc_prepped(self.shape, device, self.opts.qk_fmt)
        cos_t, sin_t = rope_tables_host(*grid)
        self.rope_cos = torch.from_numpy(cos_t).to(device)
        self.rope_sin = torch.from_numpy(sin_t).to(device)

    def group(self, V, warm_start=None, stream=None):
        g = self.gopts
        if warm_start is not None:
            g = make_group_opts(g.mode, g.k, g.iters, warm_start, tuple(g.cube))
        vc_attn_group(self.shape, g, V, self.centroids, self.labels, self.perm, self.inv_perm, self.ws, stream)

    def prep(self, Q, K, V, perm="own", q_perm=None, stream=None):
        p = self.perm if isinstance(perm, str) else perm
        vc_attn_prep(self.shape, self.opts, Q, K, V, p, q_perm, self.rope_cos, self.rope_sin, self.prepped, self.ws,
                     stream)

    def forward(self, O, q_perm=None, stream=None):
        vc_attn_forward(self.shape, self.opts, self.prepped, q_perm, O, stream)

    def forward_codes(self, O, p_codes, q_perm=None, stream=None):
        """forward() that also writes the probability codes, uint8 [B, H, N, 128 T] (debugging)."""
        vc_attn_forward_codes(self.shape, self.opts, self.prepped, q_perm, O, p_codes, stream)
