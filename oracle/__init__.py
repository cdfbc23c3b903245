"""CPU oracle for the 8-bit VC-Attention forward -- test infrastructure.

This package is the independent reference the GPU library is checked against. Only the tests,
the smoke check and the benchmark's CPU-baseline leg may import it; the product path never does.
It shares no code with the HIP library: the arithmetic lives in ``vc_oracle.c`` (plain scalar C,
built with ``-ffp-contract=off``), and this module only marshals numpy arrays into it.

Conventions: bf16 tensors are passed as ``uint16`` bit patterns; E4M3 bytes as ``uint8``.
Shapes follow the method's statement of the problem (Sec. 3.1): per (batch, head) a sequence of
N tokens of head dimension d = 128, tokens flattened from a (frames x rows x cols) latent grid.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
import threading

import numpy as np

D = 128
BLK = 128
_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "vc_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None

P_EXPCAST = 0
P_EXP_THEN_CAST = 1
GROUP_IDENTITY = 0
GROUP_CUBE = 1
GROUP_KMEANS = 2


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (one IEEE rounding per written fp32 operation)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
               "-fPIC", "-shared", _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


QK_INT8, QK_FP8, QK_MXFP4 = 0, 1, 2


class PrepCfg(C.Structure):
    _fields_ = [(n, C.c_int32) for n in ("N", "F", "Ht", "Wd", "rope", "hadamard", "smooth_k", "smooth_v",
                                         "qk_fmt")]


class AttnCfg(C.Structure):
    _fields_ = [("N", C.c_int32), ("hadamard", C.c_int32), ("smooth_v", C.c_int32), ("p_mode", C.c_int32),
                ("sm_scale", C.c_float), ("beta", C.c_float), ("qk_fmt", C.c_int32)]


class GroupCfg(C.Structure):
    _fields_ = [(n, C.c_int32) for n in ("N", "F", "Ht", "Wd", "mode", "k", "iters", "warm_start",
                                         "cube_t", "cube_h", "cube_w")]


def lib():
    global _lib
    with _lock:
        if _lib is None:
            build()
            _lib = C.CDLL(_LIB)
            _lib.or_expcast_code_u.restype = C.c_int
            _lib.or_expcast_code_acc.restype = C.c_int
            _lib.or_exp_then_cast_code_acc.restype = C.c_int
            _lib.or_e4m3_decode.restype = C.c_double
            _lib.or_e4m3_encode.restype = C.c_uint8
            _lib.or_e4m3_encode.argtypes = [C.c_float]
            _lib.or_expcast_code_u.argtypes = [C.c_float, C.c_float]
            _lib.or_expcast_code_acc.argtypes = [C.c_int32, C.c_float, C.c_float, C.c_float]
            _lib.or_exp_then_cast_code_acc.argtypes = [C.c_int32, C.c_float, C.c_float]
            _lib.or_fp4_decode.restype = C.c_double
            _lib.or_fp4_decode.argtypes = [C.c_uint8]
            _lib.or_mx_score.restype = C.c_double
    return _lib


def _p(a):
    return a.ctypes.data_as(C.c_void_p) if a is not None else None


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


# ---------------------------------------------------------------------------------------------
# scalar formats
# ---------------------------------------------------------------------------------------------

def e4m3_decode(b) -> np.ndarray:
    b = _c(b, np.uint8)
    out = np.empty(b.shape, np.float64)
    lib().or_e4m3_decode_array(C.c_int(b.size), _p(b), _p(out))
    return out


def e4m3_encode(x) -> np.ndarray:
    x = _c(x, np.float32)
    out = np.empty(x.shape, np.uint8)
    lib().or_e4m3_encode_array(C.c_int(x.size), _p(x), _p(out))
    return out


def fp4_decode(c) -> np.ndarray:
    """E2M1 (OCP MX FP4) codes 0..15 to values."""
    c = np.asarray(c, np.uint8)
    return np.vectorize(lambda v: lib().or_fp4_decode(int(v)), otypes=[np.float64])(c) if c.size else np.zeros(c.shape)


def fp4_encode(x) -> np.ndarray:
    x = _c(x, np.float32)
    out = np.empty(x.shape, np.uint8)
    lib().or_fp4_encode_array(C.c_int(x.size), _p(x), _p(out))
    return out


def mx_blocks(x):
    """MXFP4 quantization of fp32 data [..., 32k] by blocks of 32: (codes uint8 [...], scale bytes)."""
    x = _c(x, np.float32)
    assert x.shape[-1] % 32 == 0
    nb = x.size // 32
    codes = np.empty(x.shape, np.uint8)
    scales = np.empty(x.shape[:-1] + (x.shape[-1] // 32,), np.uint8)
    lib().or_mx_blocks(C.c_int(nb), _p(x), _p(codes), _p(scales))
    return codes, scales


def mx_score(q, qs, k, ks) -> float:
    """Exact score of one query row and one key row from their MX codes [128] and scales [4]."""
    q, k = _c(q, np.uint8), _c(k, np.uint8)
    qs, ks = _c(qs, np.uint8), _c(ks, np.uint8)
    return float(lib().or_mx_score(_p(q), _p(qs), _p(k), _p(ks)))


def bf16_round(x) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round to nearest even."""
    x = _c(x, np.float32)
    out = np.empty(x.shape, np.uint16)
    lib().or_bf16_round_array(C.c_int(x.size), _p(x), _p(out))
    return out


def expcast_code_u(u, beta: float = -0.35) -> np.ndarray:
    """ExpCast-FP8 byte for log2-domain scores u (Sec. 3.3, eq. direct-fp8)."""
    u = _c(u, np.float32)
    out = np.empty(u.shape, np.int32)
    lib().or_expcast_u_array(C.c_int(u.size), _p(u), C.c_float(beta), _p(out))
    return out


def expcast_code_acc(acc: int, a: float, m_new: float, beta: float = -0.35) -> int:
    return int(lib().or_expcast_code_acc(int(acc), float(a), float(m_new), float(beta)))


def exp_then_cast_code_acc(acc: int, a: float, m_new: float) -> int:
    return int(lib().or_exp_then_cast_code_acc(int(acc), float(a), float(m_new)))


def fwht_rows(x) -> np.ndarray:
    """Unnormalised 128-point Walsh-Hadamard transform of each row, fp32 butterflies."""
    x = np.array(x, dtype=np.float32, copy=True, order="C")
    assert x.shape[-1] == D
    lib().or_fwht_rows(C.c_int(x.size // D), _p(x))
    return x


# ---------------------------------------------------------------------------------------------
# rotary embedding
# ---------------------------------------------------------------------------------------------

def rope_tables(F: int, Ht: int, Wd: int, theta: float = 10000.0):
    rows = F + Ht + Wd
    cos_t = np.empty((rows, 64), np.float32)
    sin_t = np.empty((rows, 64), np.float32)
    lib().or_rope_tables(C.c_int(F), C.c_int(Ht), C.c_int(Wd), C.c_double(theta), _p(cos_t), _p(sin_t))
    return cos_t, sin_t


def rope_apply(x, grid) -> np.ndarray:
    """Rotate fp32 rows [N, 128] of one head, token n at its grid position."""
    F, Ht, Wd = grid
    x = np.array(x, dtype=np.float32, copy=True, order="C")
    cos_t, sin_t = rope_tables(F, Ht, Wd)
    lib().or_rope_apply(C.c_int(x.shape[0]), C.c_int(F), C.c_int(Ht), C.c_int(Wd), _p(cos_t), _p(sin_t), _p(x))
    return x


# ---------------------------------------------------------------------------------------------
# preprocessing, attention, grouping
# ---------------------------------------------------------------------------------------------

def prep(Q, K, V, grid, perm=None, q_perm=None, rope=True, hadamard=True, smooth_k=True, smooth_v=True,
         qk_fmt=QK_INT8):
    """Q, K, V: uint16 bf16 bits [B, H, N, 128]. perm / q_perm: int32 [B, H, N] or None.

    Returns a dict of numpy arrays (see ``or_prep_head`` in vc_oracle.c for the layouts); with
    qk_fmt = QK_FP8, q and k hold E4M3 bytes (uint8) with scales amax/448; with qk_fmt = QK_MXFP4 also q_mx / k_mx (one E2M1 code per byte [B, H, Np, 128]) and q_mxs / k_mxs
    (E8M0 scale bytes [B, H, Np, 4]).
    """
    Q, K, V = (_c(t, np.uint16) for t in (Q, K, V))
    B, H, N, d = Q.shape
    assert d == D and K.shape == Q.shape and V.shape == Q.shape
    F, Ht, Wd = grid
    assert F * Ht * Wd == N
    T = (N + BLK - 1) // BLK
    Np = T * BLK
    cos_t, sin_t = rope_tables(F, Ht, Wd)
    perm = _c(perm, np.int32) if perm is not None else None
    q_perm = _c(q_perm, np.int32) if q_perm is not None else None
    out = dict(
        q=np.zeros((B, H, Np, D), np.int8), q_scale=np.zeros((B, H, T), np.float32),
        k=np.zeros((B, H, Np, D), np.int8), k_scale=np.zeros((B, H, T), np.float32),
        k_mean=np.zeros((B, H, D), np.float32),
        v=np.zeros((B, H, Np, D), np.uint8), v_scale=np.zeros((B, H, D), np.float32),
        v_mean=np.zeros((B, H, T, D), np.uint16),
    )
    mx = qk_fmt == QK_MXFP4
    if mx:
        out.update(q_mx=np.zeros((B, H, Np, D), np.uint8), q_mxs=np.zeros((B, H, Np, 4), np.uint8),
                   k_mx=np.zeros((B, H, Np, D), np.uint8), k_mxs=np.zeros((B, H, Np, 4), np.uint8))
    cfg = PrepCfg(N, F, Ht, Wd, int(rope), int(hadamard), int(smooth_k), int(smooth_v), int(qk_fmt))
    rc = lib().or_prep(C.c_int(B * H), C.byref(cfg), _p(Q), _p(K), _p(V), _p(perm), _p(q_perm),
                       _p(cos_t), _p(sin_t), _p(out["q"]), _p(out["q_scale"]), _p(out["k"]),
                       _p(out["k_scale"]), _p(out["k_mean"]), _p(out["v"]), _p(out["v_scale"]),
                       _p(out["v_mean"]), _p(out.get("q_mx")), _p(out.get("q_mxs")), _p(out.get("k_mx")),
                       _p(out.get("k_mxs")))
    if rc != 0:
        raise MemoryError("oracle prep failed")
    if qk_fmt == QK_FP8:
        out["q"], out["k"] = out["q"].view(np.uint8), out["k"].view(np.uint8)
    out.update(N=N, grid=(F, Ht, Wd), hadamard=bool(hadamard), smooth_v=bool(smooth_v), qk_fmt=int(qk_fmt))
    return out


def attention(pp, rows, bh=None, p_mode=P_EXPCAST, sm_scale=None, beta=-0.35):
    """Quantized tiled attention on prepared operands for the given rows (prepared query order).

    rows: int array [R] (same rows for every head) ; bh: list of flat head indices (default all).
    Returns fp64 [len(bh), R, 128] (before the final bf16 rounding).
    """
    B, H = pp["q"].shape[:2]
    N = pp["N"]
    if sm_scale is None:
        sm_scale = float(np.float32(1.0 / np.sqrt(D)))
    rows = _c(rows, np.int32)
    bh = list(range(B * H)) if bh is None else list(bh)
    out = np.zeros((len(bh), rows.size, D), np.float64)
    qk_fmt = int(pp.get("qk_fmt", QK_INT8))
    cfg = AttnCfg(N, int(pp["hadamard"]), int(pp["smooth_v"]), int(p_mode), float(sm_scale), float(beta), qk_fmt)
    q = pp["q"].reshape(B * H, -1, D); qs = pp["q_scale"].reshape(B * H, -1)
    k = pp["k"].reshape(B * H, -1, D); ks = pp["k_scale"].reshape(B * H, -1)
    v = pp["v"].reshape(B * H, -1, D); vs = pp["v_scale"].reshape(B * H, D)
    vm = pp["v_mean"].reshape(B * H, -1, D)
    mx = qk_fmt == QK_MXFP4
    if mx:
        qm = pp["q_mx"].reshape(B * H, -1, D); qms = pp["q_mxs"].reshape(B * H, -1, 4)
        km = pp["k_mx"].reshape(B * H, -1, D); kms = pp["k_mxs"].reshape(B * H, -1, 4)
    for t, h in enumerate(bh):
        o = np.zeros((rows.size, D), np.float64)
        mxargs = [_p(_c(a[h], np.uint8)) for a in (qm, qms, km, kms)] if mx else [None] * 4
        lib().or_attn_head(C.byref(cfg), _p(_c(q[h].view(np.int8), np.int8)), _p(_c(qs[h], np.float32)),
                           _p(_c(k[h].view(np.int8), np.int8)), _p(_c(ks[h], np.float32)), _p(_c(v[h], np.uint8)),
                           _p(_c(vs[h], np.float32)), _p(_c(vm[h], np.uint16)), C.c_int(rows.size),
                           _p(rows), _p(o), *mxargs)
        out[t] = o
    return out


def attention_codes(pp, rows, bh=None, p_mode=P_EXPCAST, sm_scale=None, beta=-0.35):
    """The 8-bit probability codes of the recurrence for the given rows (prepared query order):
    uint8 [len(bh), R, 128 T], key order of the prepared K' (padded keys 0), each tile's codes at
    that tile's running maximum."""
    B, H = pp["q"].shape[:2]
    N = pp["N"]
    T = (N + BLK - 1) // BLK
    if sm_scale is None:
        sm_scale = float(np.float32(1.0 / np.sqrt(D)))
    rows = _c(rows, np.int32)
    bh = list(range(B * H)) if bh is None else list(bh)
    out = np.zeros((len(bh), rows.size, T * BLK), np.uint8)
    qk_fmt = int(pp.get("qk_fmt", QK_INT8))
    cfg = AttnCfg(N, int(pp["hadamard"]), int(pp["smooth_v"]), int(p_mode), float(sm_scale), float(beta), qk_fmt)
    q = pp["q"].reshape(B * H, -1, D); qs = pp["q_scale"].reshape(B * H, -1)
    k = pp["k"].reshape(B * H, -1, D); ks = pp["k_scale"].reshape(B * H, -1)
    v = pp["v"].reshape(B * H, -1, D); vs = pp["v_scale"].reshape(B * H, D)
    vm = pp["v_mean"].reshape(B * H, -1, D)
    mx = qk_fmt == QK_MXFP4
    if mx:
        qm = pp["q_mx"].reshape(B * H, -1, D); qms = pp["q_mxs"].reshape(B * H, -1, 4)
        km = pp["k_mx"].reshape(B * H, -1, D); kms = pp["k_mxs"].reshape(B * H, -1, 4)
    scratch = np.zeros((rows.size, D), np.float64)
    for t, h in enumerate(bh):
        codes = np.zeros((rows.size, T * BLK), np.uint8)
        mxargs = [_p(_c(a[h], np.uint8)) for a in (qm, qms, km, kms)] if mx else [None] * 4
        lib().or_attn_head_codes(C.byref(cfg), _p(_c(q[h].view(np.int8), np.int8)), _p(_c(qs[h], np.float32)),
                                 _p(_c(k[h].view(np.int8), np.int8)), _p(_c(ks[h], np.float32)),
                                 _p(_c(v[h], np.uint8)), _p(_c(vs[h], np.float32)), _p(_c(vm[h], np.uint16)),
                                 C.c_int(rows.size), _p(rows), _p(scratch), *mxargs, _p(codes))
        out[t] = codes
    return out


def attention_tiled_f64(Qf, Kf, Vf, rows, sm_scale=None, smooth_v=True):
    """The online recurrence with block-mean restoration on full-precision rows of one head."""
    Qf, Kf, Vf = (_c(t, np.float64) for t in (Qf, Kf, Vf))
    N = Kf.shape[0]
    if sm_scale is None:
        sm_scale = 1.0 / np.sqrt(D)
    rows = _c(rows, np.int32)
    out = np.zeros((rows.size, D), np.float64)
    lib().or_attn_tiled_f64(C.c_int(N), _p(Qf), _p(Kf), _p(Vf), C.c_double(sm_scale), C.c_int(int(smooth_v)),
                            C.c_int(rows.size), _p(rows), _p(out))
    return out


def reference_attention(Q, K, V, grid, rows, bh=None, rope=True, sm_scale=None):
    """Exact fp64 softmax attention from the bf16 inputs for the given query token rows."""
    Q, K, V = (_c(t, np.uint16) for t in (Q, K, V))
    B, H, N, _ = Q.shape
    F, Ht, Wd = grid
    if sm_scale is None:
        sm_scale = 1.0 / np.sqrt(D)
    rows = _c(rows, np.int32)
    bh = list(range(B * H)) if bh is None else list(bh)
    q = Q.reshape(B * H, N, D); k = K.reshape(B * H, N, D); v = V.reshape(B * H, N, D)
    out = np.zeros((len(bh), rows.size, D), np.float64)
    for t, h in enumerate(bh):
        o = np.zeros((rows.size, D), np.float64)
        lib().or_ref_attn_head(C.c_int(N), C.c_int(F), C.c_int(Ht), C.c_int(Wd), C.c_int(int(rope)),
                               C.c_double(sm_scale), _p(_c(q[h], np.uint16)), _p(_c(k[h], np.uint16)),
                               _p(_c(v[h], np.uint16)), C.c_int(rows.size), _p(rows), _p(o))
        out[t] = o
    return out


def group(V, grid, mode=GROUP_KMEANS, k=32, iters=8, warm_start=False, cent_in=None, cube=(4, 2, 16)):
    """Value-guided grouping per head. V: uint16 bf16 bits [B, H, N, 128].

    Returns dict(labels, perm, inv_perm int32 [B,H,N], centroids fp32 [B,H,k,128]).
    """
    V = _c(V, np.uint16)
    B, H, N, _ = V.shape
    F, Ht, Wd = grid
    assert F * Ht * Wd == N
    if warm_start:
        assert cent_in is not None
        cent_in = _c(cent_in, np.float32)
    kk = max(int(k), 1)
    out = dict(labels=np.zeros((B, H, N), np.int32), perm=np.zeros((B, H, N), np.int32),
               inv_perm=np.zeros((B, H, N), np.int32), centroids=np.zeros((B, H, kk, D), np.float32))
    cfg = GroupCfg(N, F, Ht, Wd, int(mode), int(k), int(iters), int(bool(warm_start)), *[int(c) for c in cube])
    rc = lib().or_group(C.c_int(B * H), C.byref(cfg), _p(V), _p(cent_in if warm_start else None),
                        _p(out["labels"]), _p(out["perm"]), _p(out["inv_perm"]), _p(out["centroids"]))
    if rc != 0:
        raise MemoryError("oracle group failed")
    return out


def group_codes(V_head):
    """Per-head INT8 codes of V used by the k-means (uint16 bf16 bits [N, 128])."""
    V_head = _c(V_head, np.uint16)
    N = V_head.shape[0]
    x = np.zeros((N, D), np.int8)
    s = np.zeros(1, np.float32)
    lib().or_group_codes(C.c_int(N), _p(V_head), _p(x), _p(s))
    return x, float(s[0])


def bf16_to_f32(bits) -> np.ndarray:
    """bf16 bit patterns to fp32 (exact widening)."""
    return (np.asarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32)
