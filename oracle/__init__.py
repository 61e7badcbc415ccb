"""Python access to the CPU oracle for MEC (Cho & Brand, ICML 2017).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the CPU
baseline leg of the benchmark are the only users. The GPU library never
imports this package, and this package imports nothing from the GPU library.

Arrays are numpy, C-contiguous. fp32 tensors are ``float32`` arrays; bf16
tensors are ``uint16`` arrays holding the bf16 bit patterns. Outputs of the
arithmetic routines are ``float64``.
"""
import ctypes
import os

import numpy as np

from . import brute  # noqa: F401  (independent pure-Python brute force)

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

F32, BF16, F64 = 0, 1, 2

_i64 = ctypes.c_int64
_DIMS = [_i64] * 9


def _load(path):
    """Load an oracle shared library at ``path`` and declare its signatures."""
    L = ctypes.CDLL(path)
    vp, dp = ctypes.c_void_p, ctypes.POINTER(ctypes.c_double)
    L.oracle_out_dim.argtypes = [_i64] * 3
    L.oracle_out_dim.restype = _i64
    for name in ("oracle_lowered_elems", "oracle_im2col_elems", "oracle_saving_R"):
        getattr(L, name).argtypes = _DIMS
        getattr(L, name).restype = _i64
    L.oracle_conv2d_direct.argtypes = [vp, vp, dp] + _DIMS + [ctypes.c_int]
    L.oracle_conv2d_direct.restype = None
    L.oracle_conv2d_points.argtypes = [vp, vp, vp, _i64, dp] + _DIMS + [ctypes.c_int]
    L.oracle_conv2d_points.restype = None
    L.oracle_mec_lower.argtypes = [vp, vp] + _DIMS + [ctypes.c_int]
    L.oracle_mec_lower.restype = None
    L.oracle_im2col.argtypes = [vp, vp] + _DIMS + [ctypes.c_int]
    L.oracle_im2col.restype = None
    L.oracle_mec_gemm.argtypes = [vp, vp, dp] + _DIMS + [ctypes.c_int]
    L.oracle_mec_gemm.restype = None
    L.oracle_mec_conv2d.argtypes = [vp, vp, dp] + _DIMS + [ctypes.c_int]
    L.oracle_mec_conv2d.restype = ctypes.c_int
    L.oracle_vanilla_mec.argtypes = [vp, vp, dp, vp] + [_i64] * 6
    L.oracle_vanilla_mec.restype = None
    for name in ("oracle_conv2d_dgrad", "oracle_conv2d_wgrad", "oracle_mec_dgrad_lowered",
                 "oracle_mec_wgrad_lowered", "oracle_mec_fold"):
        getattr(L, name).argtypes = [vp, vp, dp] if name != "oracle_mec_fold" else [vp, dp]
        getattr(L, name).argtypes += _DIMS + [ctypes.c_int]
        getattr(L, name).restype = None
    L.oracle_num_threads.argtypes = []
    L.oracle_num_threads.restype = ctypes.c_int
    L.oracle_set_num_threads.argtypes = [ctypes.c_int]
    L.oracle_set_num_threads.restype = None
    return L


def lib():
    """Load liboracle.so, building it first only if it is absent."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            from . import build as _build
            _build.build()
        _lib = _load(_LIB_PATH)
    return _lib


def _dtype_code(a):
    if a.dtype == np.float32:
        return F32
    if a.dtype == np.uint16:
        return BF16
    raise TypeError("oracle arrays must be float32 or uint16 (bf16 bits), got %s" % a.dtype)


def _ptr(a):
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.c_void_p)


def _dptr(a):
    assert a.flags["C_CONTIGUOUS"] and a.dtype == np.float64
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _dims(I, K, s_h, s_w):
    i_n, i_h, i_w, i_c = I.shape
    k_h, k_w, k_c2, k_c = K.shape
    if k_c2 != i_c:
        raise ValueError("K must be k_h x k_w x i_c x k_c")
    return (i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w)


def out_dim(i, k, s):
    """Eq. (1), floor reading."""
    return lib().oracle_out_dim(i, k, s)


def lowered_elems(*dims):
    """|L| = i_n*o_w*i_h*k_w*i_c (dims in Table 1 order)."""
    return lib().oracle_lowered_elems(*dims)


def im2col_elems(*dims):
    """|im2col| = i_n*o_h*o_w*k_h*k_w*i_c (dims in Table 1 order)."""
    return lib().oracle_im2col_elems(*dims)


def saving_R(*dims):
    """Eq. (4): i_n*i_c*o_w*k_w*(o_h*k_h - i_h)."""
    return lib().oracle_saving_R(*dims)


def conv2d_direct(I, K, s_h, s_w):
    """Direct convolution (fp64 result, n-h-w-c)."""
    d = _dims(I, K, s_h, s_w)
    dt = _dtype_code(I)
    assert _dtype_code(K) == dt
    o_h, o_w = out_dim(d[1], d[4], s_h), out_dim(d[2], d[5], s_w)
    O = np.empty((d[0], o_h, o_w, d[6]), np.float64)
    lib().oracle_conv2d_direct(_ptr(I), _ptr(K), _dptr(O), *d, dt)
    return O


def conv2d_points(I, K, s_h, s_w, idx):
    """Direct convolution at the (n, y, x, m) rows of idx only (fp64)."""
    d = _dims(I, K, s_h, s_w)
    dt = _dtype_code(I)
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    assert idx.ndim == 2 and idx.shape[1] == 4
    out = np.empty(idx.shape[0], np.float64)
    lib().oracle_conv2d_points(_ptr(I), _ptr(K), _ptr(idx), idx.shape[0], _dptr(out), *d, dt)
    return out


def mec_lower(I, k_h, k_w, k_c, s_h, s_w):
    """MEC compact lowering; returns L (i_n x o_w x i_h x k_w x i_c)."""
    i_n, i_h, i_w, i_c = I.shape
    o_w = out_dim(i_w, k_w, s_w)
    L = np.empty((i_n, o_w, i_h, k_w, i_c), I.dtype)
    lib().oracle_mec_lower(_ptr(I), _ptr(L), i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w,
                           _dtype_code(I))
    return L


def im2col(I, k_h, k_w, s_h, s_w):
    """im2col matrix, (i_n*o_h*o_w) x (k_h*k_w*i_c)."""
    i_n, i_h, i_w, i_c = I.shape
    o_h, o_w = out_dim(i_h, k_h, s_h), out_dim(i_w, k_w, s_w)
    M = np.empty((i_n * o_h * o_w, k_h * k_w * i_c), I.dtype)
    lib().oracle_im2col(_ptr(I), _ptr(M), i_n, i_h, i_w, i_c, k_h, k_w, 1, s_h, s_w,
                        _dtype_code(I))
    return M


def mec_gemm(L, K, i_h, i_w, s_h, s_w):
    """MEC product phase on a lowered L, from its definition (fp64 O, n-h-w-c):
    O[n, h, w, m] = sum_j L[n, w][s_h*R*h + j] * K[j, m]."""
    i_n, o_w, i_h2, k_w, i_c = L.shape
    assert i_h2 == i_h
    k_h, k_w2, i_c2, k_c = K.shape
    assert (k_w2, i_c2) == (k_w, i_c)
    o_h = out_dim(i_h, k_h, s_h)
    O = np.empty((i_n, o_h, o_w, k_c), np.float64)
    lib().oracle_mec_gemm(_ptr(L), _ptr(K), _dptr(O), i_n, i_h, i_w, i_c, k_h, k_w, k_c,
                          s_h, s_w, _dtype_code(L))
    return O


def mec_conv2d(I, K, s_h, s_w):
    """MEC end to end: the compact lowering, then the product phase (fp64 O)."""
    d = _dims(I, K, s_h, s_w)
    o_h, o_w = out_dim(d[1], d[4], s_h), out_dim(d[2], d[5], s_w)
    O = np.empty((d[0], o_h, o_w, d[6]), np.float64)
    rc = lib().oracle_mec_conv2d(_ptr(I), _ptr(K), _dptr(O), *d, _dtype_code(I))
    if rc != 0:
        raise RuntimeError("oracle_mec_conv2d failed (%d)" % rc)
    return O


def vanilla_mec(I, K, s_h, s_w):
    """MEC for one image and one channel (Section 3.2, Algorithm 1's case
    i_n = i_c = k_c = 1): returns (O fp64 o_h x o_w, L fp32)."""
    I = np.ascontiguousarray(I, np.float32)
    K = np.ascontiguousarray(K, np.float32)
    i_h, i_w = I.shape
    k_h, k_w = K.shape
    o_h, o_w = out_dim(i_h, k_h, s_h), out_dim(i_w, k_w, s_w)
    O = np.empty((o_h, o_w), np.float64)
    L = np.empty((o_w, i_h * k_w), np.float32)
    lib().oracle_vanilla_mec(_ptr(I), _ptr(K), _dptr(O), _ptr(L), i_h, i_w, k_h, k_w, s_h, s_w)
    return O, L


# ---------------------------------------------------------------- training
# Gradients of the convolution (derived from its definition; the paper gives
# no backward algorithm). G = dloss/dO has O's shape, i_n x o_h x o_w x k_c.

def _grad_dims(G, i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w):
    o_h, o_w = out_dim(i_h, k_h, s_h), out_dim(i_w, k_w, s_w)
    if G.shape != (i_n, o_h, o_w, k_c):
        raise ValueError("G must be i_n x o_h x o_w x k_c = %s, got %s"
                         % ((i_n, o_h, o_w, k_c), G.shape))
    return (i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w)


def conv2d_dgrad(G, K, i_h, i_w, s_h, s_w):
    """dI = dloss/dI of the direct convolution (fp64, n-h-w-c)."""
    k_h, k_w, i_c, k_c = K.shape
    d = _grad_dims(G, G.shape[0], i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w)
    dt = _dtype_code(G)
    assert _dtype_code(K) == dt
    dI = np.empty((d[0], i_h, i_w, i_c), np.float64)
    lib().oracle_conv2d_dgrad(_ptr(G), _ptr(K), _dptr(dI), *d, dt)
    return dI


def conv2d_wgrad(I, G, k_h, k_w, s_h, s_w):
    """dK = dloss/dK of the direct convolution (fp64, k_h x k_w x i_c x k_c)."""
    i_n, i_h, i_w, i_c = I.shape
    d = _grad_dims(G, i_n, i_h, i_w, i_c, k_h, k_w, G.shape[3], s_h, s_w)
    dt = _dtype_code(I)
    assert _dtype_code(G) == dt
    dK = np.empty((k_h, k_w, i_c, G.shape[3]), np.float64)
    lib().oracle_conv2d_wgrad(_ptr(I), _ptr(G), _dptr(dK), *d, dt)
    return dK


def mec_dgrad_lowered(G, K, i_h, i_w, s_h, s_w):
    """dL = dloss/dL through the slab products (fp64, L's shape)."""
    k_h, k_w, i_c, k_c = K.shape
    d = _grad_dims(G, G.shape[0], i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w)
    dt = _dtype_code(G)
    assert _dtype_code(K) == dt
    dL = np.empty((d[0], G.shape[2], i_h, k_w, i_c), np.float64)
    lib().oracle_mec_dgrad_lowered(_ptr(G), _ptr(K), _dptr(dL), *d, dt)
    return dL


def mec_wgrad_lowered(L, G, k_h, s_h, s_w):
    """dK as the sum over output rows of A_h^T G_h, A_h the slabs of L (fp64)."""
    i_n, o_w, i_h, k_w, i_c = L.shape
    i_w = (o_w - 1) * s_w + k_w
    d = _grad_dims(G, i_n, i_h, i_w, i_c, k_h, k_w, G.shape[3], s_h, s_w)
    dt = _dtype_code(L)
    assert _dtype_code(G) == dt
    dK = np.empty((k_h, k_w, i_c, G.shape[3]), np.float64)
    lib().oracle_mec_wgrad_lowered(_ptr(L), _ptr(G), _dptr(dK), *d, dt)
    return dK


def mec_fold(dL, i_w, s_w):
    """The adjoint of the lowering: dI[n, h, s_w*w + b, c] += dL[n, w, h, b, c]
    (fp64). dL is float32, bf16 bits (uint16) or float64."""
    i_n, o_w, i_h, k_w, i_c = dL.shape
    if out_dim(i_w, k_w, s_w) != o_w:
        raise ValueError("i_w, s_w do not give o_w = %d columns" % o_w)
    dt = F64 if dL.dtype == np.float64 else _dtype_code(dL)
    dI = np.empty((i_n, i_h, i_w, i_c), np.float64)
    lib().oracle_mec_fold(_ptr(dL), _dptr(dI), i_n, i_h, i_w, i_c, 1, k_w, 1, 1, s_w, dt)
    return dI


def num_threads():
    return lib().oracle_num_threads()


def set_num_threads(n):
    """Thread count of the oracle's later parallel loops."""
    lib().oracle_set_num_threads(int(n))
