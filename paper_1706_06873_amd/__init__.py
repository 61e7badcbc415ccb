"""MI355X (gfx950) MEC convolution: thin Python binding of ``include/mec.h``.

MEC is the memory-efficient convolution of Cho & Brand (ICML 2017): a compact
lowering of the input I into L (i_n x o_w x i_h x k_w x i_c), then o_h small
matrix products over overlapping slabs of L. Every step runs in the HIP kernels
of ``libmec.so``; this module only marshals arguments. PyTorch supplies device
memory and streams: tensors passed here must be contiguous tensors on a HIP
device. There is no CPU fallback: if the library is missing, importing this
package raises.

Layouts (paper notation): I is i_n x i_h x i_w x i_c, K is k_h x k_w x i_c x
k_c, O is i_n x o_h x o_w x k_c (fp32). I and K are both fp32 or both bf16.
"""
import ctypes
import os

# torch first: importing it loads its HIP runtime, and libmec.so then binds to
# that same runtime. Loaded the other way round, the process would map a
# second HIP runtime (the system one) beside torch's, and device memory and
# streams from one are not valid in the other.
import torch  # noqa: E402,F401

__all__ = [
    "MecError", "F32", "BF16", "LOWERED", "FUSED", "IM2COL", "lib", "output_dims",
    "workspace_bytes", "im2col_bytes", "lower", "im2col", "gemm", "conv2d", "strerror",
    "GRAD_INPUT", "GRAD_KERNEL", "GRAD_KERNEL_FROM_L", "grad_workspace_bytes", "fold",
    "dgrad_gemm", "conv2d_dgrad", "wgrad_gemm", "conv2d_wgrad", "noalloc_scratch_bytes",
    "conv2d_wgrad_noalloc",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmec.so")

F32, BF16 = 0, 1
LOWERED, FUSED, IM2COL = 0, 1, 2
GRAD_INPUT, GRAD_KERNEL, GRAD_KERNEL_FROM_L = 0, 1, 2
_ALGOS = {"lowered": LOWERED, "fused": FUSED, "im2col": IM2COL,
          LOWERED: LOWERED, FUSED: FUSED, IM2COL: IM2COL}

if not os.path.exists(LIB_PATH):
    raise ImportError("%s is not built; run `python paper_1706_06873_amd/build.py`" % LIB_PATH)

_i = ctypes.c_int
_vp = ctypes.c_void_p
_DIMS = [_i] * 9


def _load(path):
    L = ctypes.CDLL(path)
    L.mec_output_dims.argtypes = [_i] * 6 + [ctypes.POINTER(_i), ctypes.POINTER(_i)]
    L.mec_output_dims.restype = _i
    L.mec_workspace_bytes.argtypes = _DIMS + [_i, _i]
    L.mec_workspace_bytes.restype = ctypes.c_int64
    L.mec_im2col_bytes.argtypes = _DIMS + [_i]
    L.mec_im2col_bytes.restype = ctypes.c_int64
    L.mec_lower.argtypes = [_vp, _vp] + _DIMS + [_i, _vp]
    L.mec_lower.restype = _i
    L.mec_im2col.argtypes = [_vp, _vp] + _DIMS + [_i, _vp]
    L.mec_im2col.restype = _i
    L.mec_gemm.argtypes = [_vp, _vp, _vp] + _DIMS + [_i, _vp]
    L.mec_gemm.restype = _i
    L.mec_conv2d.argtypes = [_vp, _vp, _vp, _vp, ctypes.c_size_t] + _DIMS + [_i, _i, _vp]
    L.mec_conv2d.restype = _i
    L.mec_grad_workspace_bytes.argtypes = _DIMS + [_i, _i]
    L.mec_grad_workspace_bytes.restype = ctypes.c_int64
    L.mec_fold.argtypes = [_vp, _vp] + _DIMS + [_vp]
    L.mec_fold.restype = _i
    L.mec_dgrad_gemm.argtypes = [_vp, _vp, _vp] + _DIMS + [_i, _vp]
    L.mec_dgrad_gemm.restype = _i
    for name in ("mec_conv2d_dgrad", "mec_wgrad_gemm", "mec_conv2d_wgrad"):
        getattr(L, name).argtypes = [_vp, _vp, _vp, _vp, ctypes.c_size_t] + _DIMS + [_i, _vp]
        getattr(L, name).restype = _i
    L.mec_noalloc_scratch_bytes.argtypes = []
    L.mec_noalloc_scratch_bytes.restype = ctypes.c_int64
    L.mec_conv2d_wgrad_noalloc.argtypes = [_vp, _vp, _vp] + _DIMS + [_i, _vp]
    L.mec_conv2d_wgrad_noalloc.restype = _i
    L.mec_strerror.argtypes = [_i]
    L.mec_strerror.restype = ctypes.c_char_p
    L.mec_last_error.argtypes = []
    L.mec_last_error.restype = ctypes.c_char_p
    return L


def _hip_runtimes():
    """Distinct HIP runtime libraries mapped into this process."""
    try:
        with open("/proc/self/maps") as f:
            paths = {line.split()[-1] for line in f if "libamdhip64" in line}
    except OSError:
        return []
    return sorted(os.path.realpath(p) for p in paths)


lib = _load(LIB_PATH)
if len(_hip_runtimes()) > 1:
    raise ImportError("two HIP runtimes are loaded in this process (%s): libmec.so must bind to "
                      "the one torch uses" % ", ".join(_hip_runtimes()))


class MecError(RuntimeError):
    """A negative status from the library."""

    def __init__(self, status, what):
        self.status = status
        detail = lib.mec_last_error().decode() if status == -4 else ""
        super().__init__("%s: %s (status %d)%s" % (what, strerror(status), status,
                                                    " -- " + detail if detail else ""))


def strerror(status):
    return lib.mec_strerror(status).decode()


def _check(status, what):
    if status < 0:
        raise MecError(int(status), what)
    return status


def output_dims(i_h, i_w, k_h, k_w, s_h, s_w):
    """(o_h, o_w) by Eq. (1), floor reading."""
    o_h, o_w = _i(), _i()
    _check(lib.mec_output_dims(i_h, i_w, k_h, k_w, s_h, s_w, ctypes.byref(o_h), ctypes.byref(o_w)),
           "mec_output_dims")
    return o_h.value, o_w.value


def _dtype_code(t):
    import torch
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError("I and K must be float32 or bfloat16, got %s" % t.dtype)


def workspace_bytes(i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w, dtype=F32, algo=LOWERED):
    return _check(lib.mec_workspace_bytes(i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w, dtype,
                                          _ALGOS[algo]), "mec_workspace_bytes")


def im2col_bytes(i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w, dtype=F32):
    return _check(lib.mec_im2col_bytes(i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w, dtype),
                  "mec_im2col_bytes")


def _stream_handle(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _dev_ptr(t, name):
    if not t.is_cuda:
        raise ValueError("%s must be a device tensor" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    return ctypes.c_void_p(t.data_ptr())


def _same_device(t, ref, name):
    if t.device != ref.device:
        raise ValueError("%s is on %s, the inputs on %s" % (name, t.device, ref.device))


def _check_out(t, shape, dtype, ref, name):
    """A caller-supplied output must have exactly the shape, dtype and device
    the kernels write, so they never write past its end."""
    if tuple(t.shape) != tuple(shape) or t.dtype != dtype:
        raise ValueError("%s must be %s of shape %s, got %s of shape %s"
                         % (name, dtype, tuple(shape), t.dtype, tuple(t.shape)))
    _same_device(t, ref, name)


def _dims(I, K, s_h, s_w):
    if I.dim() != 4 or K.dim() != 4:
        raise ValueError("I must be i_n x i_h x i_w x i_c and K k_h x k_w x i_c x k_c")
    i_n, i_h, i_w, i_c = I.shape
    k_h, k_w, k_ic, k_c = K.shape
    if k_ic != i_c:
        raise ValueError("K's third dimension (%d) must equal i_c (%d)" % (k_ic, i_c))
    if I.dtype != K.dtype:
        raise TypeError("I and K must have the same dtype")
    _same_device(K, I, "K")
    return (i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w)


def lower(I, k_h, k_w, k_c, s_h, s_w, L=None, stream=None):
    """MEC lowering of I into L (i_n x o_w x i_h x k_w x i_c); returns L. A
    given L must hold exactly mec_workspace_bytes(..., LOWERED) bytes of I's
    dtype (any shape)."""
    import torch
    if I.dim() != 4:
        raise ValueError("I must be i_n x i_h x i_w x i_c")
    i_n, i_h, i_w, i_c = I.shape
    dt = _dtype_code(I)
    _, o_w = output_dims(i_h, i_w, k_h, k_w, s_h, s_w)
    need = workspace_bytes(i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w, dtype=dt, algo=LOWERED)
    if L is None:
        L = torch.empty((i_n, o_w, i_h, k_w, i_c), dtype=I.dtype, device=I.device)
    _same_device(L, I, "L")
    if L.numel() * L.element_size() != need or L.dtype != I.dtype:
        raise ValueError("L must hold %d bytes of %s" % (need, I.dtype))
    _check(lib.mec_lower(_dev_ptr(I, "I"), _dev_ptr(L, "L"), i_n, i_h, i_w, i_c, k_h, k_w, k_c,
                         s_h, s_w, dt, _stream_handle(stream)), "mec_lower")
    return L


def im2col(I, k_h, k_w, k_c, s_h, s_w, M=None, stream=None):
    """im2col lowering of I, rows in (n, x, y) order: M is
    i_n x o_w x o_h x k_h x k_w x i_c. Returns M. A given M must hold exactly
    mec_im2col_bytes bytes of I's dtype (any shape)."""
    import torch
    if I.dim() != 4:
        raise ValueError("I must be i_n x i_h x i_w x i_c")
    i_n, i_h, i_w, i_c = I.shape
    dt = _dtype_code(I)
    o_h, o_w = output_dims(i_h, i_w, k_h, k_w, s_h, s_w)
    need = im2col_bytes(i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w, dtype=dt)
    if M is None:
        M = torch.empty((i_n, o_w, o_h, k_h, k_w, i_c), dtype=I.dtype, device=I.device)
    _same_device(M, I, "M")
    if M.numel() * M.element_size() != need or M.dtype != I.dtype:
        raise ValueError("M must hold %d bytes of %s" % (need, I.dtype))
    _check(lib.mec_im2col(_dev_ptr(I, "I"), _dev_ptr(M, "M"), i_n, i_h, i_w, i_c, k_h, k_w, k_c,
                          s_h, s_w, dt, _stream_handle(stream)), "mec_im2col")
    return M


def _out(I, K, s_h, s_w, O):
    import torch
    d = _dims(I, K, s_h, s_w)
    o_h, o_w = output_dims(d[1], d[2], d[4], d[5], s_h, s_w)
    shape = (d[0], o_h, o_w, d[6])
    if O is None:
        O = torch.empty(shape, dtype=torch.float32, device=I.device)
    _check_out(O, shape, torch.float32, I, "O")
    return d, O


def gemm(L, K, i_h, i_w, s_h, s_w, O=None, stream=None):
    """MEC's slab products on a lowered L (i_n x o_w x i_h x k_w x i_c); returns O.
    K is k_h x k_w x i_c x k_c of L's dtype; a given O must be float32 of shape
    i_n x o_h x o_w x k_c."""
    import torch
    if L.dim() != 5 or K.dim() != 4:
        raise ValueError("L must be i_n x o_w x i_h x k_w x i_c and K k_h x k_w x i_c x k_c")
    i_n, o_w, l_ih, k_w, i_c = L.shape
    k_h, kk_w, k_ic, k_c = K.shape
    if l_ih != i_h or kk_w != k_w or k_ic != i_c:
        raise ValueError("L (%s) and K (%s) do not agree on i_h, k_w and i_c"
                         % (tuple(L.shape), tuple(K.shape)))
    if K.dtype != L.dtype:
        raise TypeError("L and K must have the same dtype")
    _same_device(K, L, "K")
    dt = _dtype_code(L)
    o_h, o_w2 = output_dims(i_h, i_w, k_h, k_w, s_h, s_w)
    if o_w2 != o_w:
        raise ValueError("L's o_w does not match i_w, k_w, s_w")
    shape = (i_n, o_h, o_w, k_c)
    if O is None:
        O = torch.empty(shape, dtype=torch.float32, device=L.device)
    _check_out(O, shape, torch.float32, L, "O")
    _check(lib.mec_gemm(_dev_ptr(L, "L"), _dev_ptr(K, "K"), _dev_ptr(O, "O"), i_n, i_h, i_w, i_c,
                        k_h, k_w, k_c, s_h, s_w, dt, _stream_handle(stream)), "mec_gemm")
    return O


def _given_workspace(need, workspace, ref):
    """(pointer, bytes) of the workspace: a given one is checked for size and
    device, else one of `need` bytes is allocated."""
    import torch
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=ref.device)
    _same_device(workspace, ref, "workspace")
    nbytes = workspace.numel() * workspace.element_size()
    if nbytes < need:
        raise ValueError("the workspace holds %d bytes, %d are needed" % (nbytes, need))
    return workspace, _dev_ptr(workspace, "workspace"), nbytes


def conv2d(I, K, s_h=1, s_w=1, algo="lowered", workspace=None, O=None, stream=None):
    """O = I * K by MEC ("lowered", "fused") or by the im2col baseline
    ("im2col"). With "lowered" or "im2col" a workspace of workspace_bytes(...)
    bytes is allocated unless given (a device tensor of at least that many
    bytes); after the call it holds L (or the im2col matrix). Returns O."""
    d, O = _out(I, K, s_h, s_w, O)
    a = _ALGOS[algo]
    dt = _dtype_code(I)
    ws_ptr, ws_bytes = None, 0
    if a != FUSED:
        need = workspace_bytes(*d, dtype=dt, algo=a)
        workspace, ws_ptr, ws_bytes = _given_workspace(need, workspace, I)
    _check(lib.mec_conv2d(_dev_ptr(I, "I"), _dev_ptr(K, "K"), _dev_ptr(O, "O"), ws_ptr, ws_bytes,
                          *d, dt, a, _stream_handle(stream)), "mec_conv2d")
    return O


# ---------------------------------------------------------------- training passes
# Gradients of the convolution through MEC's lowered layout, fp32 only. G is
# dloss/dO (O's shape, float32).

def grad_workspace_bytes(i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w, dtype=F32,
                         grad_pass=GRAD_INPUT):
    return _check(lib.mec_grad_workspace_bytes(i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w, dtype,
                                               grad_pass), "mec_grad_workspace_bytes")


def _f32(t, name):
    import torch
    if t.dtype != torch.float32:
        raise TypeError("%s must be float32" % name)
    return _dev_ptr(t, name)


def fold(dL, i_w, s_w, dI=None, stream=None):
    """The adjoint of the lowering: dI[n, h, s_w*w + b, c] += dL[n, w, h, b, c]
    for dL of L's shape (i_n x o_w x i_h x k_w x i_c, float32). Returns dI."""
    import torch
    if dL.dim() != 5:
        raise ValueError("dL must be i_n x o_w x i_h x k_w x i_c")
    i_n, o_w, i_h, k_w, i_c = dL.shape
    if output_dims(i_h, i_w, 1, k_w, 1, s_w)[1] != o_w:
        raise ValueError("i_w, k_w, s_w do not give dL's o_w")
    shape = (i_n, i_h, i_w, i_c)
    if dI is None:
        dI = torch.empty(shape, dtype=torch.float32, device=dL.device)
    _check_out(dI, shape, torch.float32, dL, "dI")
    _check(lib.mec_fold(_f32(dL, "dL"), _f32(dI, "dI"), i_n, i_h, i_w, i_c, 1, k_w, 1, 1, s_w,
                        _stream_handle(stream)), "mec_fold")
    return dI


def _grad_dims(G, K, i_h, i_w, s_h, s_w):
    if G.dim() != 4 or K.dim() != 4:
        raise ValueError("G must be i_n x o_h x o_w x k_c and K k_h x k_w x i_c x k_c")
    k_h, k_w, i_c, k_c = K.shape
    i_n = G.shape[0]
    o_h, o_w = output_dims(i_h, i_w, k_h, k_w, s_h, s_w)
    if tuple(G.shape) != (i_n, o_h, o_w, k_c):
        raise ValueError("G must be i_n x o_h x o_w x k_c = %s" % ((i_n, o_h, o_w, k_c),))
    _same_device(K, G, "K")
    return (i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w)


def dgrad_gemm(G, K, i_h, i_w, s_h=1, s_w=1, dL=None, stream=None):
    """dL = dloss/dL (L's shape, float32): G_h K^T added into every slab."""
    import torch
    d = _grad_dims(G, K, i_h, i_w, s_h, s_w)
    shape = (d[0], G.shape[2], i_h, d[5], d[3])
    if dL is None:
        dL = torch.empty(shape, dtype=torch.float32, device=G.device)
    _check_out(dL, shape, torch.float32, G, "dL")
    _check(lib.mec_dgrad_gemm(_f32(G, "G"), _f32(K, "K"), _f32(dL, "dL"), *d, F32,
                              _stream_handle(stream)), "mec_dgrad_gemm")
    return dL


def conv2d_dgrad(G, K, i_h, i_w, s_h=1, s_w=1, dI=None, workspace=None, stream=None):
    """dI = dloss/dI (I's shape, float32); on the dL path the workspace then
    holds dL, on the sub-pixel phase path the last phase's padded G and kernel."""
    import torch
    d = _grad_dims(G, K, i_h, i_w, s_h, s_w)
    shape = (d[0], i_h, i_w, d[3])
    if dI is None:
        dI = torch.empty(shape, dtype=torch.float32, device=G.device)
    _check_out(dI, shape, torch.float32, G, "dI")
    need = grad_workspace_bytes(*d, grad_pass=GRAD_INPUT)
    workspace, wp, wb = _given_workspace(need, workspace, G)
    _check(lib.mec_conv2d_dgrad(_f32(G, "G"), _f32(K, "K"), _f32(dI, "dI"), wp, wb, *d, F32,
                                _stream_handle(stream)), "mec_conv2d_dgrad")
    return dI


def wgrad_gemm(L, G, k_h, i_w, s_h=1, s_w=1, dK=None, workspace=None, stream=None):
    """dK = dloss/dK from a lowered L (i_n x o_w x i_h x k_w x i_c, float32):
    the sum over h of A_h^T G_h. Returns dK (k_h x k_w x i_c x k_c)."""
    import torch
    if L.dim() != 5 or G.dim() != 4:
        raise ValueError("L must be i_n x o_w x i_h x k_w x i_c and G i_n x o_h x o_w x k_c")
    i_n, o_w, i_h, k_w, i_c = L.shape
    k_c = G.shape[3]
    o_h, o_w2 = output_dims(i_h, i_w, k_h, k_w, s_h, s_w)
    if o_w2 != o_w or tuple(G.shape) != (i_n, o_h, o_w, k_c):
        raise ValueError("L and G do not match the shape")
    _same_device(G, L, "G")
    d = (i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w)
    shape = (k_h, k_w, i_c, k_c)
    if dK is None:
        dK = torch.empty(shape, dtype=torch.float32, device=G.device)
    _check_out(dK, shape, torch.float32, G, "dK")
    need = grad_workspace_bytes(*d, grad_pass=GRAD_KERNEL_FROM_L)
    workspace, wp, wb = _given_workspace(need, workspace, G)
    _check(lib.mec_wgrad_gemm(_f32(L, "L"), _f32(G, "G"), _f32(dK, "dK"), wp, wb, *d, F32,
                              _stream_handle(stream)), "mec_wgrad_gemm")
    return dK


def conv2d_wgrad(I, G, k_h, k_w, s_h=1, s_w=1, dK=None, workspace=None, stream=None):
    """dK = dloss/dK from I: the products read the rows of L straight from I
    (no lowered copy is made); the workspace holds the partial sums of the
    reduction's shares (grad_workspace_bytes(..., GRAD_KERNEL))."""
    import torch
    if I.dim() != 4 or G.dim() != 4:
        raise ValueError("I must be i_n x i_h x i_w x i_c and G i_n x o_h x o_w x k_c")
    i_n, i_h, i_w, i_c = I.shape
    k_c = G.shape[3]
    o_h, o_w = output_dims(i_h, i_w, k_h, k_w, s_h, s_w)
    if tuple(G.shape) != (i_n, o_h, o_w, k_c):
        raise ValueError("G must be i_n x o_h x o_w x k_c = %s" % ((i_n, o_h, o_w, k_c),))
    _same_device(G, I, "G")
    d = (i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w)
    shape = (k_h, k_w, i_c, k_c)
    if dK is None:
        dK = torch.empty(shape, dtype=torch.float32, device=G.device)
    _check_out(dK, shape, torch.float32, G, "dK")
    need = grad_workspace_bytes(*d, grad_pass=GRAD_KERNEL)
    workspace, wp, wb = _given_workspace(need, workspace, G)
    _check(lib.mec_conv2d_wgrad(_f32(I, "I"), _f32(G, "G"), _f32(dK, "dK"), wp, wb, *d, F32,
                                _stream_handle(stream)), "mec_conv2d_wgrad")
    return dK


def noalloc_scratch_bytes():
    """Bytes of the library's static device scratch (per GPU) that
    conv2d_wgrad_noalloc keeps its partial sums in."""
    return int(lib.mec_noalloc_scratch_bytes())


def conv2d_wgrad_noalloc(I, G, k_h, k_w, s_h=1, s_w=1, dK=None, stream=None):
    """dK = dloss/dK from I, as conv2d_wgrad, with the partial sums in the
    library's static device scratch instead of a workspace: the C call
    allocates nothing (for graph capture and serving loops; the caller passes
    dK). Calls that overlap on one GPU race on the scratch."""
    import torch
    if I.dim() != 4 or G.dim() != 4:
        raise ValueError("I must be i_n x i_h x i_w x i_c and G i_n x o_h x o_w x k_c")
    i_n, i_h, i_w, i_c = I.shape
    k_c = G.shape[3]
    o_h, o_w = output_dims(i_h, i_w, k_h, k_w, s_h, s_w)
    if tuple(G.shape) != (i_n, o_h, o_w, k_c):
        raise ValueError("G must be i_n x o_h x o_w x k_c = %s" % ((i_n, o_h, o_w, k_c),))
    _same_device(G, I, "G")
    shape = (k_h, k_w, i_c, k_c)
    if dK is None:
        dK = torch.empty(shape, dtype=torch.float32, device=G.device)
    _check_out(dK, shape, torch.float32, G, "dK")
    _check(lib.mec_conv2d_wgrad_noalloc(_f32(I, "I"), _f32(G, "G"), _f32(dK, "dK"), i_n, i_h, i_w,
                                        i_c, k_h, k_w, k_c, s_h, s_w, F32, _stream_handle(stream)),
           "mec_conv2d_wgrad_noalloc")
    return dK
