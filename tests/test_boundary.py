"""The C-ABI library on the CPU: it loads, exports every declared symbol, and
its host-side logic (Eq. (1), workspace sizes, argument validation) is right.

No test here launches a kernel: every call either is pure host arithmetic or
fails validation before anything is enqueued (tensor pointers are fake,
never dereferenced).
"""
import ctypes
import os
import re
import subprocess
import sys

import numpy as np
import pytest

import paper_1706_06873_amd as mec
from conftest import REPO

HEADER = os.path.join(REPO, "include", "mec.h")
FAKE = ctypes.c_void_p(0x100000)      # 4 KiB aligned, never dereferenced
ODD = ctypes.c_void_p(0x100002)       # 2-byte aligned only
NULL = ctypes.c_void_p(0)


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mec_\w+)\s*\(", text)))


def test_exports_every_declared_symbol():
    names = declared_functions()
    assert len(names) >= 7
    for name in names:
        assert hasattr(mec.lib, name), name


def test_single_hip_runtime_in_fresh_process():
    """Importing the package first (before torch) still maps one HIP runtime."""
    code = ("import paper_1706_06873_amd as m, torch; torch.cuda.is_available(); "
            "print(len(m._hip_runtimes()))")
    out = subprocess.run([sys.executable, "-c", code], cwd=REPO, capture_output=True, text=True)
    assert out.returncode == 0, out.stderr
    assert out.stdout.strip().splitlines()[-1] == "1"


def test_status_codes_match_header():
    text = open(HEADER).read()
    codes = dict((k, int(v)) for k, v in re.findall(r"(MEC_\w+)\s*=\s*(-?\d+)", text))
    assert codes["MEC_F32"] == mec.F32 and codes["MEC_BF16"] == mec.BF16
    assert codes["MEC_ALGO_LOWERED"] == mec.LOWERED and codes["MEC_ALGO_FUSED"] == mec.FUSED
    assert codes["MEC_ALGO_IM2COL"] == mec.IM2COL
    for name in ("MEC_OK", "MEC_ERR_INVALID_ARG", "MEC_ERR_WORKSPACE", "MEC_ERR_ALIGNMENT",
                 "MEC_ERR_HIP", "MEC_ERR_UNSUPPORTED"):
        msg = mec.strerror(codes[name])
        assert msg and msg != "unknown status"
    assert mec.strerror(12345) == "unknown status"


SHAPES = [
    (1, 7, 7, 1, 3, 3, 1, 1, 1),
    (32, 58, 58, 64, 3, 3, 64, 1, 1),
    (16, 226, 226, 3, 3, 3, 64, 1, 1),
    (128, 227, 227, 3, 11, 11, 96, 4, 4),
    (256, 16, 16, 512, 3, 3, 512, 1, 1),
    (2, 9, 8, 3, 4, 3, 2, 3, 2),
    (1, 224, 224, 64, 7, 7, 64, 2, 2),
    (3, 10, 10, 5, 10, 10, 7, 3, 3),
]


@pytest.mark.parametrize("shape", SHAPES)
def test_sizes_agree_with_oracle(orc, shape):
    nL = orc.lowered_elems(*shape)
    nM = orc.im2col_elems(*shape)
    for dt, es in ((mec.F32, 4), (mec.BF16, 2)):
        assert mec.workspace_bytes(*shape, dtype=dt, algo=mec.LOWERED) == nL * es
        assert mec.workspace_bytes(*shape, dtype=dt, algo=mec.FUSED) == 0
        assert mec.workspace_bytes(*shape, dtype=dt, algo=mec.IM2COL) == nM * es
        assert mec.im2col_bytes(*shape, dtype=dt) == nM * es
    o = mec.output_dims(shape[1], shape[2], shape[4], shape[5], shape[7], shape[8])
    assert o == (orc.out_dim(shape[1], shape[4], shape[7]), orc.out_dim(shape[2], shape[5], shape[8]))


def test_table3_cv4_bytes():
    # cv4 of Table 2 at batch 1: 41.7 / 142.1 MiB in Table 3
    dims = (1, 224, 224, 64, 7, 7, 64, 2, 2)
    assert mec.workspace_bytes(*dims) == 43_753_472
    assert mec.im2col_bytes(*dims) == 149_035_264


def test_workspace_is_exact_for_tiny():
    # no rounding: 105 fp32 elements
    assert mec.workspace_bytes(1, 7, 7, 1, 3, 3, 1, 1, 1) == 420
    assert mec.im2col_bytes(1, 7, 7, 1, 3, 3, 1, 1, 1) == 900


BAD_DIMS = [
    (0, 7, 7, 1, 3, 3, 1, 1, 1),
    (1, 7, 7, 0, 3, 3, 1, 1, 1),
    (1, 7, 7, 1, 8, 3, 1, 1, 1),    # k_h > i_h
    (1, 7, 7, 1, 3, 8, 1, 1, 1),    # k_w > i_w
    (1, 7, 7, 1, 3, 3, 0, 1, 1),
    (1, 7, 7, 1, 3, 3, 1, 0, 1),
    (1, 7, 7, 1, 3, 3, 1, 1, -2),
    (1 << 20, 1 << 11, 1 << 11, 1 << 9, 3, 3, 64, 1, 1),  # too large
]


@pytest.mark.parametrize("dims", BAD_DIMS)
def test_invalid_dims_rejected_everywhere(dims):
    E = -1
    L = mec.lib
    assert L.mec_workspace_bytes(*dims, 0, 0) == E
    assert L.mec_im2col_bytes(*dims, 0) == E
    assert L.mec_lower(FAKE, FAKE, *dims, 0, NULL) == E
    assert L.mec_im2col(FAKE, FAKE, *dims, 0, NULL) == E
    assert L.mec_gemm(FAKE, FAKE, FAKE, *dims, 0, NULL) == E
    assert L.mec_conv2d(FAKE, FAKE, FAKE, FAKE, 1 << 40, *dims, 0, 0, NULL) == E
    assert L.mec_conv2d(FAKE, FAKE, FAKE, NULL, 0, *dims, 0, 1, NULL) == E
    assert L.mec_conv2d(FAKE, FAKE, FAKE, FAKE, 1 << 40, *dims, 0, 2, NULL) == E


def test_output_dims_errors_and_floor():
    o_h, o_w = ctypes.c_int(-7), ctypes.c_int(-7)
    assert mec.lib.mec_output_dims(7, 7, 8, 3, 1, 1, ctypes.byref(o_h), ctypes.byref(o_w)) == -1
    assert o_h.value == -7  # nothing written on error
    assert mec.lib.mec_output_dims(7, 7, 3, 3, 0, 1, None, None) == -1
    assert mec.lib.mec_output_dims(7, 7, 3, 3, 1, 1, None, None) == 0
    assert mec.output_dims(224, 227, 7, 11, 2, 4) == (109, 55)
    assert mec.output_dims(10, 10, 10, 10, 3, 3) == (1, 1)


GOOD = (2, 9, 8, 4, 3, 3, 5, 1, 2)


def test_bad_enums_and_null_pointers():
    L = mec.lib
    assert L.mec_workspace_bytes(*GOOD, 2, 0) == -1
    assert L.mec_workspace_bytes(*GOOD, 0, 3) == -1
    assert L.mec_im2col(NULL, FAKE, *GOOD, 0, NULL) == -1
    assert L.mec_im2col(FAKE, NULL, *GOOD, 0, NULL) == -1
    assert L.mec_im2col(FAKE, FAKE, *GOOD, 2, NULL) == -1
    assert L.mec_im2col_bytes(*GOOD, -1) == -1
    assert L.mec_lower(NULL, FAKE, *GOOD, 0, NULL) == -1
    assert L.mec_lower(FAKE, NULL, *GOOD, 0, NULL) == -1
    assert L.mec_lower(FAKE, FAKE, *GOOD, 3, NULL) == -1
    assert L.mec_gemm(NULL, FAKE, FAKE, *GOOD, 0, NULL) == -1
    assert L.mec_gemm(FAKE, NULL, FAKE, *GOOD, 0, NULL) == -1
    assert L.mec_gemm(FAKE, FAKE, NULL, *GOOD, 0, NULL) == -1
    for bad in ((NULL, FAKE, FAKE), (FAKE, NULL, FAKE), (FAKE, FAKE, NULL)):
        assert L.mec_conv2d(*bad, FAKE, 1 << 30, *GOOD, 0, 0, NULL) == -1
    assert L.mec_conv2d(FAKE, FAKE, FAKE, FAKE, 1 << 30, *GOOD, 0, 7, NULL) == -1
    assert L.mec_conv2d(FAKE, FAKE, FAKE, FAKE, 1 << 30, *GOOD, 5, 0, NULL) == -1


def test_alignment_rejected():
    L = mec.lib
    # fp32 needs 4-byte alignment, bf16 2-byte; O is always fp32
    assert L.mec_lower(ODD, FAKE, *GOOD, 0, NULL) == -3
    assert L.mec_lower(FAKE, ODD, *GOOD, 0, NULL) == -3
    assert L.mec_im2col(ODD, FAKE, *GOOD, 0, NULL) == -3
    assert L.mec_im2col(FAKE, ODD, *GOOD, 0, NULL) == -3
    assert L.mec_gemm(FAKE, FAKE, ODD, *GOOD, 1, NULL) == -3
    assert L.mec_gemm(ODD, FAKE, FAKE, *GOOD, 0, NULL) == -3
    assert L.mec_conv2d(ODD, FAKE, FAKE, FAKE, 1 << 30, *GOOD, 0, 0, NULL) == -3
    assert L.mec_conv2d(FAKE, FAKE, ODD, NULL, 0, *GOOD, 1, 1, NULL) == -3
    assert L.mec_conv2d(FAKE, FAKE, FAKE, ODD, 1 << 30, *GOOD, 0, 0, NULL) == -3


def test_workspace_rejected():
    L = mec.lib
    need = mec.workspace_bytes(*GOOD)
    assert L.mec_conv2d(FAKE, FAKE, FAKE, NULL, need, *GOOD, 0, 0, NULL) == -2
    assert L.mec_conv2d(FAKE, FAKE, FAKE, FAKE, need - 1, *GOOD, 0, 0, NULL) == -2
    need16 = mec.workspace_bytes(*GOOD, dtype=mec.BF16)
    assert need16 * 2 == need
    assert L.mec_conv2d(FAKE, FAKE, FAKE, FAKE, need16 - 2, *GOOD, 1, 0, NULL) == -2
    # the im2col baseline needs the (larger) im2col matrix as workspace
    needM = mec.workspace_bytes(*GOOD, algo=mec.IM2COL)
    assert needM == mec.im2col_bytes(*GOOD) > need
    assert L.mec_conv2d(FAKE, FAKE, FAKE, FAKE, needM - 4, *GOOD, 0, 2, NULL) == -2
    assert L.mec_conv2d(FAKE, FAKE, FAKE, NULL, needM, *GOOD, 0, 2, NULL) == -2


def test_unsupported_kernel_height():
    # far taller than the fused form's on-chip tiles hold: refused before any
    # launch (from L, the flat windows take every height, so this shape is not
    # called there with these stand-in pointers)
    dims = (1, 300, 8, 1, 300, 3, 1, 1, 1)
    assert mec.lib.mec_conv2d(FAKE, FAKE, FAKE, NULL, 0, *dims, 0, 1, NULL) == -5
    assert mec.workspace_bytes(*dims) == 1 * 6 * 300 * 3 * 4


def test_python_binding_raises():
    with pytest.raises(mec.MecError) as ei:
        mec.workspace_bytes(1, 7, 7, 1, 8, 3, 1, 1, 1)
    assert ei.value.status == -1


def test_fastdiv_exhaustive_cpu(tmp_path):
    """The kernels' division by invariant integers, checked on the host against
    '/' for many divisors and dividends up to 2^31 - 1."""
    src = tmp_path / "fd.cpp"
    src.write_text(r'''
#include <cstdio>
#include <cstdint>
#include <random>
#define MEC_HD
#include "mec_internal.h"
int main() {
    std::mt19937_64 rng(1);
    uint64_t bad = 0, n = 0;
    auto check = [&](uint32_t d, uint32_t x) {
        mec::FastDiv f(d);
        ++n;
        if (f.div(x) != x / d) { if (bad < 5) printf("d=%u x=%u\n", d, x); ++bad; }
    };
    const uint32_t top = 0x7fffffffu;
    for (uint32_t d = 1; d < 70000; ++d) {
        for (uint32_t x : {0u, 1u, d - 1, d, d + 1, 2 * d - 1, 2 * d, top, top - 1, top - d})
            if (x <= top) check(d, x);
        for (int k = 0; k < 16; ++k) check(d, (uint32_t)(rng() & top));
        uint32_t q = top / d;
        check(d, q * d); check(d, q * d - 1 < top ? q * d - 1 : 0);
    }
    for (int k = 0; k < 2000000; ++k) {
        uint32_t d = (uint32_t)(rng() % top) + 1, x = (uint32_t)(rng() & top);
        check(d, x);
        if (x >= d) check(d, (x / d) * d);
    }
    for (int b = 0; b < 31; ++b) {
        for (uint32_t d : {1u << b, (1u << b) + 1, (1u << b) - 1}) {
            if (!d) continue;
            for (int k = 0; k < 2000; ++k) check(d, (uint32_t)(rng() & top));
            check(d, top);
        }
    }
    printf("%llu checks, %llu wrong\n", (unsigned long long)n, (unsigned long long)bad);
    return bad != 0;
}
''')
    exe = tmp_path / "fd"
    subprocess.run(["g++", "-O2", "-std=c++17", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
                    "-I", os.path.join(REPO, "paper_1706_06873_amd", "csrc"), str(src), "-o",
                    str(exe)], check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True)
    assert out.returncode == 0, out.stdout
    assert " 0 wrong" in out.stdout


# ---------------------------------------------------------------- training passes

def test_grad_enums_match_header():
    text = open(HEADER).read()
    codes = dict((k, int(v)) for k, v in re.findall(r"(MEC_\w+)\s*=\s*(-?\d+)", text))
    assert codes["MEC_GRAD_INPUT"] == mec.GRAD_INPUT
    assert codes["MEC_GRAD_KERNEL"] == mec.GRAD_KERNEL
    assert codes["MEC_GRAD_KERNEL_FROM_L"] == mec.GRAD_KERNEL_FROM_L


GRAD_SHAPES = SHAPES + [
    (2, 17, 15, 32, 3, 3, 40, 2, 2),    # 3x3 s2: phases too small, dL path
    (2, 21, 19, 32, 7, 7, 36, 2, 2),    # 7x7 s2: phases of 4x4 .. 3x3 taps
    (2, 21, 20, 32, 7, 5, 36, 2, 1),    # 7x5, strides 2 and 1
    (2, 19, 18, 32, 5, 5, 40, 1, 2),    # 5x5, strides 1 and 2
    (2, 15, 16, 32, 3, 5, 16, 2, 3),    # unequal strides, too small
    (2, 23, 23, 64, 11, 11, 64, 2, 2),  # phase kernels of 6 rows: dL path
    (2, 17, 15, 32, 3, 3, 42, 2, 2),    # k_c not a multiple of 4: dL path
    (2, 17, 15, 32, 1, 1, 40, 2, 2),    # s > k: dL path
    (2, 17, 15, 32, 5, 5, 40, 1, 1),    # stride 1, 5x5: dL path
]


@pytest.mark.parametrize("shape", GRAD_SHAPES)
def test_grad_workspace_sizes(orc, shape):
    nL = orc.lowered_elems(*shape)
    i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w = shape
    if i_n * i_h * i_w * i_c >= 2 ** 31:
        assert mec.lib.mec_grad_workspace_bytes(*shape, 0, 0) == -5
        return
    # dI: dL in fp32, exactly |L| * 4; or, on the sub-pixel phase path, 12 bytes of
    # alignment slack, the largest phase's padded G (rounded up to 256 bytes) and the
    # largest phase kernel
    wi = mec.grad_workspace_bytes(*shape, grad_pass=mec.GRAD_INPUT)
    expect = dgrad_phase_workspace(shape)
    assert wi == (expect if expect is not None else nL * 4)
    # dK: whole partial-sum buffers of k_h*k_w*i_c*k_c floats, 1..1024 of them
    part = mec.grad_workspace_bytes(*shape, grad_pass=mec.GRAD_KERNEL_FROM_L)
    E = k_h * k_w * i_c * k_c * 4
    assert part % E == 0 and 1 <= part // E <= 1024
    # from I: the rows of L are read from I, so the partial sums only
    assert mec.grad_workspace_bytes(*shape, grad_pass=mec.GRAD_KERNEL) == part


def dgrad_phase_workspace(shape):
    """Workspace of the sub-pixel phase path for this shape, or None where the
    library takes the dL path (its stated rule)."""
    i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w = shape
    unit = s_h == s_w == 1
    if i_c < 32 or (unit and (k_h > 3 or k_w > 3)):
        return None
    if not unit and (s_h > k_h or s_w > k_w or k_c % 4 or i_c % 4 or -(-k_h // s_h) > 5):
        return None
    if not unit and (k_h * k_w < 10 * s_h * s_w or s_h * s_w > 4):
        return None
    gp = kp = 0
    for py in range(s_h):
        for px in range(s_w):
            J, I = -(-(k_h - py) // s_h), -(-(k_w - px) // s_w)
            Ny, Nx = -(-(i_h - py) // s_h), -(-(i_w - px) // s_w)
            gp = max(gp, i_n * (Ny + J - 1) * (Nx + I - 1) * k_c)
            kp = max(kp, J * I * k_c * i_c)
    if unit:  # one phase: G padded by k - 1 on every side
        o_h, o_w = i_h - k_h + 1, i_w - k_w + 1
        assert gp == i_n * (o_h + 2 * (k_h - 1)) * (o_w + 2 * (k_w - 1)) * k_c
    return 12 + (gp * 4 + 255) // 256 * 256 + kp * 4


def test_grad_rejects_bf16_and_bad_pass():
    L = mec.lib
    assert L.mec_grad_workspace_bytes(*GOOD, 1, 0) == -5
    assert L.mec_grad_workspace_bytes(*GOOD, 2, 0) == -1
    assert L.mec_grad_workspace_bytes(*GOOD, 0, 3) == -1
    assert L.mec_dgrad_gemm(FAKE, FAKE, FAKE, *GOOD, 1, NULL) == -5
    assert L.mec_conv2d_dgrad(FAKE, FAKE, FAKE, FAKE, 1 << 30, *GOOD, 1, NULL) == -5
    assert L.mec_wgrad_gemm(FAKE, FAKE, FAKE, FAKE, 1 << 30, *GOOD, 1, NULL) == -5
    assert L.mec_conv2d_wgrad(FAKE, FAKE, FAKE, FAKE, 1 << 30, *GOOD, 1, NULL) == -5


@pytest.mark.parametrize("dims", BAD_DIMS)
def test_grad_invalid_dims(dims):
    L = mec.lib
    assert L.mec_grad_workspace_bytes(*dims, 0, 0) == -1
    assert L.mec_fold(FAKE, FAKE, *dims, NULL) == -1
    assert L.mec_dgrad_gemm(FAKE, FAKE, FAKE, *dims, 0, NULL) == -1
    assert L.mec_conv2d_dgrad(FAKE, FAKE, FAKE, FAKE, 1 << 40, *dims, 0, NULL) == -1
    assert L.mec_wgrad_gemm(FAKE, FAKE, FAKE, FAKE, 1 << 40, *dims, 0, NULL) == -1
    assert L.mec_conv2d_wgrad(FAKE, FAKE, FAKE, FAKE, 1 << 40, *dims, 0, NULL) == -1


def test_grad_null_alignment_and_workspace():
    L = mec.lib
    big = 1 << 30
    assert L.mec_fold(NULL, FAKE, *GOOD, NULL) == -1
    assert L.mec_fold(FAKE, NULL, *GOOD, NULL) == -1
    assert L.mec_fold(ODD, FAKE, *GOOD, NULL) == -3
    for bad in ((NULL, FAKE, FAKE), (FAKE, NULL, FAKE), (FAKE, FAKE, NULL)):
        assert L.mec_dgrad_gemm(*bad, *GOOD, 0, NULL) == -1
        assert L.mec_conv2d_dgrad(*bad, FAKE, big, *GOOD, 0, NULL) == -1
        assert L.mec_wgrad_gemm(*bad, FAKE, big, *GOOD, 0, NULL) == -1
        assert L.mec_conv2d_wgrad(*bad, FAKE, big, *GOOD, 0, NULL) == -1
    assert L.mec_dgrad_gemm(FAKE, ODD, FAKE, *GOOD, 0, NULL) == -3
    assert L.mec_conv2d_dgrad(FAKE, FAKE, ODD, FAKE, big, *GOOD, 0, NULL) == -3
    assert L.mec_wgrad_gemm(ODD, FAKE, FAKE, FAKE, big, *GOOD, 0, NULL) == -3
    assert L.mec_conv2d_wgrad(FAKE, FAKE, FAKE, ODD, big, *GOOD, 0, NULL) == -3
    need_i = mec.grad_workspace_bytes(*GOOD, grad_pass=mec.GRAD_INPUT)
    need_k = mec.grad_workspace_bytes(*GOOD, grad_pass=mec.GRAD_KERNEL)
    need_l = mec.grad_workspace_bytes(*GOOD, grad_pass=mec.GRAD_KERNEL_FROM_L)
    assert L.mec_conv2d_dgrad(FAKE, FAKE, FAKE, FAKE, need_i - 4, *GOOD, 0, NULL) == -2
    assert L.mec_conv2d_dgrad(FAKE, FAKE, FAKE, NULL, need_i, *GOOD, 0, NULL) == -2
    assert L.mec_conv2d_wgrad(FAKE, FAKE, FAKE, FAKE, need_k - 4, *GOOD, 0, NULL) == -2
    assert L.mec_wgrad_gemm(FAKE, FAKE, FAKE, FAKE, need_l - 4, *GOOD, 0, NULL) == -2
    assert L.mec_wgrad_gemm(FAKE, FAKE, FAKE, NULL, need_l, *GOOD, 0, NULL) == -2


# ---------------------------------------------------------------- binding validation
# Caller-supplied outputs and operands that do not match the shape must be
# refused by the binding before any library entry point that launches work is
# called. CPU tensors stand in for device ones: every check below runs before
# the binding takes a device pointer.

LAUNCHERS = ("mec_lower", "mec_im2col", "mec_gemm", "mec_conv2d", "mec_fold", "mec_dgrad_gemm",
             "mec_conv2d_dgrad", "mec_wgrad_gemm", "mec_conv2d_wgrad")


@pytest.fixture
def no_launch(monkeypatch):
    def refuse(*a, **k):
        raise AssertionError("a launching entry point was called")
    for name in LAUNCHERS:
        monkeypatch.setattr(mec.lib, name, refuse)
    return mec


def _t(*shape, dtype=None):
    import torch
    return torch.zeros(shape, dtype=dtype or torch.float32)


def test_binding_refuses_mismatched_operands(no_launch):
    import torch
    m = no_launch
    d = (2, 9, 8, 4, 3, 3, 5, 1, 1)     # i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w
    I, K = _t(2, 9, 8, 4), _t(3, 3, 4, 5)
    L = _t(2, 6, 9, 3, 4)                 # o_w = 6
    O = _t(2, 7, 6, 5)
    # gemm: K must agree with L on k_w and i_c, and share its dtype
    with pytest.raises(ValueError, match="do not agree"):
        m.gemm(L, _t(3, 2, 4, 5), 9, 8, 1, 1, O=O)
    with pytest.raises(ValueError, match="do not agree"):
        m.gemm(L, _t(3, 3, 3, 5), 9, 8, 1, 1, O=O)
    with pytest.raises(TypeError, match="same dtype"):
        m.gemm(L, _t(3, 3, 4, 5, dtype=torch.bfloat16), 9, 8, 1, 1, O=O)
    # a given O of the wrong shape or dtype
    for bad in (_t(2, 7, 6, 4), _t(2, 7, 6, 5, dtype=torch.float64), _t(2 * 7 * 6 * 5)):
        with pytest.raises(ValueError, match="O must be"):
            m.gemm(L, K, 9, 8, 1, 1, O=bad)
        with pytest.raises(ValueError, match="O must be"):
            m.conv2d(I, K, 1, 1, algo="fused", O=bad)
    # a workspace smaller than the library asks for
    need = m.workspace_bytes(*d)
    with pytest.raises(ValueError, match="workspace holds"):
        m.conv2d(I, K, 1, 1, algo="lowered", O=O, workspace=_t(need - 1, dtype=torch.uint8))
    # L and M of the wrong byte size or dtype
    with pytest.raises(ValueError, match="L must hold"):
        m.lower(I, 3, 3, 5, 1, 1, L=_t(L.numel() - 1))
    with pytest.raises(ValueError, match="L must hold"):
        m.lower(I, 3, 3, 5, 1, 1, L=_t(*L.shape, dtype=torch.bfloat16))
    with pytest.raises(ValueError, match="M must hold"):
        m.im2col(I, 3, 3, 5, 1, 1, M=_t(7))


def test_binding_refuses_mismatched_gradients(no_launch):
    import torch
    m = no_launch
    d = (2, 9, 8, 4, 3, 3, 5, 1, 1)
    I, K, G = _t(2, 9, 8, 4), _t(3, 3, 4, 5), _t(2, 7, 6, 5)
    L = _t(2, 6, 9, 3, 4)
    with pytest.raises(ValueError, match="G must be"):
        m.conv2d_dgrad(_t(2, 7, 5, 5), K, 9, 8)
    for bad in (_t(2, 9, 8, 3), _t(2, 9, 8, 4, dtype=torch.float64)):
        with pytest.raises(ValueError, match="dI must be"):
            m.conv2d_dgrad(G, K, 9, 8, dI=bad)
        with pytest.raises(ValueError, match="dI must be"):
            m.fold(_t(2, 6, 9, 3, 4), 8, 1, dI=bad)
    with pytest.raises(ValueError, match="dL must be"):
        m.dgrad_gemm(G, K, 9, 8, dL=_t(2, 6, 9, 3, 3))
    for bad in (_t(3, 3, 4, 4), _t(3, 3, 4, 5, dtype=torch.bfloat16)):
        with pytest.raises(ValueError, match="dK must be"):
            m.wgrad_gemm(L, G, 3, 8, dK=bad)
        with pytest.raises(ValueError, match="dK must be"):
            m.conv2d_wgrad(I, G, 3, 3, dK=bad)
    need = m.grad_workspace_bytes(*d, grad_pass=m.GRAD_KERNEL)
    with pytest.raises(ValueError, match="workspace holds"):
        m.conv2d_wgrad(I, G, 3, 3, workspace=_t(max(need - 4, 0), dtype=torch.uint8))
    need = m.grad_workspace_bytes(*d, grad_pass=m.GRAD_INPUT)
    with pytest.raises(ValueError, match="workspace holds"):
        m.conv2d_dgrad(G, K, 9, 8, workspace=_t(max(need - 4, 0), dtype=torch.uint8))
