"""Parity of the training passes (HIP, through the C ABI) with the CPU oracle.

Bars as for the forward pass: with small-integer inputs every partial sum is
exact in fp32, so dL, dI and dK must match the oracle bit for bit; with
uniform random inputs they must be within relative L2 error 1e-5.
"""
import numpy as np
import pytest
import torch

import paper_1706_06873_amd as mec
from paper_1706_06873_amd import workloads as wl

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
TOL = 1e-5

SHAPES = [
    # i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w
    (1, 7, 7, 1, 3, 3, 1, 1, 1),
    (2, 9, 8, 3, 3, 2, 4, 1, 1),
    (2, 11, 10, 2, 3, 3, 3, 2, 3),      # strides not dividing i - k
    (1, 10, 9, 2, 2, 2, 2, 3, 4),       # s > k: rows and columns no window covers
    (3, 6, 5, 4, 6, 5, 2, 1, 1),        # k = i
    (2, 8, 8, 5, 1, 1, 3, 1, 1),        # 1x1
    (2, 19, 17, 16, 3, 3, 40, 1, 1),    # 4-channel vectors, ragged channel tiles
    (3, 31, 30, 3, 11, 11, 96, 4, 4),   # 11x11 stride 4
    (1, 40, 9, 1, 13, 3, 7, 9, 1),      # one LDS stage (no double buffer)
    (1, 30, 9, 2, 20, 3, 5, 1, 1),      # tall kernel: 2-channel chunks
    (35, 5, 5, 2, 2, 2, 3, 1, 1),       # pairs over several 32-pair tiles
    (8, 16, 16, 64, 3, 3, 130, 1, 1),   # dK tiles ragged in both directions
    (4, 21, 19, 16, 7, 7, 40, 2, 2),    # 7x7 stride 2
    (3, 12, 11, 16, 3, 3, 70, 1, 1),    # slab wgrad, ragged channel tiles
    (2, 15, 15, 16, 5, 5, 8, 1, 2),     # slab wgrad, 5x5
    (3, 9, 9, 64, 1, 1, 40, 1, 1),      # slab wgrad, 1x1
    (2, 13, 13, 64, 3, 3, 64, 3, 2),    # stride 3: too many staged rows for the slab wgrad
    (2, 13, 13, 48, 1, 1, 64, 2, 2),    # slab wgrad, 1x1 stride 2
    (3, 10, 11, 64, 3, 3, 32, 1, 1),    # dI as a convolution of the padded G (i_c >= 32)
    (2, 12, 12, 40, 3, 2, 24, 1, 1),    # the same, 3x2, ragged channels
    (2, 9, 9, 32, 1, 1, 8, 1, 1),       # the same, 1x1
    (2, 21, 19, 32, 7, 7, 36, 2, 2),    # dI as sub-pixel phases: 7x7 s2 (4x4 .. 3x3 taps)
    (2, 21, 20, 32, 7, 5, 36, 2, 1),    # 7x5, strides 2 and 1 (4x5 and 3x5 taps)
    (2, 19, 18, 32, 5, 5, 40, 1, 2),    # 5x5, strides 1 and 2 (5x3 and 5x2 taps)
    (2, 17, 15, 32, 3, 3, 40, 2, 2),    # 3x3 s2: phases too small, dL path
    (2, 13, 12, 32, 5, 5, 24, 2, 2),    # 5x5 s2: dL path
    (1, 30, 31, 32, 11, 11, 32, 4, 4),  # 11x11 s4: sixteen phases, dL path
]


def say(*a):
    print("[case]", *a, flush=True)


def rel_l2(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.linalg.norm(ref)
    return np.linalg.norm(got - ref) / (den if den > 0 else 1.0)


def problem(seed, d, dist):
    i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w = d
    o_h, o_w = mec.output_dims(i_h, i_w, k_h, k_w, s_h, s_w)
    I, K = wl.random_case(seed, *d, dist=dist)
    g = torch.Generator().manual_seed(seed + 1)
    if dist == "int":
        G = torch.randint(-3, 4, (i_n, o_h, o_w, k_c), generator=g).float()
    else:
        G = torch.rand((i_n, o_h, o_w, k_c), generator=g) * 2 - 1
    return I, K, G


def last_phase_padded_g(G, d):
    """G zero-padded as the library pads it for its last sub-pixel phase
    (py, px) = (s_h - 1, s_w - 1): J - 1 rows above, I - 1 columns left,
    Ny + J - 1 rows and Nx + I - 1 columns in all."""
    i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w = d
    py, px = s_h - 1, s_w - 1
    J, I = -(-(k_h - py) // s_h), -(-(k_w - px) // s_w)
    Ny, Nx = -(-(i_h - py) // s_h), -(-(i_w - px) // s_w)
    out = np.zeros((G.shape[0], Ny + J - 1, Nx + I - 1, G.shape[3]), np.float32)
    rows, cols = min(G.shape[1], Ny), min(G.shape[2], Nx)
    out[:, J - 1:J - 1 + rows, I - 1:I - 1 + cols] = G[:, :rows, :cols]
    return out


@pytest.mark.parametrize("d", [(2, 21, 19, 32, 7, 7, 36, 2, 2), (3, 10, 11, 64, 3, 3, 32, 1, 1)])
def test_dgrad_phases_unaligned_workspace(orc, d):
    """The phase path with a workspace that is only 4-byte aligned."""
    say("dgrad unaligned ws", d)
    I, K, G = problem(47 + sum(d), d, "int")
    i_h, i_w, s_h, s_w = d[1], d[2], d[7], d[8]
    ref = orc.conv2d_dgrad(G.numpy(), K.numpy(), i_h, i_w, s_h, s_w)
    need = mec.grad_workspace_bytes(*d)
    ws = torch.zeros(need + 4, dtype=torch.uint8, device=DEV)[4:]
    dI = mec.conv2d_dgrad(G.to(DEV), K.to(DEV), i_h, i_w, s_h, s_w, workspace=ws)
    torch.cuda.synchronize()
    assert np.array_equal(dI.cpu().numpy(), ref.astype(np.float32))


@pytest.mark.parametrize("d", [(2, 21, 19, 32, 7, 7, 36, 2, 2), (2, 19, 18, 32, 5, 5, 40, 1, 2),
                               (3, 10, 11, 64, 3, 3, 32, 1, 1)])
def test_dgrad_phases_unaligned_g_and_di(orc, d):
    """The phase path with G and dI one element off a 16-byte boundary: element
    padding of G and element stores into the phase's pixels; nothing written
    outside dI."""
    say("dgrad unaligned G/dI", d)
    I, K, G = problem(53 + sum(d), d, "int")
    i_n, i_h, i_w, i_c, s_h, s_w = d[0], d[1], d[2], d[3], d[7], d[8]
    ref = orc.conv2d_dgrad(G.numpy(), K.numpy(), i_h, i_w, s_h, s_w).astype(np.float32)
    gbuf = torch.zeros(G.numel() + 8, device=DEV)
    Gd = gbuf[1:1 + G.numel()].view(G.shape)
    Gd.copy_(G.to(DEV))
    obuf = torch.full((ref.size + 64,), 7.0, device=DEV)
    dI = obuf[33:33 + ref.size].view(ref.shape)
    mec.conv2d_dgrad(Gd, K.to(DEV), i_h, i_w, s_h, s_w, dI=dI)
    torch.cuda.synchronize()
    b = obuf.cpu().numpy()
    assert np.all(b[:33] == 7.0) and np.all(b[33 + ref.size:] == 7.0)
    assert np.array_equal(dI.cpu().numpy(), ref)


@pytest.mark.parametrize("d", SHAPES)
@pytest.mark.parametrize("dist", ["int", "u11"])
def test_dgrad(orc, d, dist):
    say("dgrad", dist, d)
    I, K, G = problem(41 + sum(d), d, dist)
    i_h, i_w, s_h, s_w = d[1], d[2], d[7], d[8]
    ref_dL = orc.mec_dgrad_lowered(G.numpy(), K.numpy(), i_h, i_w, s_h, s_w)
    ref_dI = orc.conv2d_dgrad(G.numpy(), K.numpy(), i_h, i_w, s_h, s_w)
    Gd, Kd = G.to(DEV), K.to(DEV)
    dL = mec.dgrad_gemm(Gd, Kd, i_h, i_w, s_h, s_w)
    ws = torch.full((mec.grad_workspace_bytes(*d),), 0xFF, dtype=torch.uint8, device=DEV)
    dI = mec.conv2d_dgrad(Gd, Kd, i_h, i_w, s_h, s_w, workspace=ws)
    torch.cuda.synchronize()
    dL, dI = dL.cpu().numpy(), dI.cpu().numpy()
    wsf = ws.cpu().numpy().view(np.float32)
    if wsf.size == ref_dL.size:
        # the dL path: the workspace holds dL
        assert np.array_equal(wsf.reshape(ref_dL.shape), dL)
    else:
        # sub-pixel phases: the workspace starts with the last phase's padded G
        # (stride 1: the only phase, G zero-padded by k - 1 on every side)
        Gp = last_phase_padded_g(G.numpy(), d)
        assert np.array_equal(wsf[:Gp.size].reshape(Gp.shape), Gp)
    if dist == "int":
        assert np.array_equal(dL, ref_dL.astype(np.float32))
        assert np.array_equal(dI, ref_dI.astype(np.float32))
    else:
        assert rel_l2(dL, ref_dL) <= TOL
        assert rel_l2(dI, ref_dI) <= TOL


@pytest.mark.parametrize("d", SHAPES)
@pytest.mark.parametrize("dist", ["int", "u11"])
def test_wgrad(orc, d, dist):
    say("wgrad", dist, d)
    I, K, G = problem(43 + sum(d), d, dist)
    k_h, k_w, s_h, s_w = d[4], d[5], d[7], d[8]
    ref = orc.conv2d_wgrad(I.numpy(), G.numpy(), k_h, k_w, s_h, s_w)
    Id, Gd = I.to(DEV), G.to(DEV)
    dK = mec.conv2d_wgrad(Id, Gd, k_h, k_w, s_h, s_w)
    L = mec.lower(Id, k_h, k_w, d[6], s_h, s_w)
    dK2 = mec.wgrad_gemm(L, Gd, k_h, d[2], s_h, s_w)
    torch.cuda.synchronize()
    dK, dK2 = dK.cpu().numpy(), dK2.cpu().numpy()
    assert np.array_equal(dK, dK2)
    if dist == "int":
        assert np.abs(ref).max() < 2 ** 24
        assert np.array_equal(dK, ref.astype(np.float32))
    else:
        assert rel_l2(dK, ref) <= TOL


@pytest.mark.parametrize("d", SHAPES[:8])
def test_fold(orc, d):
    """The fold of a random dL (not one produced by the products)."""
    say("fold", d)
    i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w = d
    _, o_w = mec.output_dims(i_h, i_w, k_h, k_w, s_h, s_w)
    g = torch.Generator().manual_seed(sum(d))
    for dist in ("int", "u11"):
        if dist == "int":
            dL = torch.randint(-5, 6, (i_n, o_w, i_h, k_w, i_c), generator=g).float()
        else:
            dL = torch.rand((i_n, o_w, i_h, k_w, i_c), generator=g) * 2 - 1
        ref = orc.mec_fold(dL.numpy(), i_w, s_w)
        got = mec.fold(dL.to(DEV), i_w, s_w)
        torch.cuda.synchronize()
        got = got.cpu().numpy()
        if dist == "int":
            assert np.array_equal(got, ref.astype(np.float32))
        else:
            assert rel_l2(got, ref) <= 1e-6


def test_wgrad_reuses_forward_workspace(orc):
    """After a LOWERED forward pass the workspace holds L; the weight gradient
    can be taken from it without lowering again."""
    d = (4, 20, 19, 8, 3, 3, 16, 1, 2)
    say("wgrad from forward workspace", d)
    I, K, G = problem(77, d, "int")
    Id, Kd, Gd = I.to(DEV), K.to(DEV), G.to(DEV)
    ws = torch.empty(mec.workspace_bytes(*d), dtype=torch.uint8, device=DEV)
    mec.conv2d(Id, Kd, d[7], d[8], algo="lowered", workspace=ws)
    i_n, i_h, i_w, i_c, k_h, k_w = d[:6]
    _, o_w = mec.output_dims(i_h, i_w, k_h, k_w, d[7], d[8])
    L = ws.view(torch.float32).view(i_n, o_w, i_h, k_w, i_c)
    dK = mec.wgrad_gemm(L, Gd, k_h, i_w, d[7], d[8])
    torch.cuda.synchronize()
    ref = orc.conv2d_wgrad(I.numpy(), G.numpy(), k_h, k_w, d[7], d[8])
    assert np.array_equal(dK.cpu().numpy(), ref.astype(np.float32))


@pytest.mark.parametrize("d", [(2, 13, 12, 8, 3, 3, 12, 1, 1), (2, 13, 12, 16, 3, 3, 12, 1, 1)])
def test_unaligned_training_tensors(orc, d):
    """Tensors 4 bytes past a 16-byte boundary take the element-wise loads."""
    say("unaligned training", d)
    I, K, G = problem(5, d, "int")
    i_h, i_w, k_h, k_w = d[1], d[2], d[4], d[5]

    def off(t):
        buf = torch.zeros(t.numel() + 4, dtype=torch.float32, device=DEV)
        v = buf[1:1 + t.numel()].view(t.shape)
        v.copy_(t.to(DEV))
        return v

    Id, Kd, Gd = off(I), off(K), off(G)
    dI = torch.zeros(I.numel() + 4, device=DEV)[1:1 + I.numel()].view(I.shape)
    dK = torch.zeros(K.numel() + 4, device=DEV)[1:1 + K.numel()].view(K.shape)
    wsI = torch.zeros(mec.grad_workspace_bytes(*d) + 64, dtype=torch.uint8, device=DEV)[4:]
    wsK = torch.zeros(mec.grad_workspace_bytes(*d, grad_pass=mec.GRAD_KERNEL) + 64,
                      dtype=torch.uint8, device=DEV)[4:]
    mec.conv2d_dgrad(Gd, Kd, i_h, i_w, 1, 1, dI=dI, workspace=wsI)
    mec.conv2d_wgrad(Id, Gd, k_h, k_w, 1, 1, dK=dK, workspace=wsK)
    torch.cuda.synchronize()
    assert np.array_equal(dI.cpu().numpy(),
                          orc.conv2d_dgrad(G.numpy(), K.numpy(), i_h, i_w, 1, 1).astype(np.float32))
    assert np.array_equal(dK.cpu().numpy(),
                          orc.conv2d_wgrad(I.numpy(), G.numpy(), k_h, k_w, 1, 1).astype(np.float32))


def test_resnet_mid_full_size(orc):
    """Both gradients at the full resnet_mid layer (batch 32, 58x58x64 input,
    3x3x64x64 kernel), against the whole oracle result."""
    layer = wl.LAYERS["resnet_mid"]
    d = layer.dims
    say("training resnet_mid full", d)
    I, K = wl.make_inputs(layer)
    i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w = d
    o_h, o_w = mec.output_dims(i_h, i_w, k_h, k_w, s_h, s_w)
    G = torch.rand((i_n, o_h, o_w, k_c), generator=torch.Generator().manual_seed(1001)) * 2 - 1
    Id, Kd, Gd = I.to(DEV), K.to(DEV), G.to(DEV)
    dI = mec.conv2d_dgrad(Gd, Kd, i_h, i_w, s_h, s_w)
    dK = mec.conv2d_wgrad(Id, Gd, k_h, k_w, s_h, s_w)
    torch.cuda.synchronize()
    assert rel_l2(dI.cpu().numpy(), orc.conv2d_dgrad(G.numpy(), K.numpy(), i_h, i_w, s_h, s_w)) <= TOL
    assert rel_l2(dK.cpu().numpy(), orc.conv2d_wgrad(I.numpy(), G.numpy(), k_h, k_w, s_h, s_w)) <= TOL
