"""Pins for the oracle's training passes (gradients of the convolution).

The paper gives no backward algorithm, so the gradients are pinned by what
mathematics fixes, never by re-typing the oracle's loops:
  * adjointness: <conv(I, K), G> = <I, dgrad(G, K)> = <K, wgrad(I, G)>, exact
    on small integers, which ties both gradients to the already pinned forward;
  * the pure-Python brute force, which builds each gradient entry from the
    forward convolution of a basis image or basis kernel (linearity);
  * torch's CPU autograd of conv2d in fp64 (a library routine);
  * closed forms of the 7x7 worked example and of delta gradients;
  * the MEC forms (slab adjoint + fold, sum of A_h^T G_h) against the direct
    forms, and the fold as the adjoint of the lowering.
"""
import numpy as np
import pytest
import torch

from oracle import brute

F32 = np.float32

SHAPES = [
    # i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w
    (1, 7, 7, 1, 3, 3, 1, 1, 1),
    (2, 9, 8, 3, 3, 2, 4, 1, 1),
    (2, 11, 10, 2, 3, 3, 3, 2, 3),    # strides not dividing i - k
    (1, 10, 9, 2, 2, 2, 2, 3, 4),     # s > k: pixels no window covers
    (3, 6, 5, 4, 6, 5, 2, 1, 1),      # k = i
    (1, 13, 12, 3, 5, 4, 5, 2, 2),
    (2, 8, 8, 5, 1, 1, 3, 1, 1),      # 1x1
]


def ints(rng, shape):
    return rng.integers(-3, 4, size=shape).astype(F32)


def out_hw(d):
    i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w = d
    return (i_h - k_h) // s_h + 1, (i_w - k_w) // s_w + 1


def rand_problem(seed, d):
    rng = np.random.default_rng(seed)
    i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w = d
    o_h, o_w = out_hw(d)
    return (ints(rng, (i_n, i_h, i_w, i_c)), ints(rng, (k_h, k_w, i_c, k_c)),
            ints(rng, (i_n, o_h, o_w, k_c)))


@pytest.mark.parametrize("d", SHAPES)
def test_adjoint_identities_exact(orc, d):
    I, K, G = rand_problem(sum(d), d)
    s_h, s_w = d[7], d[8]
    O = orc.conv2d_direct(I, K, s_h, s_w)
    dI = orc.conv2d_dgrad(G, K, d[1], d[2], s_h, s_w)
    dK = orc.conv2d_wgrad(I, G, d[4], d[5], s_h, s_w)
    lhs = float(np.sum(O * G.astype(np.float64)))
    assert lhs == float(np.sum(I.astype(np.float64) * dI))
    assert lhs == float(np.sum(K.astype(np.float64) * dK))


@pytest.mark.parametrize("d", [
    (1, 5, 5, 1, 3, 3, 1, 1, 1),
    (2, 5, 6, 2, 2, 3, 2, 2, 1),
    (1, 6, 5, 1, 2, 2, 3, 3, 2),
    (1, 4, 4, 2, 4, 4, 1, 1, 1),
])
def test_brute_force_by_linearity(orc, d):
    I, K, G = rand_problem(7 * sum(d), d)
    s_h, s_w = d[7], d[8]
    bI = np.array(brute.dgrad(G.astype(int).tolist(), K.astype(int).tolist(), d[1], d[2], s_h, s_w))
    bK = np.array(brute.wgrad(I.astype(int).tolist(), G.astype(int).tolist(), d[4], d[5], s_h, s_w))
    assert np.array_equal(orc.conv2d_dgrad(G, K, d[1], d[2], s_h, s_w), bI)
    assert np.array_equal(orc.conv2d_wgrad(I, G, d[4], d[5], s_h, s_w), bK)


@pytest.mark.parametrize("d", SHAPES + [(4, 20, 19, 8, 3, 3, 16, 1, 1), (2, 31, 30, 3, 11, 11, 8, 4, 4)])
def test_torch_autograd_fp64(orc, d):
    rng = np.random.default_rng(3 * sum(d))
    i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w = d
    o_h, o_w = out_hw(d)
    I = rng.uniform(-1, 1, (i_n, i_h, i_w, i_c)).astype(F32)
    K = rng.uniform(-1, 1, (k_h, k_w, i_c, k_c)).astype(F32)
    G = rng.uniform(-1, 1, (i_n, o_h, o_w, k_c)).astype(F32)
    x = torch.from_numpy(I.astype(np.float64)).permute(0, 3, 1, 2).requires_grad_()
    w = torch.from_numpy(K.astype(np.float64)).permute(3, 2, 0, 1).detach().requires_grad_()
    y = torch.nn.functional.conv2d(x, w, stride=(s_h, s_w))
    y.backward(torch.from_numpy(G.astype(np.float64)).permute(0, 3, 1, 2))
    tI = x.grad.permute(0, 2, 3, 1).numpy()
    tK = w.grad.permute(2, 3, 1, 0).numpy()
    dI = orc.conv2d_dgrad(G, K, i_h, i_w, s_h, s_w)
    dK = orc.conv2d_wgrad(I, G, k_h, k_w, s_h, s_w)
    assert np.allclose(dI, tI, rtol=1e-12, atol=1e-12)
    assert np.allclose(dK, tK, rtol=1e-12, atol=1e-11)


def test_worked_example_closed_forms(orc):
    """7x7 input I[h, w] = 7h + w, 3x3 kernel K[a, b] = 3a + b + 1, G = 1:
    dK[a, b] = sum over the 5x5 outputs of I[y + a, x + b] = 25(7a + b) + 400;
    dI[h, x] sums K over the windows covering (h, x): corners get one kernel
    element each (K[0,0] = 1 at (0,0), K[0,2] = 3 at (0,6), K[2,0] = 7 at
    (6,0), K[2,2] = 9 at (6,6)), the centre all nine (45). A flipped kernel
    would swap the corner values."""
    I = (7 * np.arange(7).reshape(7, 1) + np.arange(7).reshape(1, 7)).astype(F32).reshape(1, 7, 7, 1)
    K = (3 * np.arange(3).reshape(3, 1) + np.arange(3).reshape(1, 3) + 1).astype(F32).reshape(3, 3, 1, 1)
    G = np.ones((1, 5, 5, 1), F32)
    dK = orc.conv2d_wgrad(I, G, 3, 3, 1, 1)[:, :, 0, 0]
    for a in range(3):
        for b in range(3):
            assert dK[a, b] == 25 * (7 * a + b) + 400
    dI = orc.conv2d_dgrad(G, K, 7, 7, 1, 1)[0, :, :, 0]
    assert (dI[0, 0], dI[0, 6], dI[6, 0], dI[6, 6], dI[3, 3]) == (1, 3, 7, 9, 45)
    assert dI.sum() == 25 * K.sum()


@pytest.mark.parametrize("d", [(2, 12, 11, 3, 3, 4, 5, 2, 3), (1, 9, 9, 2, 2, 2, 3, 3, 3)])
def test_delta_gradients(orc, d):
    """A gradient that is 1 at one output (n0, y0, x0, m0) stamps the kernel
    K[:, :, :, m0] into dI at (y0*s_h, x0*s_w), unflipped, and copies the input
    patch there into dK[:, :, :, m0]."""
    i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w = d
    o_h, o_w = out_hw(d)
    I, K, _ = rand_problem(11, d)
    n0, y0, x0, m0 = i_n - 1, o_h - 1, o_w // 2, k_c - 1
    G = np.zeros((i_n, o_h, o_w, k_c), F32)
    G[n0, y0, x0, m0] = 1
    dI = orc.conv2d_dgrad(G, K, i_h, i_w, s_h, s_w)
    want = np.zeros_like(dI)
    want[n0, y0 * s_h:y0 * s_h + k_h, x0 * s_w:x0 * s_w + k_w, :] = K[:, :, :, m0]
    assert np.array_equal(dI, want)
    dK = orc.conv2d_wgrad(I, G, k_h, k_w, s_h, s_w)
    wantK = np.zeros_like(dK)
    wantK[:, :, :, m0] = I[n0, y0 * s_h:y0 * s_h + k_h, x0 * s_w:x0 * s_w + k_w, :]
    assert np.array_equal(dK, wantK)


@pytest.mark.parametrize("d", SHAPES)
def test_mec_forms_equal_direct(orc, d):
    I, K, G = rand_problem(5 * sum(d), d)
    i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w = d
    dL = orc.mec_dgrad_lowered(G, K, i_h, i_w, s_h, s_w)
    assert dL.shape == (i_n, out_hw(d)[1], i_h, k_w, i_c)
    assert np.array_equal(orc.mec_fold(dL, i_w, s_w), orc.conv2d_dgrad(G, K, i_h, i_w, s_h, s_w))
    L = orc.mec_lower(I, k_h, k_w, k_c, s_h, s_w)
    assert np.array_equal(orc.mec_wgrad_lowered(L, G, k_h, s_h, s_w),
                          orc.conv2d_wgrad(I, G, k_h, k_w, s_h, s_w))


@pytest.mark.parametrize("d", SHAPES)
def test_dL_rows_past_last_slab_are_zero(orc, d):
    _, K, G = rand_problem(9 * sum(d), d)
    i_h, s_h, k_h = d[1], d[7], d[4]
    dL = orc.mec_dgrad_lowered(G, K, i_h, d[2], s_h, d[8])
    used = (out_hw(d)[0] - 1) * s_h + k_h
    assert not dL[:, :, used:].any()


@pytest.mark.parametrize("d", SHAPES)
def test_fold_is_adjoint_of_lowering(orc, d):
    rng = np.random.default_rng(13 * sum(d))
    i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w = d
    I = ints(rng, (i_n, i_h, i_w, i_c))
    L = orc.mec_lower(I, k_h, k_w, k_c, s_h, s_w)
    Y = ints(rng, L.shape)
    lhs = float(np.sum(L.astype(np.float64) * Y))
    assert lhs == float(np.sum(I.astype(np.float64) * orc.mec_fold(Y, i_w, s_w)))
    # fp64 and fp32 inputs of the fold agree
    assert np.array_equal(orc.mec_fold(Y, i_w, s_w), orc.mec_fold(Y.astype(np.float64), i_w, s_w))
