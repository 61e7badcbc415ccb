"""Seeded random shapes through every algorithm and both training passes.

A fixed generator draws convolutions over kernel sizes 1-11, strides 1-4
(also larger than the kernel), 1-256 channels, ragged sizes and batches up
to 32,
so that the per-shape kernel choices (fixed and generic tiles, the split
reduction, the streaming kernel, the element-gathering bf16 form, the
sub-pixel phases of dI) meet shapes nobody picked by hand. Inputs are small
integers, so every result must match the oracle bit for bit.
"""
import random

import numpy as np
import pytest
import torch

import paper_1706_06873_amd as mec
from paper_1706_06873_amd import workloads as wl

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def draw_shapes(n, seed, batches, extent, max_mac):
    rng = random.Random(seed)
    out = []
    while len(out) < n:
        k_h = rng.choice([1, 2, 3, 3, 3, 4, 5, 7, 11])
        k_w = k_h if rng.random() < 0.7 else rng.choice([1, 2, 3, 5, 7])
        s_h = rng.choice([1, 1, 1, 2, 2, 3, 4])
        s_w = s_h if rng.random() < 0.7 else rng.choice([1, 2, 3])
        i_c = rng.choice([1, 2, 3, 4, 8, 16, 24, 32, 48, 64, 96, 128, 256])
        k_c = rng.choice([1, 3, 4, 8, 30, 40, 64, 72, 96, 128, 136, 256])
        i_h = k_h + rng.randint(0, extent)
        i_w = k_w + rng.randint(0, extent)
        i_n = rng.choice(batches)
        o_h, o_w = (i_h - k_h) // s_h + 1, (i_w - k_w) // s_w + 1
        if i_n * o_h * o_w * k_c * k_h * k_w * i_c > max_mac:
            continue
        out.append((i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w))
    return out


# small shapes; then fewer, larger ones with enough tiles for the split
# reduction, the streaming kernel and several tiles per compute unit
SHAPES = draw_shapes(160, 20261202, [1, 2, 3, 5], 24, 4e7) + \
    draw_shapes(24, 777, [8, 16, 32], 40, 3e8)


def say(*a):
    print("[case]", *a, flush=True)


def host(t):
    return wl.to_oracle_array(t)


@pytest.mark.parametrize("dims", SHAPES)
def test_random_forward(orc, dims):
    say("random forward", dims)
    k_h, k_w, k_c, s_h, s_w = dims[4:]
    for dtype in ("f32", "bf16"):
        I, K = wl.random_case(7 + sum(dims), *dims, dtype=dtype, dist="int")
        ref = orc.conv2d_direct(host(I), host(K), s_h, s_w)
        assert np.abs(ref).max() < 2 ** 24
        L = mec.lower(I.to(DEV), k_h, k_w, k_c, s_h, s_w)
        torch.cuda.synchronize()
        assert np.array_equal(host(L.cpu()), orc.mec_lower(host(I), k_h, k_w, k_c, s_h, s_w)), dtype
        for algo in ("lowered", "fused", "im2col"):
            O = mec.conv2d(I.to(DEV), K.to(DEV), s_h, s_w, algo=algo)
            torch.cuda.synchronize()
            assert np.array_equal(O.cpu().numpy(), ref.astype(np.float32)), (dtype, algo)


@pytest.mark.parametrize("dims", SHAPES)
def test_random_gradients(orc, dims):
    say("random gradients", dims)
    i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w = dims
    o_h, o_w = mec.output_dims(i_h, i_w, k_h, k_w, s_h, s_w)
    I, K = wl.random_case(11 + sum(dims), *dims, dist="int")
    G = torch.randint(-3, 4, (i_n, o_h, o_w, k_c), generator=torch.Generator().manual_seed(sum(dims))).float()
    ref_dI = orc.conv2d_dgrad(G.numpy(), K.numpy(), i_h, i_w, s_h, s_w)
    ref_dK = orc.conv2d_wgrad(I.numpy(), G.numpy(), k_h, k_w, s_h, s_w)
    dI = mec.conv2d_dgrad(G.to(DEV), K.to(DEV), i_h, i_w, s_h, s_w)
    dK = mec.conv2d_wgrad(I.to(DEV), G.to(DEV), k_h, k_w, s_h, s_w)
    torch.cuda.synchronize()
    assert np.array_equal(dI.cpu().numpy(), ref_dI.astype(np.float32))
    assert np.array_equal(dK.cpu().numpy(), ref_dK.astype(np.float32))
