"""The no-alloc weight gradient (mec_conv2d_wgrad_noalloc): partial sums in
the library's static device scratch, no allocation in the call. Checked
against the entry point it mirrors (mec_conv2d_wgrad, same kernels and
splits: bit for bit) and against the oracle, on two calls in a row, the
second with a smaller input, so the scratch holds the first call's partial
sums when the second starts."""
import ctypes

import numpy as np
import pytest
import torch

import paper_1706_06873_amd as mec
from paper_1706_06873_amd import workloads as wl

DEV = "cuda:0"


def test_noalloc_refuses_beyond_scratch():
    """A shape whose partial sums exceed the static array is refused before
    anything is enqueued (fake pointers, never dereferenced)."""
    d = (1, 16, 16, 512, 11, 11, 512, 1, 1)
    assert mec.grad_workspace_bytes(*d, grad_pass=mec.GRAD_KERNEL) > mec.noalloc_scratch_bytes()
    fake = ctypes.c_void_p(0x100000)
    st = mec.lib.mec_conv2d_wgrad_noalloc(fake, fake, fake, *d, mec.F32, None)
    assert st == -6, st
    assert "static scratch" in mec.strerror(st)
    # bf16 is refused as for mec_conv2d_wgrad
    assert mec.lib.mec_conv2d_wgrad_noalloc(fake, fake, fake, 1, 9, 9, 4, 3, 3, 4, 1, 1, mec.BF16, None) == -5


def _problem(seed, d, dist):
    I, K = wl.random_case(seed, *d, dtype="f32", dist=dist)
    o_h, o_w = mec.output_dims(d[1], d[2], d[4], d[5], d[7], d[8])
    g = torch.Generator().manual_seed(seed + 1)
    if dist == "int":
        G = torch.randint(-3, 4, (d[0], o_h, o_w, d[6]), generator=g).to(torch.float32)
    else:
        G = torch.rand((d[0], o_h, o_w, d[6]), generator=g) * 2 - 1
    return I, G


@pytest.mark.gpu
@pytest.mark.parametrize("dist", ["int", "u11"])
def test_noalloc_matches_workspace_entry_point(orc, dist):
    big = (4, 30, 29, 64, 3, 3, 64, 1, 1)      # slab-reuse weight-gradient kernel
    small = (2, 13, 12, 16, 5, 5, 40, 2, 1)    # plain tiles, strided, fewer shares
    for d in (big, small):
        print("[case] noalloc wgrad", dist, d, flush=True)
        assert mec.grad_workspace_bytes(*d, grad_pass=mec.GRAD_KERNEL) <= mec.noalloc_scratch_bytes()
        I, G = _problem(sum(d), d, dist)
        Id, Gd = I.to(DEV), G.to(DEV)
        k_h, k_w, s_h, s_w = d[4], d[5], d[7], d[8]
        dK = torch.full((k_h, k_w, d[3], d[6]), 7.0, device=DEV)
        mec.conv2d_wgrad_noalloc(Id, Gd, k_h, k_w, s_h, s_w, dK=dK)
        ref_dev = mec.conv2d_wgrad(Id, Gd, k_h, k_w, s_h, s_w)
        torch.cuda.synchronize()
        got = dK.cpu().numpy()
        assert np.array_equal(got, ref_dev.cpu().numpy())
        ref = orc.conv2d_wgrad(I.numpy(), G.numpy(), k_h, k_w, s_h, s_w)
        if dist == "int":
            assert np.array_equal(got, ref.astype(np.float32))
        else:
            assert np.linalg.norm(got - ref) / np.linalg.norm(ref) <= 1e-5
