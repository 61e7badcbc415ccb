"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Bars: L bit for bit; O within relative L2 error 1e-5 for fp32 inputs, and for
bf16 inputs within 1e-5 of the oracle fed the same bf16 values (the GPU
accumulates in fp32) and within 1e-2 of the oracle fed the fp32 values before
rounding. With small-integer inputs every partial sum is exact in fp32, so O
must then match bit for bit.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_1706_06873_amd as mec
from paper_1706_06873_amd import workloads as wl

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
TOL_F32 = 1e-5
TOL_BF16_VS_F32 = 1e-2


def say(*a):
    print("[case]", *a, flush=True)


def rel_l2(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.linalg.norm(ref)
    return np.linalg.norm(got - ref) / (den if den > 0 else 1.0)


def to_dev(t):
    return t.to(DEV)


def host(t):
    return wl.to_oracle_array(t)


def case(seed, dims, dtype="f32", dist="u11"):
    return wl.random_case(seed, *dims, dtype=dtype, dist=dist)


# Shapes that reach every kernel configuration and the ragged edges: pairs not
# a multiple of 32, o_h not a multiple of the h tile, k_c not a multiple of 32,
# R not a multiple of the r-chunk, s not dividing i - k, s >= k, k = i.
SWEEP = [
    # i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w
    (1, 7, 7, 1, 3, 3, 1, 1, 1),
    (2, 19, 17, 64, 3, 3, 64, 1, 1),     # f32 wide
    (3, 20, 21, 16, 3, 3, 40, 1, 2),     # wide, ragged channels
    (2, 23, 25, 3, 3, 3, 64, 1, 1),      # narrow (R = 9)
    (3, 31, 30, 3, 11, 11, 96, 4, 4),    # tall (11x11 s4)
    (1, 35, 33, 3, 11, 11, 100, 4, 3),   # tall, ragged channels and strides
    (2, 27, 29, 3, 11, 11, 30, 4, 4),    # tall, k_c not a multiple of 4 (scalar K loads)
    (2, 13, 12, 5, 5, 5, 33, 2, 2),
    (1, 30, 9, 2, 20, 3, 7, 1, 1),       # generic HT=4 (tall k_h)
    (1, 40, 9, 1, 13, 3, 130, 9, 1),     # generic HT=4, large s_h
    (1, 60, 9, 1, 20, 3, 130, 16, 1),    # generic HT=1 (hrows of HT=4 too many)
    (2, 9, 9, 4, 3, 3, 8, 3, 3),         # s == k
    (1, 11, 10, 3, 2, 2, 5, 4, 3),       # s > k
    (2, 6, 5, 7, 6, 5, 3, 1, 1),         # k == i: o = 1 x 1
    (4, 8, 8, 8, 1, 1, 16, 1, 1),        # 1x1
    (1, 3, 70, 2, 3, 1, 1, 1, 1),        # o_h = 1, many pairs
    (33, 4, 4, 4, 2, 2, 33, 1, 1),       # pairs = 99
    (1, 5, 200, 64, 3, 3, 8, 1, 1),      # input rows wider than the lowering's LDS stage
    (2, 6, 130, 33, 3, 2, 5, 1, 3),      # wide odd rows
    (16, 28, 28, 128, 3, 3, 128, 1, 1),  # 3x3 tiles of 2 output rows (many channel tiles)
    (2, 21, 19, 16, 7, 7, 40, 2, 2),     # 7x7 s2, 16-byte rows, ragged channels
    (1, 23, 25, 3, 7, 7, 70, 2, 3),      # 7x7 s2, short rows, k_c not a multiple of 4
    (2, 14, 13, 32, 5, 5, 64, 1, 2),     # 5x5 s1, 16-byte rows
    (2, 14, 13, 32, 5, 5, 66, 1, 1),     # 5x5 s1, k_c not a multiple of 4
    (2, 15, 14, 16, 2, 2, 40, 1, 1),     # 2x2 s1, 16-byte rows
    (2, 17, 16, 8, 4, 4, 64, 1, 1),      # 4x4 s1, 16-byte rows
    (3, 12, 13, 32, 4, 3, 36, 1, 2),     # 4x3, s_w = 2
]

SWEEP_BF16 = [
    (2, 19, 17, 64, 3, 3, 64, 1, 1),     # bf16 8-wide loads
    (2, 10, 10, 16, 3, 3, 96, 1, 1),
    (3, 17, 15, 3, 3, 3, 40, 1, 2),      # bf16 generic
    (2, 31, 30, 3, 11, 11, 64, 4, 4),    # bf16 tall -> HT=1
    (1, 12, 12, 8, 5, 3, 130, 2, 1),
    (2, 6, 5, 7, 6, 5, 3, 1, 1),
    (1, 4, 400, 64, 3, 3, 16, 1, 1),     # wide rows (gather lowering)
    (3, 18, 16, 40, 3, 3, 136, 1, 1),    # bf16 3x3: two channel tiles, the second ragged
    (2, 9, 40, 24, 3, 3, 8, 1, 2),       # bf16 3x3, R not a multiple of the r-chunk
    (2, 14, 13, 32, 5, 5, 136, 1, 1),    # bf16 5x5 s1: two channel tiles, the second ragged
    (2, 21, 19, 16, 7, 7, 40, 2, 2),     # bf16 7x7 s2, ragged channels (the 64-channel tile)
    (3, 29, 27, 16, 7, 7, 64, 2, 2),     # bf16 7x7 s2, 64 channels, ragged pairs and rows
    (1, 21, 23, 8, 7, 7, 24, 2, 2),      # bf16 7x7 s2, fewer channels than one block
    (2, 21, 19, 16, 7, 7, 96, 2, 2),     # bf16 7x7 s2, the 128-channel tile
    (2, 35, 33, 3, 11, 11, 104, 4, 3),   # bf16 11x11 s4, rows of 33 gathered by element, two channel tiles
    (1, 27, 29, 5, 11, 11, 40, 4, 4),    # the same, rows of 55
    (1, 23, 25, 3, 7, 7, 72, 2, 3),      # bf16 7x7 s2, rows of 21: the generic kernel
]


def run_conv(I, K, s_h, s_w, algo):
    O = mec.conv2d(to_dev(I), to_dev(K), s_h, s_w, algo=algo)
    torch.cuda.synchronize()
    return O.cpu().numpy()


@pytest.mark.parametrize("dims", SWEEP)
@pytest.mark.parametrize("algo", ["lowered", "fused"])
def test_conv_f32_sweep(orc, dims, algo):
    say("conv f32", algo, dims)
    I, K = case(sum(dims), dims)
    s_h, s_w = dims[7], dims[8]
    ref = orc.conv2d_direct(host(I), host(K), s_h, s_w)
    got = run_conv(I, K, s_h, s_w, algo)
    assert got.shape == ref.shape
    assert rel_l2(got, ref) <= TOL_F32


@pytest.mark.parametrize("dims", SWEEP)
@pytest.mark.parametrize("algo", ["lowered", "fused"])
def test_conv_f32_integer_inputs_bitwise(orc, dims, algo):
    say("conv f32 int", algo, dims)
    I, K = case(7 + sum(dims), dims, dist="int")
    s_h, s_w = dims[7], dims[8]
    ref = orc.conv2d_direct(host(I), host(K), s_h, s_w)
    assert np.abs(ref).max() < 2 ** 24
    got = run_conv(I, K, s_h, s_w, algo)
    assert np.array_equal(got, ref.astype(np.float32))


@pytest.mark.parametrize("dims", SWEEP_BF16)
@pytest.mark.parametrize("algo", ["lowered", "fused"])
def test_conv_bf16_sweep(orc, dims, algo):
    say("conv bf16", algo, dims)
    I32, K32 = case(3 * sum(dims), dims, dtype="f32")
    I, K = I32.to(torch.bfloat16), K32.to(torch.bfloat16)
    s_h, s_w = dims[7], dims[8]
    ref_bf = orc.conv2d_direct(host(I), host(K), s_h, s_w)
    ref_32 = orc.conv2d_direct(host(I32), host(K32), s_h, s_w)
    got = run_conv(I, K, s_h, s_w, algo)
    assert rel_l2(got, ref_bf) <= TOL_F32
    assert rel_l2(got, ref_32) <= TOL_BF16_VS_F32


@pytest.mark.parametrize("dims", SWEEP_BF16)
def test_conv_bf16_integer_inputs_bitwise(orc, dims):
    say("conv bf16 int", dims)
    I, K = case(11 + sum(dims), dims, dtype="bf16", dist="int")
    s_h, s_w = dims[7], dims[8]
    ref = orc.conv2d_direct(host(I), host(K), s_h, s_w)
    for algo in ("lowered", "fused"):
        assert np.array_equal(run_conv(I, K, s_h, s_w, algo), ref.astype(np.float32))


@pytest.mark.parametrize("dims", SWEEP + SWEEP_BF16)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_lower_bitwise_sweep(orc, dims, dtype):
    say("lower", dtype, dims)
    I, _ = case(5 * sum(dims), dims, dtype=dtype)
    k_h, k_w, k_c, s_h, s_w = dims[4:]
    ref = orc.mec_lower(host(I), k_h, k_w, k_c, s_h, s_w)
    L = mec.lower(to_dev(I), k_h, k_w, k_c, s_h, s_w)
    torch.cuda.synchronize()
    got = host(L.cpu())
    assert got.shape == ref.shape and np.array_equal(got, ref)


# Short or unaligned runs take the strip lowering. Enough images x rows that a
# workgroup owns chunks of several rows (the chunk height grows with
# i_n * i_h), with I and L placed off their 16-byte boundaries and at several
# offsets from a 128-byte line (the unit a workgroup owns in L).
STRIP_CASES = [
    (8, 150, 20, 3, 5, 5, 4, 1, 1),       # R = 15
    (16, 200, 21, 3, 11, 11, 4, 4, 4),    # R = 33, the 11x11 stride-4 layout
    (12, 256, 13, 1, 1, 1, 2, 1, 1),      # R = 1: a granule spans several rows
    (6, 180, 40, 2, 3, 1, 3, 2, 2),       # R = 2
    (8, 160, 19, 5, 3, 3, 4, 1, 2),       # R = 15, stride 2
]


@pytest.mark.parametrize("dims", STRIP_CASES)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("offs", [(0, 0), (1, 3), (3, 1), (2, 5), (1, 21)])
def test_lower_strip_offsets_and_guards(orc, dims, dtype, offs):
    """L bit for bit, and nothing written outside it, for I and L starting
    ioff and loff (+ 24 guard) elements past a 256-byte boundary."""
    ioff, loff = offs
    say("lower strip", dtype, dims, offs)
    I, _ = case(31 * sum(dims) + ioff, dims, dtype=dtype)
    k_h, k_w, k_c, s_h, s_w = dims[4:]
    ref = orc.mec_lower(host(I), k_h, k_w, k_c, s_h, s_w)
    tdt = I.dtype
    ibuf = torch.zeros(I.numel() + 16, dtype=tdt, device=DEV)
    Id = ibuf[ioff:ioff + I.numel()].view(I.shape)
    Id.copy_(I.to(DEV))
    nL = ref.size
    guard = 24
    lbuf = torch.full((nL + 2 * guard,), -3.0, dtype=tdt, device=DEV)
    Ld = lbuf[guard + loff:guard + loff + nL]
    mec.lower(Id, k_h, k_w, k_c, s_h, s_w, L=Ld)
    torch.cuda.synchronize()
    out = lbuf.cpu()
    assert np.array_equal(host(out[guard + loff:guard + loff + nL]).reshape(ref.shape), ref)
    assert bool((out[:guard + loff] == -3.0).all()) and bool((out[guard + loff + nL:] == -3.0).all())


# fp32 3x3 stride-1 layers whose tile cost model picks 4-row and 14-row tiles
# (small layers pick 2-row tiles, e.g. (16, 28, 28, 128, ...) in the sweep).
@pytest.mark.parametrize("dims", [
    (8, 66, 66, 16, 3, 3, 192, 1, 1),    # 4 output rows per tile
    (8, 58, 58, 16, 3, 3, 256, 1, 1),    # 14 output rows per tile
])
def test_row_tile_choices_bitwise(orc, dims):
    say("row tiles", dims)
    I, K = case(3 * sum(dims), dims, dist="int")
    s_h, s_w = dims[7], dims[8]
    ref = orc.conv2d_direct(host(I), host(K), s_h, s_w).astype(np.float32)
    for algo in ("lowered", "fused"):
        assert np.array_equal(run_conv(I, K, s_h, s_w, algo), ref), algo


# 3x3 layers over 1-3 channels (R <= 10) take the streaming product kernel: a
# persistent workgroup walks several tiles. Shapes with more tiles than the
# ~768 resident workgroups, ragged pairs, rows and channel tiles, and k_c not
# a multiple of 4 (element K loads, element O stores).
STREAM_CASES = [
    (16, 130, 130, 3, 3, 3, 64, 1, 1),   # 1024 tiles
    (20, 100, 61, 3, 3, 3, 100, 1, 1),   # 962 tiles, every dimension ragged
    (32, 90, 90, 3, 3, 3, 30, 1, 1),     # 968 tiles, k_c = 30
    (8, 60, 60, 1, 3, 3, 64, 1, 2),      # R = 3, stride 2 along w
    (6, 41, 47, 2, 3, 3, 36, 1, 1),      # R = 6
]


@pytest.mark.parametrize("dims", STREAM_CASES)
def test_stream_products(orc, dims):
    say("stream", dims)
    s_h, s_w = dims[7], dims[8]
    I, K = case(11 + sum(dims), dims)
    ref = orc.conv2d_direct(host(I), host(K), s_h, s_w)
    Ii, Ki = case(13 + sum(dims), dims, dist="int")
    refi = orc.conv2d_direct(host(Ii), host(Ki), s_h, s_w)
    assert np.abs(refi).max() < 2 ** 24
    for algo in ("lowered", "fused"):
        assert rel_l2(run_conv(I, K, s_h, s_w, algo), ref) <= TOL_F32, algo
        assert np.array_equal(run_conv(Ii, Ki, s_h, s_w, algo), refi.astype(np.float32)), algo


@pytest.mark.parametrize("shift", [1, 3])
def test_stream_unaligned(orc, shift):
    """The streaming kernel with I, K, L and O off their 16-byte boundaries:
    element K loads and element O stores."""
    dims = (6, 41, 47, 3, 3, 3, 36, 1, 1)
    say("stream unaligned", shift, dims)
    I, K = case(23, dims, dist="int")
    ref = orc.conv2d_direct(host(I), host(K), 1, 1).astype(np.float32)

    def offset_copy(t):
        buf = torch.zeros(t.numel() + 8, dtype=t.dtype, device=DEV)
        v = buf[shift:shift + t.numel()].view(t.shape)
        v.copy_(t.to(DEV))
        return v

    Id, Kd = offset_copy(I), offset_copy(K)
    Od = torch.zeros(ref.size + 8, dtype=torch.float32, device=DEV)[shift:shift + ref.size].view(ref.shape)
    ws = torch.zeros(mec.workspace_bytes(*dims) + 64, dtype=torch.uint8, device=DEV)[4 * shift:]
    for algo in ("lowered", "fused"):
        Od.zero_()
        mec.conv2d(Id, Kd, 1, 1, algo=algo, O=Od, workspace=ws)
        torch.cuda.synchronize()
        assert np.array_equal(Od.cpu().numpy(), ref), algo


def test_stream_output_not_written_outside(orc):
    dims = (20, 100, 61, 3, 3, 3, 100, 1, 1)
    say("stream guard", dims)
    I, K = case(17, dims)
    ref = orc.conv2d_direct(host(I), host(K), 1, 1).astype(np.float32)
    buf = torch.full((ref.size + 4096,), 7.0, dtype=torch.float32, device=DEV)
    O = buf[1024:1024 + ref.size].view(ref.shape)
    for algo in ("lowered", "fused"):
        mec.conv2d(to_dev(I), to_dev(K), 1, 1, algo=algo, O=O)
        torch.cuda.synchronize()
        b = buf.cpu().numpy()
        assert np.all(b[:1024] == 7.0) and np.all(b[1024 + ref.size:] == 7.0)
        assert rel_l2(O.cpu().numpy(), ref) <= TOL_F32


# fp32 3x3 layers with few tiles and long reductions split each tile's r-chunks
# between two workgroups that add into a zeroed O (cv11/cv12-like shapes).
SPLIT_CASES = [
    (4, 14, 14, 256, 3, 3, 256, 1, 1),
    (2, 7, 7, 512, 3, 3, 512, 1, 1),
    (3, 16, 15, 64, 3, 3, 100, 1, 1),    # ragged channel tile
]


@pytest.mark.parametrize("dims", SPLIT_CASES)
@pytest.mark.parametrize("algo", ["lowered", "fused"])
def test_split_reduction(orc, dims, algo):
    """Within tolerance on floats, bit for bit on small integers, and the same
    bits on a second run (two partial sums onto +0 commute exactly)."""
    say("split", algo, dims)
    s_h, s_w = dims[7], dims[8]
    I, K = case(29 + sum(dims), dims)
    ref = orc.conv2d_direct(host(I), host(K), s_h, s_w)
    O1 = run_conv(I, K, s_h, s_w, algo)
    assert rel_l2(O1, ref) <= TOL_F32
    assert np.array_equal(run_conv(I, K, s_h, s_w, algo), O1)
    Ii, Ki = case(31 + sum(dims), dims, dist="int")
    refi = orc.conv2d_direct(host(Ii), host(Ki), s_h, s_w)
    assert np.array_equal(run_conv(Ii, Ki, s_h, s_w, algo), refi.astype(np.float32))


# bf16 3x3 layers with few tiles split their reduction the same way.
# fp32 layers whose tiles are staged by direct-to-LDS loads (rows of a
# multiple of 16): 3x3 14-row tiles, and 5x5 tiles from I; ragged pairs, rows
# and channel tiles.
DMA_CASES_F32 = [
    (33, 30, 29, 16, 3, 3, 72, 1, 1),    # 891 pairs, 28 rows, channels 64 + 8
    (40, 60, 58, 32, 3, 3, 64, 1, 1),    # 2240 pairs, 58 rows (four 14-row tiles and one of 2)
    (3, 17, 21, 32, 5, 5, 72, 1, 1),     # 5x5 (from I only): ragged pairs, rows, channels
]


@pytest.mark.parametrize("dims", DMA_CASES_F32)
@pytest.mark.parametrize("algo", ["lowered", "fused"])
def test_f32_direct_to_lds_tiles(orc, dims, algo):
    say("f32 dma", algo, dims)
    assert (dims[5] * dims[3]) % 16 == 0
    s_h, s_w = dims[7], dims[8]
    Ii, Ki = case(61 + sum(dims), dims, dist="int")
    refi = orc.conv2d_direct(host(Ii), host(Ki), s_h, s_w)
    assert np.abs(refi).max() < 2 ** 24
    assert np.array_equal(run_conv(Ii, Ki, s_h, s_w, algo), refi.astype(np.float32))
    I, K = case(67 + sum(dims), dims)
    assert rel_l2(run_conv(I, K, s_h, s_w, algo), orc.conv2d_direct(host(I), host(K), s_h, s_w)) <= TOL_F32


# fp32 tall kernels over short rows (11x11 at strides 3 and 4, other k_h >= 9,
# k_h of 5 to 8 at strides of 2 and more down, and, fused, k_h >= 3 over rows of
# at most 10 elements, with rows of L of at most 48 elements): the flat-window kernel (one wave per workgroup, 8 pairs x 4 output
# rows per MFMA block, rows of L streamed through a ring in LDS). The cases
# reach a ragged last pair group, o_h not a multiple of 4, one, two and three
# 32-channel blocks, several channel tiles, pair groups across images, s_w = 1,
# 2 and 3, i_c = 1, 2, 3 and 6, strides of 2 to 16 down, and o = 1 x 1.
RING_CASES = [
    (1, 35, 31, 3, 11, 11, 96, 4, 4),     # 3 row groups: items of 2 and 1 groups
    (2, 39, 27, 3, 11, 11, 40, 4, 4),     # two channel blocks, the second 8 wide
    (1, 47, 35, 3, 11, 11, 100, 4, 4),    # two channel tiles of 96, the second 4 wide
    (3, 23, 19, 3, 11, 11, 20, 4, 4),     # one channel block; 9 pairs (ragged pair group)
    (1, 11, 11, 3, 11, 11, 96, 4, 4),     # k = i: o = 1 x 1
    (2, 30, 30, 2, 11, 11, 33, 4, 3),     # i_c = 2 (R = 22), s_w = 3
    (3, 30, 25, 1, 11, 11, 1, 4, 4),      # i_c = 1, k_c = 1
    (5, 15, 15, 3, 11, 11, 8, 4, 4),      # o = 2 x 2, pair groups across images
    (1, 19, 40, 3, 11, 11, 96, 4, 1),     # s_w = 1
    (1, 43, 20, 3, 11, 11, 130, 4, 4),    # two channel tiles, the second 34 wide
    (2, 40, 31, 3, 11, 11, 96, 3, 3),     # stride 3
    (3, 29, 27, 3, 11, 11, 40, 3, 4),     # stride 3 down, 4 across
    (2, 33, 20, 2, 9, 5, 70, 3, 2),       # 9x5 over 2 channels (R = 10), stride 3 x 2
    (1, 40, 9, 1, 13, 3, 130, 9, 1),      # 13x3, stride 9 down (R = 3)
    (1, 60, 9, 1, 20, 3, 130, 16, 1),     # 20x3, stride 16 down
    (2, 29, 25, 3, 7, 7, 64, 2, 2),       # 7x7 stride 2 over 3 channels (cv3-like)
    (3, 21, 19, 3, 5, 5, 40, 2, 2),       # 5x5 stride 2, two channel blocks
    (1, 23, 30, 6, 5, 5, 100, 2, 3),      # 5x5 over 6 channels, stride 2 x 3, two channel tiles
    (2, 20, 17, 2, 6, 3, 33, 3, 2),       # 6x3 stride 3 down over 2 channels
    (2, 18, 20, 3, 3, 3, 64, 1, 1),       # 3x3 over 3 channels (R = 9), stride 1
    (3, 11, 13, 1, 3, 3, 20, 1, 1),       # 3x3 over 1 channel (R = 3)
    (1, 16, 33, 2, 5, 5, 40, 1, 2),       # 5x5 over 2 channels (R = 10), stride 1 x 2
]


@pytest.mark.parametrize("dims", RING_CASES)
@pytest.mark.parametrize("algo", ["lowered", "fused"])
def test_ring_products(orc, dims, algo):
    say("ring", algo, dims)
    s_h, s_w = dims[7], dims[8]
    Ii, Ki = case(71 + sum(dims), dims, dist="int")
    refi = orc.conv2d_direct(host(Ii), host(Ki), s_h, s_w)
    assert np.abs(refi).max() < 2 ** 24
    assert np.array_equal(run_conv(Ii, Ki, s_h, s_w, algo), refi.astype(np.float32))
    I, K = case(73 + sum(dims), dims)
    assert rel_l2(run_conv(I, K, s_h, s_w, algo), orc.conv2d_direct(host(I), host(K), s_h, s_w)) <= TOL_F32


# Windows of at most two blocks of k-steps (3x3 over 1 to 3 channels, 5x5 over
# one, and the like): K held in registers for the whole item, fills issued
# three blocks ahead of their reads, and waits counted per block. The cases
# reach 1, 2 and 3 channel blocks, two channel tiles, blocks of 8 steps (one
# and two of them), a 5x5 stride-2 kernel (also from L), and, at stride 8
# down, blocks whose chunks the ring could not take that far ahead (those wait
# for everything in flight).
SHORT_RING_CASES = [
    (2, 18, 20, 3, 3, 3, 96, 1, 1),       # three channel blocks
    (1, 19, 21, 3, 3, 3, 130, 1, 1),      # two channel tiles, the second 34 wide
    (2, 20, 24, 1, 3, 5, 40, 1, 1),       # 15 elements: one block of 8 steps
    (2, 21, 22, 2, 4, 4, 33, 1, 1),       # 32 elements: two blocks of 8 steps
    (2, 23, 25, 1, 5, 5, 40, 2, 2),       # 5x5 stride 2 over one channel
    (3, 58, 10, 3, 3, 3, 40, 8, 1),       # stride 8 down: lead cut short by the ring
    (2, 58, 12, 2, 3, 5, 70, 8, 2),       # the same with three channel blocks, stride 8 x 2
]


@pytest.mark.parametrize("dims", SHORT_RING_CASES)
@pytest.mark.parametrize("algo", ["lowered", "fused"])
def test_ring_short_windows(orc, dims, algo):
    say("ring short", algo, dims)
    s_h, s_w = dims[7], dims[8]
    Ii, Ki = case(79 + sum(dims), dims, dist="int")
    refi = orc.conv2d_direct(host(Ii), host(Ki), s_h, s_w)
    assert np.abs(refi).max() < 2 ** 24
    assert np.array_equal(run_conv(Ii, Ki, s_h, s_w, algo), refi.astype(np.float32))
    I, K = case(81 + sum(dims), dims)
    assert rel_l2(run_conv(I, K, s_h, s_w, algo), orc.conv2d_direct(host(I), host(K), s_h, s_w)) <= TOL_F32


# Short windows whose launch splits the items of its last partial round:
# one-group items of 3x3 over 3 channels at 64 channels (16 pieces), and
# two-group items at 40 channels (32 pieces), on 2048 wave slots.
SHORT_SPLIT_CASES = [
    ((257, 6, 66, 3, 3, 3, 64, 1, 1), (1, 2048, 16)),
    ((257, 10, 66, 3, 3, 3, 40, 1, 1), (2, 2048, 32)),
]


@pytest.mark.parametrize("dims,plan", SHORT_SPLIT_CASES)
def test_ring_short_split_tail(orc, dims, plan):
    n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w = dims
    KR = k_h * k_w * i_c
    bs = ring_block_steps(KR)
    nb = 3 if k_c > 64 else 2 if k_c > 32 else 1
    o_h, o_w = i_h - k_h + 1, i_w - k_w + 1
    slots = 8 * torch.cuda.get_device_properties(0).multi_processor_count
    got = ring_plan(-(-n * o_w // 8), -(-o_h // 4), -(-k_c // (32 * nb)), nb, slots,
                    -(-((KR + 1) // 2) // bs) * bs)
    say("ring short split", dims, "plan", got)
    if slots == 2048:
        assert got == plan
    I, K = case(87 + sum(dims), dims, dist="int")
    ref = orc.conv2d_direct(host(I), host(K), s_h, s_w)
    assert np.abs(ref).max() < 2 ** 24
    assert np.array_equal(run_conv(I, K, s_h, s_w, "fused"), ref.astype(np.float32))


def ring_block_steps(KR):
    """k-steps per block of the ring kernel: 7 where whole blocks of 7 pad the
    window's ceil(KR / 2) steps less than blocks of 8."""
    st = (KR + 1) // 2
    return 7 if (st + 6) // 7 * 7 < (st + 7) // 8 * 8 else 8


def _ring_rounds_cost(n, work, slots):
    """n workgroups of `work` k-steps plus a start of 37 over `slots` wave
    slots, in sixteenths of a k-step: whole rounds at two waves per SIMD; a
    last round over at most half the slots with products at 0.7 of the time,
    over more than half 17/16 of a whole round."""
    q, r = divmod(n, slots)
    t = q * (work + 37) * 16
    if r:
        t += work * 56 // 5 + 37 * 16 if 2 * r <= slots else (work + 37) * 17
    return t


def ring_plan(pgroups, ngroups, n_tiles, nb, slots, steps):
    """The ring launch's layout as the library chooses it: (row groups per
    item, whole items, split pieces). 1 to 16 groups per item, minimising the
    estimated time of the busiest slot (an item's products: gpi * steps * nb
    k-steps of one channel block; a split piece's: steps); the items of a
    last, partial round of at most a quarter of the slots split into one
    workgroup per row group and 32-channel block."""
    best, best_cost = (1, pgroups * ngroups * n_tiles, 0), None
    for gpi in range(1, min(16, ngroups) + 1):
        items = pgroups * -(-ngroups // gpi) * n_tiles
        rounds, r = divmod(items, slots)
        split = n_tiles == 1 and nb * gpi > 1 and rounds > 0 and r > 0 and 4 * r <= slots
        work = gpi * steps * nb
        if split:
            cost = rounds * (work + 37) * 16 + _ring_rounds_cost(r * nb * gpi, steps, slots)
        else:
            cost = _ring_rounds_cost(items, work, slots)
        if best_cost is None or cost < best_cost:
            best, best_cost = (gpi, items - r if split else items, r * nb * gpi if split else 0), cost
    return best


def ring_split_batch(slots, o_h, o_w, k_c, gpi):
    """Smallest batch whose ring launch has `gpi` row groups per item and
    splits at least 5 leftover items."""
    nb = 3 if k_c > 64 else 2 if k_c > 32 else 1
    KR = 11 * 33
    steps = -(-((KR + 1) // 2) // ring_block_steps(KR)) * ring_block_steps(KR)
    for n in range(1, 8 * slots):
        plan = ring_plan(-(-n * o_w // 8), -(-o_h // 4), -(-k_c // (32 * nb)), nb, slots, steps)
        if plan[0] == gpi and plan[2] >= 5 * nb * gpi:
            return n, plan
    raise AssertionError("no batch")


# Items of more than 8 row groups, in a single round of fewer items than
# wave slots (3x3 over one and three channels, fused, 8 channels): 10 groups
# per item, each pair group's whole height, the last group one row; 9 and 8
# groups per item over 17 groups; 16 groups per item, the last one one row.
LONG_ITEM_CASES = [
    ((175, 39, 49, 1, 3, 3, 8, 1, 1), 10),
    ((126, 68, 49, 3, 3, 3, 8, 1, 1), 9),
    ((197, 63, 49, 1, 3, 3, 8, 1, 1), 16),
]


@pytest.mark.parametrize("dims,gpi", LONG_ITEM_CASES)
def test_ring_long_items(orc, dims, gpi):
    """Bit for bit with integer inputs, full output, at the plan the library
    takes on a device of 256 compute units (checked against the plan model)."""
    n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w = dims
    o_h, o_w = i_h - k_h + 1, i_w - k_w + 1
    KR = k_h * k_w * i_c
    bs = ring_block_steps(KR)
    slots = 8 * torch.cuda.get_device_properties(0).multi_processor_count
    plan = ring_plan(-(-n * o_w // 8), -(-o_h // 4), 1, 1, slots, -(-((KR + 1) // 2) // bs) * bs)
    say("ring long items", dims, "plan", plan)
    if slots == 2048:
        assert plan[0] == gpi and plan[1] < slots and plan[2] == 0
    I, K = case(89 + sum(dims), dims, dist="int")
    ref = orc.conv2d_direct(host(I), host(K), s_h, s_w)
    assert np.abs(ref).max() < 2 ** 24
    assert np.array_equal(run_conv(I, K, s_h, s_w, "fused"), ref.astype(np.float32))


_SPLIT_TAIL = {}


@pytest.mark.parametrize("gpi", [1, 2, 3])
@pytest.mark.parametrize("k_c", [96, 40])
@pytest.mark.parametrize("algo", ["lowered", "fused"])
def test_ring_split_tail(orc, gpi, k_c, algo):
    """The items past the last whole round of the wave slots (eight waves per
    compute unit) run one row group and 32-channel block per workgroup: full
    output compared bit for bit with integer inputs, at batches sized from the
    device's compute units so that such a remainder exists, with items of one
    row group (o_h = 10: three groups, the last one half full), of two (o_h =
    7: two groups, the second one three rows) and of three (o_h = 10). o_w = 7
    puts pair groups across images."""
    slots = 8 * torch.cuda.get_device_properties(0).multi_processor_count
    o_h = 7 if gpi == 2 else 10
    n, plan = ring_split_batch(slots, o_h, 7, k_c, gpi)
    dims = (n, 4 * o_h + 7, 35, 3, 11, 11, k_c, 4, 4)
    say("ring split tail", algo, dims, "plan", plan)
    I, K = case(83 + k_c + gpi, dims, dist="int")
    if (gpi, k_c) not in _SPLIT_TAIL:  # the oracle's result, shared by both algorithms
        _SPLIT_TAIL[(gpi, k_c)] = orc.conv2d_direct(host(I), host(K), 4, 4)
    ref = _SPLIT_TAIL[(gpi, k_c)]
    assert np.abs(ref).max() < 2 ** 24
    assert np.array_equal(run_conv(I, K, 4, 4, algo), ref.astype(np.float32))


# fp32 7x7 stride 2 tiles, rows per tile by the tile count: 2 rows split
# between two workgroups (few tiles), 2 rows unsplit (4-row tiles short of one
# per compute unit, 2-row tiles not), 4 rows (a tile per compute unit), with
# one and two channel tiles and ragged pairs, rows and channels. Bit for bit on
# integers (the split adds exactly two partial sums onto zero).
K7S2_CASES = [
    (2, 21, 19, 16, 7, 7, 40, 2, 2),      # 2 rows, split
    (3, 30, 31, 8, 7, 7, 100, 2, 2),      # 2 rows, split, two channel tiles
    (8, 100, 100, 8, 7, 7, 64, 2, 2),     # 2 rows: 144 4-row tiles, 288 2-row tiles
    (16, 100, 99, 8, 7, 7, 60, 2, 2),     # 4 rows: 288 tiles
    (8, 101, 100, 4, 7, 7, 100, 2, 2),    # 4 rows, two channel tiles
]


@pytest.mark.parametrize("dims", K7S2_CASES)
@pytest.mark.parametrize("algo", ["lowered", "fused"])
def test_k7s2_row_choice(orc, dims, algo):
    say("7x7 stride 2", algo, dims)
    s_h, s_w = dims[7], dims[8]
    Ii, Ki = case(107 + sum(dims), dims, dist="int")
    refi = orc.conv2d_direct(host(Ii), host(Ki), s_h, s_w)
    assert np.abs(refi).max() < 2 ** 24
    assert np.array_equal(run_conv(Ii, Ki, s_h, s_w, algo), refi.astype(np.float32))
    I, K = case(109 + sum(dims), dims)
    assert rel_l2(run_conv(I, K, s_h, s_w, algo), orc.conv2d_direct(host(I), host(K), s_h, s_w)) <= TOL_F32


# fp32 5x5 stride 1, rows per tile by the tile count: 2 rows split between two
# workgroups (few tiles), 2 rows unsplit, 4 rows; from L and from I (whose
# direct-to-LDS form needs rows of a multiple of 16), ragged pairs, rows and
# channels.
K5S1_CASES = [
    (1, 24, 24, 96, 5, 5, 256, 1, 1),     # 2 rows, split (40 tiles)
    (2, 15, 17, 8, 5, 5, 40, 1, 1),       # 2 rows, split, rows of 40
    (8, 24, 24, 96, 5, 5, 200, 1, 1),     # 2 rows (200 tiles), k_c ragged
    (32, 40, 39, 16, 5, 5, 64, 1, 1),     # 4 rows (315 tiles)
]


@pytest.mark.parametrize("dims", K5S1_CASES)
@pytest.mark.parametrize("algo", ["lowered", "fused"])
def test_k5s1_row_choice(orc, dims, algo):
    say("5x5 stride 1", algo, dims)
    s_h, s_w = dims[7], dims[8]
    Ii, Ki = case(113 + sum(dims), dims, dist="int")
    refi = orc.conv2d_direct(host(Ii), host(Ki), s_h, s_w)
    assert np.abs(refi).max() < 2 ** 24
    assert np.array_equal(run_conv(Ii, Ki, s_h, s_w, algo), refi.astype(np.float32))
    I, K = case(115 + sum(dims), dims)
    assert rel_l2(run_conv(I, K, s_h, s_w, algo), orc.conv2d_direct(host(I), host(K), s_h, s_w)) <= TOL_F32


# fp32 3x3 stride 2 tiles (32 pairs x 2 output rows, 5 staged rows): rows of
# a multiple of 4 (16-byte loads), short rows (element loads of I and L), k_c
# not a multiple of 4 (element loads of K), ragged pairs, rows and channels,
# s_w = 1.
K3S2_CASES = [
    (3, 21, 19, 64, 3, 3, 72, 2, 2),
    (2, 17, 18, 3, 3, 3, 40, 2, 2),
    (2, 15, 16, 5, 3, 3, 30, 2, 2),
    (2, 19, 20, 8, 3, 3, 64, 2, 1),
    (1, 9, 9, 128, 3, 3, 136, 2, 2),
]


@pytest.mark.parametrize("dims", K3S2_CASES)
@pytest.mark.parametrize("algo", ["lowered", "fused"])
def test_k3s2_tiles(orc, dims, algo):
    say("3x3 stride 2", algo, dims)
    s_h, s_w = dims[7], dims[8]
    Ii, Ki = case(101 + sum(dims), dims, dist="int")
    refi = orc.conv2d_direct(host(Ii), host(Ki), s_h, s_w)
    assert np.abs(refi).max() < 2 ** 24
    assert np.array_equal(run_conv(Ii, Ki, s_h, s_w, algo), refi.astype(np.float32))
    I, K = case(103 + sum(dims), dims)
    assert rel_l2(run_conv(I, K, s_h, s_w, algo), orc.conv2d_direct(host(I), host(K), s_h, s_w)) <= TOL_F32


# fp32 from L, kernels taller than one row with no tile of their own: the
# windows of Section 3.2's flat view as the rows of one plain product through
# the k_h = 1 tiles. Rows of a multiple of 4 (16-byte loads) and not, k_c
# above and below 64 and not a multiple of 4, ragged pairs and output rows,
# windows overlapping by several rows (stride 1, 2) or none (stride = k_h).
FLAT_CASES = [
    (3, 21, 19, 64, 3, 3, 72, 2, 2),      # 3x3 stride 2, rows of 192
    (2, 25, 23, 32, 5, 5, 30, 2, 2),      # 5x5 stride 2, k_c not a multiple of 4
    (3, 18, 20, 16, 2, 2, 128, 2, 2),     # 2x2 stride 2: windows side by side
    (1, 31, 29, 3, 11, 11, 96, 1, 1),     # 11x11 stride 1 (rows of 33: element loads)
    (2, 33, 35, 3, 11, 11, 40, 2, 3),     # 11x11 stride 2
    (2, 45, 41, 3, 11, 11, 100, 5, 5),    # 11x11 stride 5: beyond the ring
    (2, 30, 28, 16, 7, 7, 64, 1, 1),      # 7x7 stride 1
    (3, 20, 22, 5, 3, 3, 9, 3, 3),        # 3x3 stride 3, rows of 15
    (2, 15, 14, 64, 1, 1, 40, 2, 2),      # 1x1 stride 2: every other row of L
]


@pytest.mark.parametrize("dims", FLAT_CASES)
@pytest.mark.parametrize("algo", ["lowered", "fused"])
def test_flat_window_products(orc, dims, algo):
    """From L the flat windows; from I the same shapes take the generic kernel
    (2-row tiles first where the kernel fits them) or the 3x3 stride-2 tiles."""
    say("flat windows", algo, dims)
    s_h, s_w = dims[7], dims[8]
    Ii, Ki = case(91 + sum(dims), dims, dist="int")
    refi = orc.conv2d_direct(host(Ii), host(Ki), s_h, s_w)
    assert np.abs(refi).max() < 2 ** 24
    assert np.array_equal(run_conv(Ii, Ki, s_h, s_w, algo), refi.astype(np.float32))
    I, K = case(93 + sum(dims), dims)
    assert rel_l2(run_conv(I, K, s_h, s_w, algo), orc.conv2d_direct(host(I), host(K), s_h, s_w)) <= TOL_F32


# bf16 from L, windows overlapping most (k_h >= 5 s_h) with no tile of their
# own: the flat windows gathered element by element (96 channels or fewer, or
# 128-channel tiles) or in 16-byte pieces (length and strides multiples of 8).
FLAT_CASES_BF16 = [
    (2, 25, 23, 3, 11, 11, 40, 1, 1),     # 11x11 stride 1, windows of 363
    (1, 30, 20, 8, 11, 3, 136, 2, 2),     # windows of 264, 16-byte pieces, two channel tiles
    (2, 24, 20, 5, 10, 3, 104, 2, 1),     # windows of 150, gathered, one ragged channel tile
]


@pytest.mark.parametrize("dims", FLAT_CASES_BF16)
def test_flat_window_products_bf16(orc, dims):
    say("flat windows bf16", dims)
    s_h, s_w = dims[7], dims[8]
    Ii, Ki = case(95 + sum(dims), dims, dtype="bf16", dist="int")
    refi = orc.conv2d_direct(host(Ii), host(Ki), s_h, s_w)
    assert np.abs(refi).max() < 2 ** 24
    assert np.array_equal(run_conv(Ii, Ki, s_h, s_w, "lowered"), refi.astype(np.float32))
    I32, K32 = case(97 + sum(dims), dims, dtype="f32")
    I, K = I32.to(torch.bfloat16), K32.to(torch.bfloat16)
    got = run_conv(I, K, s_h, s_w, "lowered")
    assert rel_l2(got, orc.conv2d_direct(host(I), host(K), s_h, s_w)) <= TOL_F32
    assert rel_l2(got, orc.conv2d_direct(host(I32), host(K32), s_h, s_w)) <= TOL_BF16_VS_F32


@pytest.mark.parametrize("shift", [1, 3])
@pytest.mark.parametrize("which", ["long", "short"])
def test_ring_unaligned_and_guarded(orc, shift, which):
    """I, K, L and O one or three elements off their 16-byte boundaries, O
    inside a guard band: element loads and stores only, nothing written
    outside O. An 11x11 stride-4 window, and a short one (3x3 over 3
    channels, three channel blocks)."""
    dims = RING_CASES[2] if which == "long" else SHORT_RING_CASES[0]
    s_h, s_w = dims[7], dims[8]
    say("ring unaligned", which, shift, dims)
    I, K = case(79 + shift, dims, dist="int")
    ref = orc.conv2d_direct(host(I), host(K), s_h, s_w).astype(np.float32)

    def offset_copy(t):
        buf = torch.zeros(t.numel() + 8, dtype=t.dtype, device=DEV)
        v = buf[shift:shift + t.numel()].view(t.shape)
        v.copy_(t.to(DEV))
        return v

    Id, Kd = offset_copy(I), offset_copy(K)
    buf = torch.full((ref.size + 64,), 7.0, dtype=torch.float32, device=DEV)
    Od = buf[32 + shift:32 + shift + ref.size].view(ref.shape)
    ws = torch.zeros(mec.workspace_bytes(*dims) + 64, dtype=torch.uint8, device=DEV)[4 * shift:]
    for algo in ("lowered", "fused"):
        buf.fill_(7.0)
        mec.conv2d(Id, Kd, s_h, s_w, algo=algo, O=Od, workspace=ws)
        torch.cuda.synchronize()
        b = buf.cpu().numpy()
        assert np.all(b[:32 + shift] == 7.0) and np.all(b[32 + shift + ref.size:] == 7.0), algo
        assert np.array_equal(Od.cpu().numpy(), ref), algo


# bf16 tiles staged by direct-to-LDS loads (rows of a multiple of 32): 3x3 in
# the 14-row form where its tiles fill at least 192 compute units, else 2
# rows; 5x5.
DMA_CASES_BF16 = [
    (95, 20, 19, 32, 3, 3, 136, 1, 1),   # 14 rows: 204 tiles; ragged pairs (1615), rows (18), channels
    (3, 13, 11, 64, 3, 3, 72, 1, 1),     # 2 rows: ragged pairs, odd row count, one ragged channel tile
    (2, 9, 10, 128, 3, 3, 264, 1, 1),    # 2 rows: three channel tiles, the last 8 wide
    (3, 17, 21, 32, 5, 5, 72, 1, 1),     # 5x5: ragged pairs, rows, channels
]


def tiles14(dims):
    i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w = dims
    o_h, o_w = mec.output_dims(i_h, i_w, k_h, k_w, s_h, s_w)
    return -(-i_n * o_w // 32) * -(-o_h // 14) * -(-k_c // 128)


@pytest.mark.parametrize("dims", DMA_CASES_BF16)
@pytest.mark.parametrize("algo", ["lowered", "fused"])
def test_bf16_direct_to_lds_tiles(orc, dims, algo):
    say("bf16 dma", algo, dims)
    assert (dims[5] * dims[3]) % 32 == 0
    assert (tiles14(dims) >= 192) == (dims == DMA_CASES_BF16[0])
    s_h, s_w = dims[7], dims[8]
    Ii, Ki = case(53 + sum(dims), dims, dtype="bf16", dist="int")
    refi = orc.conv2d_direct(host(Ii), host(Ki), s_h, s_w)
    assert np.abs(refi).max() < 2 ** 24
    assert np.array_equal(run_conv(Ii, Ki, s_h, s_w, algo), refi.astype(np.float32))
    I32, K32 = case(59 + sum(dims), dims, dtype="f32")
    I, K = I32.to(torch.bfloat16), K32.to(torch.bfloat16)
    got = run_conv(I, K, s_h, s_w, algo)
    assert rel_l2(got, orc.conv2d_direct(host(I), host(K), s_h, s_w)) <= TOL_F32
    assert rel_l2(got, orc.conv2d_direct(host(I32), host(K32), s_h, s_w)) <= TOL_BF16_VS_F32


SPLIT_CASES_BF16 = [
    (2, 7, 7, 512, 3, 3, 512, 1, 1),     # 12 tiles of 48 r-chunks
    (3, 9, 8, 256, 3, 3, 136, 1, 1),     # ragged channel tile
]


@pytest.mark.parametrize("dims", SPLIT_CASES_BF16)
@pytest.mark.parametrize("algo", ["lowered", "fused"])
def test_split_reduction_bf16(orc, dims, algo):
    say("split bf16", algo, dims)
    s_h, s_w = dims[7], dims[8]
    I32, K32 = case(41 + sum(dims), dims, dtype="f32")
    I, K = I32.to(torch.bfloat16), K32.to(torch.bfloat16)
    ref = orc.conv2d_direct(host(I), host(K), s_h, s_w)
    O1 = run_conv(I, K, s_h, s_w, algo)
    assert rel_l2(O1, ref) <= TOL_F32
    assert np.array_equal(run_conv(I, K, s_h, s_w, algo), O1)
    Ii, Ki = case(43 + sum(dims), dims, dtype="bf16", dist="int")
    refi = orc.conv2d_direct(host(Ii), host(Ki), s_h, s_w)
    assert np.abs(refi).max() < 2 ** 24
    assert np.array_equal(run_conv(Ii, Ki, s_h, s_w, algo), refi.astype(np.float32))


def test_split_reduction_unaligned_o(orc):
    """O off its 16-byte boundary: element atomics, nothing written outside O."""
    dims = SPLIT_CASES[0]
    say("split unaligned", dims)
    I, K = case(37, dims, dist="int")
    ref = orc.conv2d_direct(host(I), host(K), 1, 1).astype(np.float32)
    buf = torch.full((ref.size + 64,), 7.0, dtype=torch.float32, device=DEV)
    O = buf[33:33 + ref.size].view(ref.shape)
    for algo in ("lowered", "fused"):
        mec.conv2d(to_dev(I), to_dev(K), 1, 1, algo=algo, O=O)
        torch.cuda.synchronize()
        b = buf.cpu().numpy()
        assert np.all(b[:33] == 7.0) and np.all(b[33 + ref.size:] == 7.0)
        assert np.array_equal(O.cpu().numpy(), ref), algo


def im2col_ref(orc, I, k_h, k_w, s_h, s_w):
    """The oracle's im2col (rows n, y, x) reordered to the library's (n, x, y)."""
    i_n, i_h, i_w, i_c = I.shape
    o_h, o_w = orc.out_dim(i_h, k_h, s_h), orc.out_dim(i_w, k_w, s_w)
    M = orc.im2col(host(I), k_h, k_w, s_h, s_w).reshape(i_n, o_h, o_w, k_h, k_w, i_c)
    return np.ascontiguousarray(M.transpose(0, 2, 1, 3, 4, 5))


@pytest.mark.parametrize("dims", SWEEP + SWEEP_BF16)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_im2col_bitwise_sweep(orc, dims, dtype):
    say("im2col", dtype, dims)
    I, _ = case(13 * sum(dims), dims, dtype=dtype)
    k_h, k_w, k_c, s_h, s_w = dims[4:]
    ref = im2col_ref(orc, I, k_h, k_w, s_h, s_w)
    M = mec.im2col(to_dev(I), k_h, k_w, k_c, s_h, s_w)
    torch.cuda.synchronize()
    got = host(M.cpu())
    assert got.shape == ref.shape and np.array_equal(got, ref)


@pytest.mark.parametrize("dims", SWEEP + SWEEP_BF16)
def test_conv_im2col_baseline(orc, dims):
    """The im2col + product baseline computes the same convolution."""
    say("conv im2col", dims)
    I, K = case(17 + sum(dims), dims, dist="int")
    s_h, s_w = dims[7], dims[8]
    ref = orc.conv2d_direct(host(I), host(K), s_h, s_w)
    got = run_conv(I, K, s_h, s_w, "im2col")
    assert np.array_equal(got, ref.astype(np.float32))
    Ib, Kb = I.to(torch.bfloat16), K.to(torch.bfloat16)
    refb = orc.conv2d_direct(host(Ib), host(Kb), s_h, s_w)
    assert np.array_equal(run_conv(Ib, Kb, s_h, s_w, "im2col"), refb.astype(np.float32))


@pytest.mark.parametrize("dims", [
    (1, 40, 30, 256, 3, 3, 8, 1, 1),      # fp32 runs of 3 KB: output rows split in blocks
    (2, 50, 20, 300, 5, 2, 4, 3, 2),      # blocks with stride 3, runs not 16-byte multiples
    (1, 30, 12, 2000, 3, 4, 3, 1, 3),     # runs of 8000 elements: only a few rows per block
])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_im2col_row_blocks(orc, dims, dtype):
    say("im2col row blocks", dtype, dims)
    I, _ = case(29 + sum(dims), dims, dtype=dtype)
    k_h, k_w, k_c, s_h, s_w = dims[4:]
    ref = im2col_ref(orc, I, k_h, k_w, s_h, s_w)
    M = mec.im2col(to_dev(I), k_h, k_w, k_c, s_h, s_w)
    torch.cuda.synchronize()
    assert np.array_equal(host(M.cpu()), ref)


def test_im2col_workspace_holds_M(orc):
    dims = (3, 20, 21, 16, 3, 3, 40, 1, 2)
    say("im2col workspace", dims)
    I, K = case(23, dims)
    k_h, k_w, k_c, s_h, s_w = dims[4:]
    ws = torch.empty(mec.workspace_bytes(*dims, algo=mec.IM2COL), dtype=torch.uint8, device=DEV)
    O = mec.conv2d(to_dev(I), to_dev(K), s_h, s_w, algo="im2col", workspace=ws)
    torch.cuda.synchronize()
    ref_M = im2col_ref(orc, I, k_h, k_w, s_h, s_w)
    assert np.array_equal(ws.cpu().numpy().view(np.float32).reshape(ref_M.shape), ref_M)
    ref = orc.conv2d_direct(host(I), host(K), s_h, s_w)
    assert rel_l2(O.cpu().numpy(), ref) <= TOL_F32


@pytest.mark.parametrize("shift", [1, 2, 3])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_unaligned_tensors(orc, shift, dtype):
    """Tensors that start off a 16-byte boundary take the element-wise paths."""
    dims = (2, 19, 17, 64, 3, 3, 64, 1, 1)
    say("unaligned", dtype, shift, dims)
    I, K = case(99, dims, dtype=dtype, dist="int")
    k_h, k_w, k_c, s_h, s_w = dims[4:]
    tdt = I.dtype

    def offset_copy(t):
        buf = torch.zeros(t.numel() + 8, dtype=tdt, device=DEV)
        v = buf[shift:shift + t.numel()].view(t.shape)
        v.copy_(t.to(DEV))
        return v

    Id, Kd = offset_copy(I), offset_copy(K)
    assert Id.data_ptr() % 16 != 0
    Lbuf = torch.zeros(orc.lowered_elems(*dims) + 8, dtype=tdt, device=DEV)
    Ld = Lbuf[shift:shift + orc.lowered_elems(*dims)]
    mec.lower(Id, k_h, k_w, k_c, s_h, s_w, L=Ld)
    ref_L = orc.mec_lower(host(I), k_h, k_w, k_c, s_h, s_w)
    ref = orc.conv2d_direct(host(I), host(K), s_h, s_w).astype(np.float32)
    Obuf = torch.zeros(ref.size + 8, dtype=torch.float32, device=DEV)
    Od = Obuf[shift:shift + ref.size].view(ref.shape)
    es = 2 if dtype == "bf16" else 4
    ws = torch.zeros(mec.workspace_bytes(*dims, dtype=mec.BF16 if dtype == "bf16" else mec.F32)
                     + 64, dtype=torch.uint8, device=DEV)[es * shift:]
    torch.cuda.synchronize()
    assert np.array_equal(host(Ld.cpu()).reshape(ref_L.shape), ref_L)
    for algo in ("lowered", "fused"):
        Od.zero_()
        mec.conv2d(Id, Kd, s_h, s_w, algo=algo, O=Od, workspace=ws)
        torch.cuda.synchronize()
        assert np.array_equal(Od.cpu().numpy(), ref), algo
    # im2col baseline on the same unaligned tensors
    nM = orc.im2col_elems(*dims)
    Md = torch.zeros(nM + 8, dtype=tdt, device=DEV)[shift:shift + nM]
    mec.im2col(Id, k_h, k_w, k_c, s_h, s_w, M=Md)
    torch.cuda.synchronize()
    ref_M = im2col_ref(orc, I, k_h, k_w, s_h, s_w)
    assert np.array_equal(host(Md.cpu()).reshape(ref_M.shape), ref_M)
    wsM = torch.zeros(nM * es + 64, dtype=torch.uint8, device=DEV)[es * shift:]
    Od.zero_()
    mec.conv2d(Id, Kd, s_h, s_w, algo="im2col", O=Od, workspace=wsM)
    torch.cuda.synchronize()
    assert np.array_equal(Od.cpu().numpy(), ref), "im2col"


@pytest.mark.parametrize("dims", SWEEP[:8])
def test_workspace_holds_L_and_gemm_alone(orc, dims):
    say("workspace/gemm", dims)
    I, K = case(2 * sum(dims), dims)
    k_h, k_w, k_c, s_h, s_w = dims[4:]
    ws = torch.empty(mec.workspace_bytes(*dims), dtype=torch.uint8, device=DEV)
    O = mec.conv2d(to_dev(I), to_dev(K), s_h, s_w, algo="lowered", workspace=ws)
    ref_L = orc.mec_lower(host(I), k_h, k_w, k_c, s_h, s_w)
    torch.cuda.synchronize()
    assert np.array_equal(ws.cpu().numpy().view(np.float32).reshape(ref_L.shape), ref_L)
    # the product phase alone, on the oracle's L
    O2 = mec.gemm(to_dev(torch.from_numpy(ref_L)), to_dev(K), dims[1], dims[2], s_h, s_w)
    ref = orc.mec_gemm(ref_L, host(K), dims[1], dims[2], s_h, s_w)
    torch.cuda.synchronize()
    assert rel_l2(O2.cpu().numpy(), ref) <= TOL_F32
    assert np.array_equal(O2.cpu().numpy(), O.cpu().numpy())


def test_output_not_written_outside(orc):
    """O of a ragged shape written exactly in place: a guard band stays intact."""
    dims = (3, 31, 30, 3, 11, 11, 100, 4, 3)
    say("guard", dims)
    I, K = case(5, dims)
    ref = orc.conv2d_direct(host(I), host(K), dims[7], dims[8]).astype(np.float32)
    buf = torch.full((ref.size + 4096,), 7.0, dtype=torch.float32, device=DEV)
    O = buf[1024:1024 + ref.size].view(ref.shape)
    for algo in ("lowered", "fused"):
        mec.conv2d(to_dev(I), to_dev(K), dims[7], dims[8], algo=algo, O=O)
        torch.cuda.synchronize()
        b = buf.cpu().numpy()
        assert np.all(b[:1024] == 7.0) and np.all(b[1024 + ref.size:] == 7.0)
        assert rel_l2(O.cpu().numpy(), ref) <= TOL_F32


# ---------------------------------------------------------------- the five layers

LAYERS = wl.LAYER_ORDER


@pytest.mark.parametrize("name", LAYERS)
def test_layer_lower_full_bitwise(orc, name):
    layer = wl.LAYERS[name]
    say("layer lower full", name)
    I, _ = wl.make_inputs(layer)
    k_h, k_w, k_c, s_h, s_w = layer.dims[4:]
    Ld = mec.lower(to_dev(I), k_h, k_w, k_c, s_h, s_w)
    ref = orc.mec_lower(host(I), k_h, k_w, k_c, s_h, s_w)
    torch.cuda.synchronize()
    assert np.array_equal(host(Ld.cpu()), ref)


@pytest.mark.parametrize("name", LAYERS)
def test_layer_reduced_batch_full_compare(orc, name):
    """Full output compared at a batch of 2 (all spatial tiles, ragged edges)."""
    layer = wl.LAYERS[name]
    say("layer reduced batch", name)
    I, K = wl.make_inputs(layer, i_n=min(2, layer.i_n))
    s_h, s_w = layer.s_h, layer.s_w
    ref = orc.conv2d_direct(host(I), host(K), s_h, s_w)
    ref32 = None
    if layer.dtype == "bf16":
        # the 1e-2 bar is sized for the fp32 values before rounding to bf16
        I32, K32 = wl.make_inputs(layer, i_n=min(2, layer.i_n), round_bf16=False)
        assert torch.equal(I32.to(torch.bfloat16), I)
        ref32 = orc.conv2d_direct(host(I32), host(K32), s_h, s_w)
    for algo in ("lowered", "fused"):
        got = run_conv(I, K, s_h, s_w, algo)
        assert rel_l2(got, ref) <= TOL_F32, algo
        if ref32 is not None:
            assert rel_l2(got, ref32) <= TOL_BF16_VS_F32, algo


@pytest.mark.parametrize("name", LAYERS)
def test_layer_full_size_sampled(orc, name):
    """Full-size layers in the benchmark's launch configuration, checked on
    sampled outputs the oracle computes one by one (corners included), and
    LOWERED == FUSED bit for bit (same staged values, same reduction order)
    where both take the same kernel."""
    layer = wl.LAYERS[name]
    say("layer full sampled", name)
    I, K = wl.make_inputs(layer)
    s_h, s_w = layer.s_h, layer.s_w
    Id, Kd = to_dev(I), to_dev(K)
    O1 = mec.conv2d(Id, Kd, s_h, s_w, algo="lowered")
    O2 = mec.conv2d(Id, Kd, s_h, s_w, algo="fused")
    torch.cuda.synchronize()
    shape = tuple(O1.shape)
    rng = np.random.default_rng(layer.seed)
    idx = np.stack([rng.integers(0, d, 3000) for d in shape], axis=1)
    corners = np.array([[n, y, x, m] for n in (0, shape[0] - 1) for y in (0, shape[1] - 1)
                        for x in (0, shape[2] - 1) for m in (0, shape[3] - 1)])
    idx = np.concatenate([idx, corners])
    ref = orc.conv2d_points(host(I), host(K), s_h, s_w, idx)
    g1 = O1.cpu().numpy()
    assert rel_l2(g1[tuple(idx.T)], ref) <= TOL_F32
    i_n, i_h, i_w, i_c, k_h, k_w, k_c, _, _ = layer.dims
    KR = k_h * k_w * i_c
    short = -(-((KR + 1) // 2) // ring_block_steps(KR)) <= 2
    if layer.dtype == "f32" and 3 <= k_h < 9 and s_h == 1 and k_w * i_c <= 10 and not short:
        # rows of at most 10 elements and windows longer than two blocks:
        # fused through the ring kernel, from L through the streaming kernel --
        # the same sums in another order
        assert rel_l2(O2.cpu().numpy(), g1) <= TOL_F32
    else:
        assert torch.equal(O1, O2)
    assert np.isfinite(g1).all()


def test_lowered_tensor_beyond_2_31_elements(orc):
    """A layer whose L has more than 2^31 elements (9.7 GB in fp32): the
    lowering and the products index it with 64-bit offsets. The first and the
    last image's L (the last starts past element 2^31) are compared with the
    oracle's lowering bit for bit; O on sampled outputs of every image, and
    LOWERED == FUSED there."""
    dims = (12, 1024, 1026, 64, 3, 3, 16, 1, 1)
    i_n, i_h, i_w, i_c, k_h, k_w, k_c, s_h, s_w = dims
    assert orc.lowered_elems(*dims) > 2 ** 31
    say("beyond 2^31", dims)
    g = torch.Generator(device=DEV).manual_seed(12)
    Id = torch.randint(-3, 4, (i_n, i_h, i_w, i_c), generator=g, device=DEV).float()
    Kd = torch.randint(-3, 4, (k_h, k_w, i_c, k_c), generator=g, device=DEV).float()
    ws = torch.empty(mec.workspace_bytes(*dims), dtype=torch.uint8, device=DEV)
    O1 = mec.conv2d(Id, Kd, s_h, s_w, algo="lowered", workspace=ws)
    O2 = mec.conv2d(Id, Kd, s_h, s_w, algo="fused")
    torch.cuda.synchronize()
    o_w = orc.out_dim(i_w, k_w, s_w)
    L = ws.view(torch.float32).view(i_n, o_w, i_h, k_w, i_c)
    I = Id.cpu().numpy()
    K = Kd.cpu().numpy()
    for n in (0, i_n - 1):
        ref_L = orc.mec_lower(np.ascontiguousarray(I[n:n + 1]), k_h, k_w, k_c, s_h, s_w)
        assert np.array_equal(L[n:n + 1].cpu().numpy(), ref_L), n
        del ref_L
    shape = tuple(O1.shape)
    rng = np.random.default_rng(5)
    idx = np.stack([rng.integers(0, d, 2000) for d in shape], axis=1)
    idx[:12, 0] = np.arange(12)
    ref = orc.conv2d_points(I, K, s_h, s_w, idx)
    sel = tuple(torch.from_numpy(idx.T.copy()).to(DEV))
    got1, got2 = O1[sel].cpu().numpy(), O2[sel].cpu().numpy()
    assert np.array_equal(got1, ref.astype(np.float32))
    assert np.array_equal(got1, got2)


# ---------------------------------------------------------------- Table 2 and the stride sweep

@pytest.mark.parametrize("name", list(wl.TABLE2))
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_table2_layer_all_algos_bitwise(orc, name, dtype):
    """Each benchmark layer of Table 2 (batch 1, small-integer inputs): MEC from
    L, MEC fused and the im2col baseline all equal the oracle bit for bit."""
    layer = wl.table2_layer(name, i_n=1, dtype=dtype, dist="int")
    say("table2", name, dtype, layer.dims)
    I, K = wl.make_inputs(layer)
    s = layer.s_h
    ref = orc.conv2d_direct(host(I), host(K), s, s)
    assert np.abs(ref).max() < 2 ** 24
    for algo in ("lowered", "fused", "im2col"):
        assert np.array_equal(run_conv(I, K, s, s, algo), ref.astype(np.float32)), algo


@pytest.mark.parametrize("name", ["cv1", "cv4", "cv5", "cv12"])
def test_table2_layer_float_inputs(orc, name):
    layer = wl.table2_layer(name, i_n=2)
    say("table2 float", name, layer.dims)
    I, K = wl.make_inputs(layer)
    s = layer.s_h
    ref = orc.conv2d_direct(host(I), host(K), s, s)
    for algo in ("lowered", "fused", "im2col"):
        assert rel_l2(run_conv(I, K, s, s, algo), ref) <= TOL_F32, algo


@pytest.mark.parametrize("stride", list(range(1, 11)))
def test_stride_sweep_cv1_bitwise(orc, stride):
    """cv1 with s = 1..10 (Fig. 4(a)), including s >= k_w / 2 and the strides
    where s does not divide i - k."""
    layer = wl.table2_layer("cv1", i_n=1, stride=stride, dist="int")
    say("stride sweep", stride, layer.dims)
    I, K = wl.make_inputs(layer)
    ref = orc.conv2d_direct(host(I), host(K), stride, stride).astype(np.float32)
    for algo in ("lowered", "fused", "im2col"):
        assert np.array_equal(run_conv(I, K, stride, stride, algo), ref), algo
