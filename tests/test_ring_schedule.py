"""CPU model of the ring kernel's memory schedule (paper_1706_06873_amd/csrc/
mec_gemm_ring.hip): the fills of each pair's ring of 8 chunks of 64 elements,
the K loads, the O stores and the waits, replayed as one in-order queue of
vector memory operations ("s_waitcnt vmcnt(N)" retires all but the newest N,
the order in which the hardware counter retires loads, direct-to-LDS loads
and stores). Every ring read of every block must find its chunk in its slot,
filled and landed, and every wait count must fit the 6-bit counter. The model
follows the kernel's rules for both schedules: windows of more than two blocks
(fills one block ahead, a full wait at each block) and short windows (K held in
registers, fills five blocks ahead, waits counted per block). Runs on the CPU.
"""
import pytest

RP, RR, CH, NCH = 8, 4, 64, 8      # pairs, output rows per group, chunk, chunks per ring
LEAD = 5                           # short windows: blocks of lead


def block_steps(KR):
    st = (KR + 1) // 2
    return 7 if (st + 6) // 7 * 7 < (st + 7) // 8 * 8 else 8


def geometry(k_h, R, s_h):
    KR = k_h * R
    bs = block_steps(KR)
    nks = ((KR + 1) // 2 + bs - 1) // bs * bs
    return KR, bs, nks, nks // bs, s_h * R


def usable(k_h, R, s_h):
    KR, bs, nks, nblk, srow = geometry(k_h, R, s_h)
    if (RR - 1) * srow + 4 * bs + 62 > CH * NCH - 1:
        return False
    return 2 * (nks - bs) <= RR * srow


class Queue:
    def __init__(self):
        self.ops, self.landed, self.slot = [], set(), [-1] * NCH

    def fill(self, c):
        self.slot[c % NCH] = c
        self.landed.discard(c)
        self.ops += [("F", c)] * RP

    def other(self, n):
        self.ops += [("X", None)] * n

    def wait(self, n):
        assert 0 <= n <= 63
        while len(self.ops) > n:
            kind, c = self.ops.pop(0)
            if kind == "F":
                self.landed.add(c)


def check_reads(q, g, b, bs, srow):
    for u in range(bs):
        for ii in range(RR):
            for kofs in range(2):
                c = (g * RR * srow + ii * srow + 2 * (b * bs + u) + kofs) // CH
                assert q.slot[c % NCH] == c, ("overwritten or never filled", c, g, b)
                assert c in q.landed, ("read before it landed", c, g, b)


def long_item(k_h, R, s_h, o_h, g_begin, g_end, NB):
    """ring_item without SHORT: K loaded one block ahead, a full wait at each block."""
    KR, bs, nks, nblk, srow = geometry(k_h, R, s_h)
    lo = lambda g, b: (g * RR * srow + 2 * bs * b) // CH
    hi = lambda g, b: (g * RR * srow + (RR - 1) * srow + 2 * bs * b + 2 * bs - 1) // CH
    q, filled = Queue(), [lo(g_begin, 0) - 1]

    def fill_upto(t):
        for c in range(filled[0] + 1, t + 1):
            q.fill(c)
        filled[0] = max(filled[0], t)

    q.other(bs * NB)
    fill_upto(min(hi(g_begin, 1 if nblk > 1 else 0), lo(g_begin, 0) + NCH - 1))
    q.wait(0)
    for g in range(g_begin, g_end):
        for b in range(nblk):
            if b > 0 or g > g_begin:
                q.wait(0)
            if filled[0] < hi(g, b):
                fill_upto(hi(g, b))
                q.wait(0)
            q.other(bs * NB)
            if b + 1 < nblk:
                fill_upto(min(hi(g, b + 1), lo(g, b) + NCH - 1))
            check_reads(q, g, b, bs, srow)
        if g + 1 < g_end:
            fill_upto(min(hi(g + 1, 1 if nblk > 1 else 0), lo(g + 1, 0) + NCH - 1))
        q.other(min(RR, o_h - g * RR) * 4 * NB)
    q.wait(0)


def short_item(k_h, R, s_h, o_h, g_begin, g_end, NB):
    """ring_item with SHORT: K held for the item, fills LEAD blocks ahead, counted waits."""
    KR, bs, nks, nblk, srow = geometry(k_h, R, s_h)
    assert nblk <= 2
    nbeta = (g_end - g_begin) * nblk
    gb = lambda beta: (g_begin + beta // nblk, beta % nblk)
    lo = lambda beta: (gb(beta)[0] * RR * srow + 2 * bs * gb(beta)[1]) // CH
    hi = lambda beta: (gb(beta)[0] * RR * srow + (RR - 1) * srow + 2 * bs * gb(beta)[1] + 2 * bs - 1) // CH
    q, filled = Queue(), [lo(0) - 1]

    def fill_upto(t):
        n = max(0, t - filled[0])
        for c in range(filled[0] + 1, t + 1):
            q.fill(c)
        filled[0] = max(filled[0], t)
        return RP * n

    q.other(2 * bs * NB)
    fill_upto(min(hi(min(LEAD - 1, nbeta - 1)), lo(0) + NCH - 1))
    q.wait(0)
    mark, nops = [filled[0]] * LEAD, [0] * LEAD
    for beta in range(nbeta):
        g, b = gb(beta)
        n, later = -1, 0
        for i in range(LEAD - 1, -1, -1):
            if hi(beta) <= mark[i]:
                n = later
            later += nops[i]
        ops = 0
        if n >= 0:
            q.wait(min(n >> 3, 7) * 8)
        else:
            ops += fill_upto(hi(beta))
            q.wait(0)
        ops += fill_upto(min(hi(min(beta + LEAD, nbeta - 1)), lo(beta) + NCH - 1))
        check_reads(q, g, b, bs, srow)
        if b + 1 == nblk:
            rows = min(RR, o_h - g * RR)
            q.other(rows * 4 * NB)
            ops += rows * 4 * NB
        mark, nops = mark[1:] + [filled[0]], nops[1:] + [ops]
    q.wait(0)


def shapes(short):
    """(k_h, R, s_h, o_h) the ring accepts, with two heights: a few groups and
    enough for items of up to 16 groups."""
    out = []
    for k_h in range(2, 24):
        for R in (1, 3, 5, 8, 9, 10, 21, 33, 48):
            for s_h in (1, 2, 3, 4, 8, 16):
                if not usable(k_h, R, s_h):
                    continue
                if (geometry(k_h, R, s_h)[3] <= 2) != short:
                    continue
                for o_h in (6, 66):
                    out.append((k_h, R, s_h, o_h))
    return out


@pytest.mark.parametrize("short", [False, True])
def test_ring_schedule_reads_land_before_use(short):
    item = short_item if short else long_item
    cases = shapes(short)
    assert len(cases) > 50
    for k_h, R, s_h, o_h in cases:
        ngroups = (o_h + RR - 1) // RR
        for NB in (1, 3):
            for gpi in (1, 2, 7, 16):
                for g0 in range(0, ngroups, gpi):
                    item(k_h, R, s_h, o_h, g0, min(g0 + gpi, ngroups), NB)


def test_ring_schedule_full_size_layers():
    """alexnet_conv1 (11x11 over 3 channels, stride 4: 14 groups, two-group
    items) and vgg_first (3x3 over 3 channels: 56 groups, 14-group items)."""
    for g0 in range(0, 14, 2):
        long_item(11, 33, 4, 55, g0, min(g0 + 2, 14), 3)
    for g0 in range(0, 56, 14):
        short_item(3, 9, 1, 224, g0, min(g0 + 14, 56), 2)


def test_ring_schedule_model_catches_a_late_wait():
    """The model is not vacuous: a queue whose waits retire nothing makes
    reads race their fills, and both schedules then fail; a lead of one block
    (the long schedule's) still passes the short schedule's wait rule."""
    global LEAD
    saved = LEAD
    try:
        LEAD = 1
        short_item(3, 9, 1, 224, 0, 14, 2)  # a lead of one block is still correct
    finally:
        LEAD = saved

    class Early(Queue):
        def wait(self, n):  # retires nothing: every read then races its fill
            assert 0 <= n <= 63

    original = Queue
    try:
        globals()["Queue"] = Early
        with pytest.raises(AssertionError):
            short_item(3, 9, 1, 224, 0, 14, 2)
        with pytest.raises(AssertionError):
            long_item(11, 33, 4, 55, 0, 2, 3)
    finally:
        globals()["Queue"] = original
