"""The stream-K GEMM schedule's arithmetic, modelled on the host.

The kernels (gemm.hip: sk_plan, sk_range, sk_owner, sk_next_item and k_gemm_fix's contributor
walk) split T tiles of nk K steps over P workgroups: whole data-parallel units first, then a
stream-K tail over the first Pk workgroups, whose range cuts leave fp32 partial tiles that the fixup
adds.  This model restates those formulas and checks, for fixed and random (T, P, nk), that every
(tile, K step) is computed exactly once, that every partial slot is written once and read by exactly
the fixup of its tile, and that the fixup's pieces of a tile cover K in order.  The plan's whole-tile
rules (a short K with fewer tiles than workgroups, one wave at least 7/8 full, whole waves when the
last one is at least half full) give an empty tail; `whole_tiles` restates them.
"""
import random

import pytest

NO_SPLIT_STEPS = 64   # kNoSplitSteps
MIN_STEPS = 12        # kSkMinSteps


def plan(T, P, nk):
    if T < P and nk <= NO_SPLIT_STEPS:
        return 1, T, T, nk, 0, P
    s = 1 if (T >= P or T == 0) else min(-(-P // T), nk)
    U = T * s
    dp = U // P * P
    tail = U - dp
    pc = dp // T if tail > 0 else 0
    ln = (pc + 1) * nk // s - pc * nk // s
    I = tail * ln
    Pk = min(P, max(tail, -(-I // MIN_STEPS))) if I > 0 else P
    return s, U, dp, ln, I, Pk


def whole_tiles(T, P, nk):
    """True when the plan runs every tile whole (no K pieces, no stream-K tail)."""
    return (T < P and nk <= NO_SPLIT_STEPS) or (T >= P and 2 * (T % P) >= P) or (T < P and 8 * T >= 7 * P)


def rng(I, P, w):
    return I * w // P, I * (w + 1) // P


def owner(I, P, a):
    return ((a + 1) * P - 1) // I


def check(T, P, nk):
    s, U, dp, ln, I, Pk = plan(T, P, nk)
    ln = max(ln, 1)
    cover, slots, direct = {}, {}, set()
    for pid in range(P):
        u = pid
        b, e = rng(I, Pk, pid) if pid < Pk else (I, I)
        it = b
        while True:
            if u < dp:
                pc, t = divmod(u, T)
                kb, ke = pc * nk // s, (pc + 1) * nk // s
                slot = None if s == 1 else u
                u += P
            elif it < e:
                v = it // ln
                k0 = it - v * ln
                k1 = min(ln, k0 + e - it)
                pc, t = divmod(dp + v, T)
                base = pc * nk // s
                kb, ke = base + k0, base + k1
                whole = s == 1 and k0 == 0 and k1 == ln
                slot = None if whole else P + 2 * pid + (0 if it == b else 1)
                it += k1 - k0
            else:
                break
            assert 0 <= kb < ke <= nk
            for k in range(kb, ke):
                assert (t, k) not in cover
                cover[(t, k)] = pid
            if slot is None:
                direct.add(t)
            else:
                assert slot not in slots and slot < 3 * P
                slots[slot] = (t, kb, ke)
    assert len(cover) == T * nk
    read, fixed = set(), set()
    for f in range(T if s > 1 else U - dp):
        t = f if s > 1 else dp + f
        got, skip = [], False
        for pc in range(s):
            u = pc * T + t
            if u < dp:
                got.append(u)
                continue
            a0 = (u - dp) * ln
            w0, w1 = owner(I, Pk, a0), owner(I, Pk, a0 + ln - 1)
            if s == 1 and w0 == w1:
                skip = True
                break
            for w in range(w0, w1 + 1):
                b, e = rng(I, Pk, w)
                if b < e:
                    got.append(P + 2 * w + (0 if b // ln == u - dp else 1))
        if skip:
            assert t in direct
            continue
        ks = []
        for sl in got:
            assert sl in slots and slots[sl][0] == t and sl not in read
            read.add(sl)
            ks.append(slots[sl][1:])
        ks.sort()
        assert ks[0][0] == 0 and ks[-1][1] == nk
        assert all(ks[i][1] == ks[i + 1][0] for i in range(len(ks) - 1))
        assert t not in direct
        fixed.add(t)
    assert read == set(slots)
    assert fixed | direct == set(range(T)) and not (fixed & direct)


@pytest.mark.parametrize("T,P,nk", [(528, 256, 48), (396, 256, 48), (132, 256, 192), (1, 256, 128),
                                    (257, 256, 5), (3, 7, 100), (0, 256, 4), (100, 256, 65)])
def test_schedule_fixed_cases(T, P, nk):
    check(T, P, nk)


def test_short_tail_goes_to_fewer_workgroups():
    # 528 tiles on 256 workgroups: two whole waves, then 16 tiles x 48 steps over 64 workgroups
    assert not whole_tiles(528, 256, 48)
    s, U, dp, ln, I, Pk = plan(528, 256, 48)
    assert (s, dp, ln, I, Pk) == (1, 512, 48, 768, 64)


def test_projections_at_the_64x64_workload():
    # 2254 image rows (12 row tiles of 192) + 512 text rows (3): 15 row tiles, D = 3072, F = 12288,
    # 256 CUs.  QKV 720 tiles and MLP up 960 run whole waves (3 and 4, the last 208 and 192 tiles),
    # the attention output and MLP down 240 tiles in one wave (K = 3072: 48 steps; K = 12288: 192
    # steps, but the wave is more than 7/8 full)
    R = 12 + 3
    for N, K in [(3 * 3072, 3072), (12288, 3072), (3072, 3072), (3072, 12288)]:
        T = R * -(-N // 192)
        assert whole_tiles(T, 256, K // 64), (N, K)
    assert [R * -(-N // 192) for N in (9216, 12288, 3072)] == [720, 960, 240]


def test_schedule_random_cases():
    r = random.Random(0)
    for _ in range(600):
        check(r.randint(0, 700), r.choice([1, 2, 7, 64, 255, 256]), r.randint(1, 200))
