"""The stream-K GEMM schedule's arithmetic, modelled on the host.

The kernels (gemm.hip: sk_plan, sk_range, sk_owner, sk_next_item and k_gemm_fix's contributor
walk) split T tiles of nk K steps over P workgroups: whole data-parallel units first, then a
stream-K tail over the first Pk workgroups, whose range cuts leave fp32 partial tiles that the fixup
adds.  This model restates those formulas and checks, for fixed and random (T, P, nk), that every
(tile, K step) is computed exactly once, that every partial slot is written once and read by exactly
the fixup of its tile, and that the fixup's pieces of a tile cover K in order.  The plan's whole-tile
rules (one short wave, whole waves of 256 x 256 tiles) give an empty tail and are not modelled.
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


def test_mlp_up_tail_goes_to_fewer_workgroups():
    # 528 tiles on 256 workgroups: two whole waves, then 16 tiles x 48 steps over 64 workgroups
    s, U, dp, ln, I, Pk = plan(528, 256, 48)
    assert (s, dp, ln, I, Pk) == (1, 512, 48, 768, 64)


def test_schedule_random_cases():
    r = random.Random(0)
    for _ in range(600):
        check(r.randint(0, 700), r.choice([1, 2, 7, 64, 255, 256]), r.randint(1, 200))


# The column split of a two-launch projection (gemm.hip: col_range): R row tiles of 256 rows, N
# columns, P workgroups.  Phase 1 takes [0, split) in 256 x 256 tiles, phase 2 [split, N) in
# 256 x 192 tiles.
def col_split(R, N, P):
    TN = -(-N // 256)
    split = N
    if R > 0 and P < R * TN <= 2 * P:
        ta = P // R
        if ta >= 1 and R * (-(-(N - ta * 256) // 192)) <= P:
            split = ta * 256
    return split


def test_qkv_split_at_the_64x64_workload():
    # 2254 image rows (9 tiles) + 512 text rows (2): 11 row tiles; QKV N = 9216 on 256 CUs
    split = col_split(11, 9216, 256)
    assert split == 23 * 256
    assert 11 * 23 == 253 and 11 * -(-(9216 - split) // 192) == 198
    # the MLP up projection (528 tiles, more than two waves) is not split
    assert col_split(11, 12288, 256) == 12288


@pytest.mark.parametrize("seed", range(100))
def test_col_split_partitions_the_columns_into_single_waves(seed):
    r = random.Random(seed)
    P = r.choice([64, 104, 256, 304])
    R = r.randint(1, 40)
    N = 64 * r.randint(1, 300)
    split = col_split(R, N, P)
    assert 0 < split <= N
    if split < N:
        # both launches are one wave of whole tiles, and together they cover every column once
        assert split % 256 == 0
        assert R * (split // 256) <= P
        assert R * -(-(N - split) // 192) <= P
        assert R * -(-N // 256) > P  # only a projection that needed a second wave is split
    else:
        assert not (P < R * -(-N // 256) <= 2 * P) or R * -(-(N - (P // R) * 256) // 192) > P or P // R < 1
