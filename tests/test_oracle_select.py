"""Pins of the oracle's score / select / compact / compress / decompress steps (CPU only).

Each test checks the oracle against something other than itself: hand-worked fixtures, textbook
closed forms, a library routine (scipy's Sobel filter and binary dilation), brute-force
enumeration on tiny grids, or an identity of the method.
"""
import os

import numpy as np
import pytest
from scipy import ndimage

from oracle import hilo_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _read_table(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(line)
    return rows


def _read_kv(name):
    out = {}
    for line in _read_table(name):
        k, *v = line.split()
        out[k] = np.array([float(t) for t in v])
    return out


# ---------------------------------------------------------------------------------------- score

def test_score_impulse_fixture():
    want = np.array([[int(t) for t in r.split()] for r in _read_table("sobel_impulse_5x5.txt")])
    x = np.zeros((1, 25, 1), np.float32)
    x[0, 2 * 5 + 2, 0] = 1.0
    E = O.score(x, 5, 5)
    np.testing.assert_array_equal(E.reshape(5, 5), want)


def test_score_constant_field_is_zero():
    x = np.full((2, 6 * 8, 5), 3.25, np.float32)
    assert (O.score(x, 6, 8) == 0).all()


@pytest.mark.parametrize("a", [0.5, 1.0, 0.125, 3.0])
def test_score_column_ramp_closed_form(a):
    # x = a * j: interior gx = 8a (1+2+1 rows times a 2a column difference), border columns see a
    # replicated neighbour so gx = 4a; gy = 0 everywhere.
    H, W = 5, 7
    j = np.arange(W, dtype=np.float32)
    x = np.broadcast_to(a * j[None, :, None], (H, W, 2)).reshape(1, H * W, 2).astype(np.float32)
    E = O.score(x, H, W).reshape(H, W)
    interior = 2 * int(np.floor((8 * a) ** 2 * 2 ** 16))
    border = 2 * int(np.floor((4 * a) ** 2 * 2 ** 16))
    assert (E[:, 1:-1] == interior).all()
    assert (E[:, 0] == border).all() and (E[:, -1] == border).all()


def test_score_row_ramp_is_transpose_of_column_ramp():
    H, W = 6, 6
    i = np.arange(H, dtype=np.float32)
    xr = np.broadcast_to(0.75 * i[:, None, None], (H, W, 3)).reshape(1, H * W, 3).astype(np.float32)
    xc = np.broadcast_to(0.75 * i[None, :, None], (H, W, 3)).reshape(1, H * W, 3).astype(np.float32)
    np.testing.assert_array_equal(O.score(xr, H, W).reshape(H, W), O.score(xc, H, W).reshape(H, W).T)


def test_score_matches_scipy_sobel_on_exact_integers():
    # Integer-valued fields keep every Sobel sum and square exact in float32, so the oracle must
    # agree bit for bit with scipy's Sobel filter (replicate border = mode "nearest").
    rng = np.random.default_rng(7)
    H, W, D = 9, 11, 6
    x = rng.integers(-40, 41, size=(H, W, D)).astype(np.float64)
    # scipy smooths along every axis but the derivative one, so filter each channel's 2-D plane
    gx = np.stack([ndimage.sobel(x[:, :, c], axis=1, mode="nearest") for c in range(D)], -1)
    gy = np.stack([ndimage.sobel(x[:, :, c], axis=0, mode="nearest") for c in range(D)], -1)
    v = np.minimum(gx * gx + gy * gy, 2.0 ** 22)
    want = np.floor(v * 2 ** 16).astype(np.int64).sum(-1)
    got = O.score(x.reshape(1, H * W, D).astype(np.float32), H, W).reshape(H, W)
    np.testing.assert_array_equal(got, want)


def test_score_channel_permutation_invariance():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((2, 8 * 6, 16)).astype(np.float32)
    E = O.score(x, 8, 6)
    perm = rng.permutation(16)
    np.testing.assert_array_equal(O.score(x[:, :, perm], 8, 6), E)


def test_score_cap_and_nan():
    x = np.zeros((1, 9, 2), np.float32)
    x[0, 4, 0] = 1e6      # huge edge: capped per channel at 2^22 * 2^16
    x[0, 4, 1] = np.nan   # NaN energy takes the cap as well
    E = O.score(x, 3, 3).reshape(3, 3)
    cap = 2 ** 38
    assert E[1, 1] == 0 or E[1, 1] == cap  # centre: gx = gy = 0 for channel 0; NaN for channel 1
    assert E[0, 1] == 2 * cap  # both channels capped on the impulse's upper neighbour


# ----------------------------------------------------------------------------------- select

def _fixture_case():
    kv = _read_kv("select_4x4.txt")
    E = kv["energy"].astype(np.int64).reshape(1, 16)
    force = kv["force"].astype(np.uint8).reshape(1, 16)
    return kv, E, force


def test_select_fixture_threshold():
    kv, E, force = _fixture_case()
    fine = O.select_threshold(E, force, 4, 4, 0, [0.09])
    np.testing.assert_array_equal(fine[0], kv["thr_fine_blocks"].astype(bool))
    idx_map, fine_idx, pool_idx, counts = O.compact(fine, 4, 4)
    np.testing.assert_array_equal(idx_map[0], kv["thr_idx_map"])
    np.testing.assert_array_equal(counts[0], kv["thr_counts"])
    fine = O.select_threshold(E, None, 4, 4, 0, [0.09])
    np.testing.assert_array_equal(fine[0], kv["thr_noforce_fine_blocks"].astype(bool))
    idx_map, _, _, counts = O.compact(fine, 4, 4)
    np.testing.assert_array_equal(idx_map[0], kv["thr_noforce_idx_map"])
    np.testing.assert_array_equal(counts[0], kv["thr_noforce_counts"])


def test_select_fixture_topk():
    kv, E, force = _fixture_case()
    np.testing.assert_array_equal(O.select_topk(E, force, 4, 4, 0, [3])[0],
                                  kv["topk3_fine_blocks"].astype(bool))
    fine = O.select_topk(E, None, 4, 4, 0, [3])
    np.testing.assert_array_equal(fine[0], kv["topk3_noforce_fine_blocks"].astype(bool))
    idx_map, _, _, counts = O.compact(fine, 4, 4)
    np.testing.assert_array_equal(idx_map[0], kv["topk3_noforce_idx_map"])
    np.testing.assert_array_equal(counts[0], kv["topk3_noforce_counts"])
    np.testing.assert_array_equal(O.select_topk(E, force, 4, 4, 0, [1])[0],
                                  kv["topk1_fine_blocks"].astype(bool))


@pytest.mark.parametrize("r", [0, 1, 2])
def test_dilation_matches_scipy(r):
    rng = np.random.default_rng(11 + r)
    f = (rng.random((3, 10, 12)) < 0.08)
    want = np.stack([ndimage.binary_dilation(fi, structure=np.ones((2 * r + 1, 2 * r + 1)))
                     if r > 0 else fi for fi in f])
    got = O.dilate(f.reshape(3, -1).astype(np.uint8), 10, 12, r, 3).reshape(3, 10, 12)
    np.testing.assert_array_equal(got, want)


def _random_energy(rng, G, H, W, ties=False):
    if ties:
        return rng.integers(0, 4, size=(G, H * W)).astype(np.int64)
    return rng.integers(0, 2 ** 40, size=(G, H * W)).astype(np.int64)


def _brute_topk(E, F, H, W, K):
    """Enumerate all K'-subsets of non-forced blocks on a tiny grid; the top-k set is the one whose
    sorted (B desc, index asc) key sequence is lexicographically smallest."""
    import itertools

    B = O.block_sums(E[None], H, W)[0]
    cand = [b for b in range(B.size) if not F[b]]
    k = max(0, K - int(F.sum()))
    best = None
    for sub in itertools.combinations(cand, min(k, len(cand))):
        key = sorted(((-B[b], b) for b in sub))
        if best is None or key < best[0]:
            best = (key, sub)
    fine = F.copy()
    for b in best[1]:
        fine[b] = True
    return fine


@pytest.mark.parametrize("seed", range(6))
def test_topk_brute_force(seed):
    rng = np.random.default_rng(100 + seed)
    H, W = 4, 6
    E = _random_energy(rng, 1, H, W, ties=seed % 2 == 0)
    force = (rng.random((1, H * W)) < 0.1).astype(np.uint8)
    F = O.forced_blocks(force, H, W, 0, 1)[0]
    for K in range(0, H * W // 4 + 1):
        got = O.select_topk(E, force, H, W, 0, [K])[0]
        np.testing.assert_array_equal(got, _brute_topk(E[0], F, H, W, K))
        assert got.sum() == max(K, F.sum())


@pytest.mark.parametrize("seed", range(4))
def test_threshold_brute_force_and_counts(seed):
    rng = np.random.default_rng(200 + seed)
    H, W = 6, 8
    E = _random_energy(rng, 2, H, W)
    force = (rng.random((2, H * W)) < 0.05).astype(np.uint8)
    tau = [0.2, 0.05]
    fine = O.select_threshold(E, force, H, W, 1, tau)
    dil = ndimage.binary_dilation(force.reshape(2, H, W)[0] > 0, structure=np.ones((3, 3)))
    for g in range(2):
        fg = ndimage.binary_dilation(force.reshape(2, H, W)[g] > 0, structure=np.ones((3, 3)))
        emax = E[g].max()
        for b in range(H * W // 4):
            I, J = divmod(b, W // 2)
            s = sum(int(E[g][(2 * I + di) * W + 2 * J + dj]) for di in (0, 1) for dj in (0, 1))
            forced = fg[2 * I:2 * I + 2, 2 * J:2 * J + 2].any()
            # mean normalised energy of the block exceeds tau
            assert fine[g][b] == (forced or (s / 4.0) / emax > tau[g] + 0.0) or \
                abs((s / 4.0) / emax - tau[g]) < 1e-12
    del dil
    idx_map, fine_idx, pool_idx, counts = O.compact(fine, H, W)
    NB = H * W // 4
    for g in range(2):
        n = int(fine[g].sum())
        assert counts[g, 0] == 4 * n and counts[g, 1] == NB - n
        assert counts[g].sum() == NB + 3 * n  # kept-token count equals the rule's count


def test_threshold_monotone_in_tau_and_flat_grid():
    rng = np.random.default_rng(5)
    E = _random_energy(rng, 1, 8, 8)
    prev = None
    for tau in [0.0, 0.05, 0.1, 0.2, 0.4, 0.8, 1.1]:
        f = O.select_threshold(E, None, 8, 8, 0, [tau])[0]
        if prev is not None:
            assert not (f & ~prev).any()  # raising tau never adds blocks
        prev = f
    assert not prev.any()  # tau > 1: no block's mean can exceed the maximum
    flat = np.zeros((1, 64), np.int64)
    force = np.zeros((1, 64), np.uint8)
    force[0, 9] = 1
    f = O.select_threshold(flat, force, 8, 8, 0, [0.0])[0]
    assert f.sum() == 1 and f[0]


def test_threshold_at_midpoint_equals_topk():
    # threshold at the midpoint between the k-th and (k+1)-th normalised block means selects exactly
    # the top-k set (two independent code paths of the oracle agree)
    rng = np.random.default_rng(9)
    H, W = 8, 10
    E = _random_energy(rng, 1, H, W)
    B = np.sort(O.block_sums(E, H, W)[0])[::-1] / 4.0 / E.max()
    for k in [1, 3, 7, 15]:
        tau = 0.5 * (B[k - 1] + B[k])
        np.testing.assert_array_equal(O.select_threshold(E, None, H, W, 0, [tau]),
                                      O.select_topk(E, None, H, W, 0, [k]))


def test_compact_edge_cases():
    H, W = 6, 4
    NB = H * W // 4
    allf = np.ones((1, NB), bool)
    idx_map, fine_idx, pool_idx, counts = O.compact(allf, H, W)
    np.testing.assert_array_equal(idx_map[0], np.arange(H * W))  # 0% compression: identity
    np.testing.assert_array_equal(counts[0], [H * W, 0])
    nonef = np.zeros((1, NB), bool)
    idx_map, fine_idx, pool_idx, counts = O.compact(nonef, H, W)
    np.testing.assert_array_equal(counts[0], [0, NB])
    np.testing.assert_array_equal(idx_map[0], O.block_of(H, W))
    # consistency of the three index arrays on a random selection
    rng = np.random.default_rng(1)
    fine = rng.random((3, NB)) < 0.5
    idx_map, fine_idx, pool_idx, counts = O.compact(fine, H, W)
    blk = O.block_of(H, W)
    for g in range(3):
        nf = counts[g, 0]
        for p in range(H * W):
            k = idx_map[g, p]
            if fine[g][blk[p]]:
                assert fine_idx[g, k] == p
            else:
                assert pool_idx[g, k - nf] == blk[p]
        assert (np.diff(fine_idx[g, :nf]) > 0).all()


def test_layout_offsets():
    counts = np.array([[8, 2], [4, 3], [0, 6], [12, 0]], np.int32)
    cu, seg = O.layout(counts, 2, 2, 5)
    np.testing.assert_array_equal(seg, [0, 10, 22, 28])
    np.testing.assert_array_equal(cu, [0, 22, 45])


# ------------------------------------------------------------------------ compress / decompress

def _pipeline_front(x, H, W, fine, B, I, L, x_txt):
    idx_map, fine_idx, pool_idx, counts = O.compact(fine, H, W)
    cu, seg = O.layout(counts, B, I, L)
    Z = O.compress(x, x_txt, H, W, fine_idx, pool_idx, counts, cu, seg, L)
    return Z, idx_map, cu, seg


def test_constant_blocks_pool_and_broadcast_losslessly():
    rng = np.random.default_rng(4)
    H, W, D, B, I, L = 6, 8, 5, 2, 2, 3
    G = B * I
    coarse = rng.standard_normal((G, H // 2, W // 2, D)).astype(np.float32)
    x = np.repeat(np.repeat(coarse, 2, axis=1), 2, axis=2).reshape(G, H * W, D)
    x_txt = rng.standard_normal((B, L, D)).astype(np.float32)
    fine = rng.random((G, H * W // 4)) < 0.4
    Z, idx_map, cu, seg = _pipeline_front(x, H, W, fine, B, I, L, x_txt)
    y_img, y_txt = O.decompress(Z, idx_map, cu, seg, L, B)
    np.testing.assert_array_equal(y_img, x)
    np.testing.assert_array_equal(y_txt, x_txt)


def test_fine_rows_are_copies_and_decompress_compress_identity():
    rng = np.random.default_rng(6)
    H, W, D, B, I, L = 8, 6, 4, 1, 2, 2
    G = B * I
    x = rng.standard_normal((G, H * W, D)).astype(np.float32)
    x_txt = rng.standard_normal((B, L, D)).astype(np.float32)
    fine = rng.random((G, H * W // 4)) < 0.5
    Z, idx_map, cu, seg = _pipeline_front(x, H, W, fine, B, I, L, x_txt)
    blk = O.block_of(H, W)
    y_img, y_txt = O.decompress(Z, idx_map, cu, seg, L, B)
    for g in range(G):
        fp = fine[g][blk]
        np.testing.assert_array_equal(y_img[g][fp], x[g][fp])
        # pooled patches carry the exact mean of their block
        for p in np.flatnonzero(~fp):
            i, j = divmod(p, W)
            i0, j0 = i - i % 2, j - j % 2
            m = (x[g][i0 * W + j0].astype(np.float64) + x[g][i0 * W + j0 + 1] + x[g][(i0 + 1) * W + j0]
                 + x[g][(i0 + 1) * W + j0 + 1]) / 4
            np.testing.assert_array_equal(y_img[g][p], m)
    # compressing the decompressed grid again reproduces Z exactly (broadcast rows re-pool to themselves)
    idx_map2, fine_idx, pool_idx, counts = O.compact(fine, H, W)
    Z2 = O.compress(y_img, y_txt, H, W, fine_idx, pool_idx, counts, cu, seg, L)
    np.testing.assert_array_equal(Z2, Z)
