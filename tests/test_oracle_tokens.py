"""Token sets of the compressed grid (partition, overlap: every block's low-frequency token next to
the kept fine patches, drop: kept fine patches only) and the delta form of the reassembly, pinned
by a hand-worked example, count identities and closed forms."""
import numpy as np
import pytest

from oracle import hilo_oracle as O
from paper_2606_13898_amd import inputs


def test_hand_worked_4x4_index_maps():
    # 4x4 grid, blocks 0 and 3 kept: fine patches in raster order 0 1 4 5 10 11 14 15 (rows 0..7)
    fine = np.array([[True, False, False, True]])
    im, fi, pi, counts = O.compact(fine, 4, 4, "overlap")
    np.testing.assert_array_equal(im[0], [0, 1, 9, 9, 2, 3, 9, 9, 10, 10, 4, 5, 10, 10, 6, 7])
    np.testing.assert_array_equal(fi[0, :8], [0, 1, 4, 5, 10, 11, 14, 15])
    np.testing.assert_array_equal(pi[0], [0, 1, 2, 3])
    np.testing.assert_array_equal(counts[0], [8, 4])
    im, fi, pi, counts = O.compact(fine, 4, 4, "drop")
    np.testing.assert_array_equal(im[0], [0, 1, -1, -1, 2, 3, -1, -1, -1, -1, 4, 5, -1, -1, 6, 7])
    np.testing.assert_array_equal(counts[0], [8, 0])
    im, fi, pi, counts = O.compact(fine, 4, 4, "partition")
    np.testing.assert_array_equal(im[0], [0, 1, 8, 8, 2, 3, 8, 8, 9, 9, 4, 5, 9, 9, 6, 7])
    np.testing.assert_array_equal(counts[0], [8, 2])


@pytest.mark.parametrize("K", [0, 1, 7, 20])
def test_token_counts(K):
    shp = inputs.BlockShape(2, 1, 8, 10, 3, 32, 2, 16, 64, "f32")
    wl = inputs.make_workload("smallx", shape=shp, seed=31, with_block=False)
    NB = shp.n_blocks
    keep = np.full(shp.grids, K)
    want = {"partition": NB + 3 * K, "overlap": NB + 4 * K, "drop": 4 * K}
    for tokens, n_img in want.items():
        res = O.pipeline(wl.x_img, wl.x_txt, shp, None, 0, "topk", keep=keep, with_block=False, tokens=tokens)
        assert (res["counts"].sum(axis=1) == n_img).all()
        assert res["cu"][-1] == shp.batch * (n_img + shp.text_len)


def test_overlap_rows_are_fine_patches_and_every_block_mean():
    shp = inputs.BlockShape(1, 1, 6, 8, 2, 16, 2, 8, 64, "f32")
    wl = inputs.make_workload("smallx", shape=shp, seed=32, with_block=False)
    keep = np.array([5])
    res = O.pipeline(wl.x_img, wl.x_txt, shp, None, 0, "topk", keep=keep, with_block=False, tokens="overlap")
    x = wl.x_img[0].astype(np.float64).reshape(6, 8, -1)
    means = x.reshape(3, 2, 4, 2, -1).mean(axis=(1, 3)).reshape(12, -1)  # block raster
    nf = int(res["counts"][0, 0])
    np.testing.assert_allclose(res["Z"][nf:nf + 12], means, rtol=0, atol=1e-12)
    np.testing.assert_array_equal(res["Z"][:nf], wl.x_img[0][res["fine_idx"][0, :nf]].astype(np.float64))


def _zero_gates(mod):
    m = mod.copy()
    m[:, :, 2] = 0.0
    m[:, :, 5] = 0.0
    return m


@pytest.mark.parametrize("tokens", ["partition", "overlap", "drop"])
def test_delta_with_an_identity_block_returns_the_input(tokens):
    shp = inputs.BlockShape(2, 1, 6, 8, 3, 32, 2, 16, 64, "f32")
    wl = inputs.make_workload("smallx", shape=shp, seed=33)
    res = O.pipeline(wl.x_img, wl.x_txt, shp, None, 0, "topk", keep=wl.keep, weights=wl.weights,
                     mod=_zero_gates(wl.mod), tokens=tokens, delta=True)
    np.testing.assert_array_equal(res["y_img"], wl.x_img.astype(np.float64))


def test_broadcast_overlap_with_an_identity_block_gives_fine_patches_and_block_means():
    shp = inputs.BlockShape(1, 1, 6, 8, 3, 32, 2, 16, 64, "f32")
    wl = inputs.make_workload("smallx", shape=shp, seed=34)
    res = O.pipeline(wl.x_img, wl.x_txt, shp, None, 0, "topk", keep=wl.keep, weights=wl.weights,
                     mod=_zero_gates(wl.mod), tokens="overlap")
    x = wl.x_img[0].astype(np.float64).reshape(6, 8, -1)
    means = x.reshape(3, 2, 4, 2, -1).mean(axis=(1, 3))
    bcast = np.repeat(np.repeat(means, 2, axis=0), 2, axis=1).reshape(48, -1)
    fine_patch = res["fine"][0][O.block_of(6, 8)]
    want = np.where(fine_patch[:, None], x.reshape(48, -1), bcast)
    np.testing.assert_allclose(res["y_img"][0], want, rtol=0, atol=1e-12)


def test_delta_equals_broadcast_when_every_block_is_fine():
    shp = inputs.BlockShape(1, 1, 6, 8, 3, 32, 2, 16, 64, "f32")
    wl = inputs.make_workload("smallx", shape=shp, seed=35, keep_frac=1.0)
    a = O.pipeline(wl.x_img, wl.x_txt, shp, None, 0, "topk", keep=wl.keep, weights=wl.weights, mod=wl.mod,
                   tokens="partition")
    b = O.pipeline(wl.x_img, wl.x_txt, shp, None, 0, "topk", keep=wl.keep, weights=wl.weights, mod=wl.mod,
                   tokens="partition", delta=True)
    np.testing.assert_allclose(b["y_img"], a["y_img"], rtol=0, atol=1e-13)
