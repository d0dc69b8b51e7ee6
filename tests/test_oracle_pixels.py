"""The pixel-space scorer (Sobel on the RGB image, summed over each token's 16 x 16 pixels), pinned
by closed forms and scipy's Sobel filter."""
import numpy as np
import pytest
from scipy import ndimage

from oracle import hilo_oracle as O
from paper_2606_13898_amd import inputs


def test_flat_image_has_no_energy():
    rgb = np.full((2, 3, 32, 48), 0.37, dtype=np.float32)
    assert (O.score_pixels(rgb, 2, 3) == 0).all()


def test_horizontal_ramp_closed_form():
    """I = a x on one channel: gx = 8a inside (4a at the first and last image column, clamped), gy = 0.
    With a = 1/16 the per-pixel energies 1/4 and 1/16 are exact: q = 16384 and 4096."""
    H, W = 2, 3
    rgb = np.zeros((1, 3, 16 * H, 16 * W), dtype=np.float32)
    rgb[0, 1] = (np.arange(16 * W, dtype=np.float32) / 16.0)[None, :]
    E = O.score_pixels(rgb, H, W).reshape(H, W)
    edge = 15 * 16 * 16384 + 16 * 4096  # 15 interior columns + the clamped image-edge column
    np.testing.assert_array_equal(E, [[edge, 256 * 16384, edge], [edge, 256 * 16384, edge]])


@pytest.mark.parametrize("seed", [0, 1])
def test_matches_scipy_sobel_on_integer_images(seed):
    """Small integers: every float32 operation is exact, so the energy must equal scipy's Sobel
    (nearest-mode border = replicated) squared, scaled and pooled."""
    rng = np.random.default_rng(seed)
    H, W = 3, 2
    rgb = rng.integers(-20, 21, size=(2, 3, 16 * H, 16 * W)).astype(np.float32)
    E = O.score_pixels(rgb, H, W)
    for g in range(2):
        tot = np.zeros((16 * H, 16 * W), dtype=np.int64)
        for c in range(3):
            x = rgb[g, c].astype(np.float64)
            gx = ndimage.sobel(x, axis=1, mode="nearest")
            gy = ndimage.sobel(x, axis=0, mode="nearest")
            tot += ((gx * gx + gy * gy) * 65536).astype(np.int64)
        want = tot.reshape(H, 16, W, 16).sum(axis=(1, 3)).reshape(-1)
        np.testing.assert_array_equal(E[g], want)


def test_channel_order_does_not_matter_and_textured_regions_score_high():
    shp = inputs.BlockShape(1, 1, 8, 10, 0, 64, 1, 64, 64, "f32")
    rgb = inputs.pixel_image(shp, 3)
    E = O.score_pixels(rgb, 8, 10)
    np.testing.assert_array_equal(E, O.score_pixels(rgb[:, ::-1].copy(), 8, 10))
    # the threshold of the paper on the normalised map picks a non-trivial subset
    Bs = O.block_sums(E, 8, 10).astype(np.float64)
    frac = float((Bs > 4 * 0.1 * E.max()).mean())
    assert 0.05 < frac < 0.95
