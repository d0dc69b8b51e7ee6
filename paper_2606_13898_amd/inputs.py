"""Seeded synthetic inputs for the compressed DiT block (shared by the HIP path and the oracle).

This module draws numbers and nothing else: it holds none of the method's arithmetic (no score,
no selection, no pooling, no block maths).  Both sides of every parity check take their inputs
from here, so that they see the same bits.

Workloads.  The paper times its DiT on internal editing cases that are not available (Sec. 3.3,
"Speedup Analysis"); these synthetic latents stand in for them with the paper's shapes:

* the token grid follows from the 8x VAE and 2x patch-embed compression of the high-frequency
  branch (Sec. 2.3, "HiLo-Token Selection"): 1024^2 -> 64x64 tokens, 2048^2 -> 128x128 tokens;
* the edit masks follow the mask statistics of Sec. 2.3 ("Mask Distribution"): most masks are
  small, scattered holes come first, then elongated holes, then square or irregular blobs.

Every array is numpy; bf16 workloads are rounded to bf16 once here (round-to-nearest-even, done by
torch's dtype cast), so the float32 arrays handed to the oracle hold exactly the bits that the
device receives.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np

F32 = "f32"
BF16 = "bf16"


@dataclasses.dataclass(frozen=True)
class BlockShape:
    """Shape of one compressed-block problem.

    batch      samples B in one launch
    images     grids per sample I (1, or 2 for target + source conditioning)
    grid_h/w   latent patch grid (even)
    text_len   text/condition tokens per sample L_t
    dim        hidden width D = heads * head_dim
    mlp_dim    MLP hidden width (4 D)
    dtype      storage dtype of inputs, weights and outputs ("f32" or "bf16")
    """

    batch: int
    images: int
    grid_h: int
    grid_w: int
    text_len: int
    dim: int
    heads: int
    head_dim: int
    mlp_dim: int
    dtype: str

    @property
    def grids(self) -> int:
        return self.batch * self.images

    @property
    def n_patches(self) -> int:
        return self.grid_h * self.grid_w

    @property
    def n_blocks(self) -> int:
        return self.n_patches // 4

    @property
    def max_tokens(self) -> int:
        return self.batch * (self.images * self.n_patches + self.text_len)


@dataclasses.dataclass
class Workload:
    """Everything one block call consumes.

    x_img   [G][N][D] float32 (bf16-representable for bf16 shapes), N = grid_h*grid_w raster
    x_txt   [B][L_t][D] float32
    force   [G][N] uint8 edit mask (1 = inside the user mask) or None
    keep    [G] int32 kept-fine blocks per grid for top-k selection
    weights list of two dicts (index 0 image stream, 1 text stream) with
            w_qkv [3D][D], b_qkv [3D], w_o [D][D], b_o [D], w1 [F][D], b1 [F], w2 [D][F], b2 [D]
    mod     [B][2][6][D] float32: shift1, scale1, gate1, shift2, scale2, gate2 per sample/stream
    """

    name: str
    shape: BlockShape
    x_img: np.ndarray
    x_txt: np.ndarray
    force: Optional[np.ndarray]
    keep: np.ndarray
    dilate_r: int
    weights: Optional[List[Dict[str, np.ndarray]]]
    mod: Optional[np.ndarray]


def to_bf16_values(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even) and return them widened to float32."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy()


def _store(a: np.ndarray, dtype: str) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.float32)
    return to_bf16_values(a) if dtype == BF16 else a


# --------------------------------------------------------------------------------------------
# field generators
# --------------------------------------------------------------------------------------------

def _coords(h: int, w: int):
    u = (2.0 * (np.arange(w) + 0.5) / w - 1.0)[None, :].repeat(h, 0)
    v = (2.0 * (np.arange(h) + 0.5) / h - 1.0)[:, None].repeat(w, 1)
    return u, v


def smooth_background(rng: np.random.Generator, h: int, w: int, d: int) -> np.ndarray:
    """Per-channel random degree-3 polynomial in (u, v) plus N(0, 0.01) iid noise -> [h*w][d]."""
    u, v = _coords(h, w)
    basis = [u ** a * v ** b for a in range(4) for b in range(4 - a)]  # 10 monomials
    basis = np.stack([m.reshape(-1) for m in basis], axis=1).astype(np.float32)  # [N][10]
    alpha = rng.normal(0.0, 0.2, size=(basis.shape[1], d)).astype(np.float32)
    field = basis @ alpha
    field += rng.normal(0.0, 0.01, size=field.shape).astype(np.float32)
    return field


def region_mask(rng: np.random.Generator, h: int, w: int, target: float, tol: float,
                n_min: int = 3, n_max: int = 5) -> np.ndarray:
    """Union of seeded rectangles/ellipses with semi-axes U[0.08, 0.3] * side, rejection-sampled
    until the union covers target +- tol of the grid.  Returns bool [h][w]."""
    ii, jj = np.mgrid[0:h, 0:w]
    for _ in range(10000):
        m = np.zeros((h, w), dtype=bool)
        for _ in range(int(rng.integers(n_min, n_max + 1))):
            ci, cj = rng.uniform(0, h), rng.uniform(0, w)
            ai, aj = rng.uniform(0.08, 0.3) * h, rng.uniform(0.08, 0.3) * w
            if rng.random() < 0.5:
                m |= (np.abs(ii + 0.5 - ci) <= ai) & (np.abs(jj + 0.5 - cj) <= aj)
            else:
                m |= ((ii + 0.5 - ci) / ai) ** 2 + ((jj + 0.5 - cj) / aj) ** 2 <= 1.0
        if abs(m.mean() - target) <= tol:
            return m
    raise RuntimeError("region rejection sampling did not converge")


def square_mask(rng: np.random.Generator, h: int, w: int, side: int) -> np.ndarray:
    i0 = int(rng.integers(0, h - side + 1))
    j0 = int(rng.integers(0, w - side + 1))
    m = np.zeros((h, w), dtype=bool)
    m[i0:i0 + side, j0:j0 + side] = True
    return m


def octave_noise(rng: np.random.Generator, h: int, w: int, d: int) -> np.ndarray:
    """Sum of 3 octaves of Gaussian-filtered N(0,1) noise (sigma = 1, 2, 4 patches, weights
    1, 1/2, 1/4, each octave normalised to unit std), renormalised to unit std -> [h][w][d]."""
    from scipy.ndimage import gaussian_filter

    total = np.zeros((h, w, d), dtype=np.float32)
    for o in range(3):
        n = rng.standard_normal((h, w, d), dtype=np.float32)
        n = gaussian_filter(n, sigma=(2.0 ** o, 2.0 ** o, 0.0), mode="wrap")
        n /= n.std()
        total += n * (2.0 ** -o)
    total /= total.std()
    return total


def edit_mask(rng: np.random.Generator, h: int, w: int, target: float = 0.15,
              tol: float = 0.02) -> np.ndarray:
    """User edit mask with the shape mix of the paper's mask statistics: a union of 1-4 shapes drawn
    from scattered discs, elongated bars and square/irregular blobs; area target +- tol."""
    ii, jj = np.mgrid[0:h, 0:w]
    for _ in range(10000):
        m = np.zeros((h, w), dtype=bool)
        for _ in range(int(rng.integers(1, 5))):
            kind = rng.choice(3, p=[0.55, 0.25, 0.20])
            if kind == 0:  # scattered holes: several small discs
                for _ in range(int(rng.integers(3, 9))):
                    ci, cj = rng.uniform(0, h), rng.uniform(0, w)
                    r = rng.uniform(0.03, 0.08) * h
                    m |= (ii + 0.5 - ci) ** 2 + (jj + 0.5 - cj) ** 2 <= r * r
            elif kind == 1:  # elongated bar at a random angle
                ci, cj = rng.uniform(0, h), rng.uniform(0, w)
                th = rng.uniform(0, np.pi)
                ln, wd = rng.uniform(0.3, 0.8) * h, rng.uniform(0.03, 0.08) * h
                a = (ii + 0.5 - ci) * np.cos(th) + (jj + 0.5 - cj) * np.sin(th)
                b = -(ii + 0.5 - ci) * np.sin(th) + (jj + 0.5 - cj) * np.cos(th)
                m |= (np.abs(a) <= ln / 2) & (np.abs(b) <= wd / 2)
            else:  # square or irregular blob (square with a wobbly edge)
                ci, cj = rng.uniform(0, h), rng.uniform(0, w)
                s = rng.uniform(0.1, 0.3) * h
                wob = 1.0 + 0.25 * np.sin(3 * np.arctan2(ii + 0.5 - ci, jj + 0.5 - cj) + rng.uniform(0, 6))
                m |= np.maximum(np.abs(ii + 0.5 - ci), np.abs(jj + 0.5 - cj)) <= s * wob / 2
        if abs(m.mean() - target) <= tol:
            return m
    raise RuntimeError("edit-mask rejection sampling did not converge")


def block_weights(rng: np.random.Generator, d: int, f: int, dtype: str) -> List[Dict[str, np.ndarray]]:
    """Two streams (image, text) of DiT-block weights, every entry N(0, 0.02), nn.Linear [out][in]."""
    out = []
    for _ in range(2):
        ws = {}
        for name, shp in (("w_qkv", (3 * d, d)), ("b_qkv", (3 * d,)), ("w_o", (d, d)), ("b_o", (d,)),
                          ("w1", (f, d)), ("b1", (f,)), ("w2", (d, f)), ("b2", (d,))):
            ws[name] = _store(rng.normal(0.0, 0.02, size=shp).astype(np.float32), dtype)
        out.append(ws)
    return out


def modulation(rng: np.random.Generator, b: int, d: int, gate_std: float = 0.1) -> np.ndarray:
    """adaLN modulation [B][2 streams][6][D]: shift and scale ~ N(0, 0.1), gate ~ N(0, gate_std)
    (the same draws as gate_std = 0.1, the gates scaled).

    The gate scale sets how large the block's update is next to the residual stream (here a
    perturbation of ~20%).  It also sets the size of the unavoidable bf16 error: rounding the
    projection inputs (normalised rows, GELU activations) to bf16 costs ~0.1% of each update, so
    gates of std 0.3 would put even an exact emulation of the bf16 roundings at a max-abs error of
    ~0.024 against a float64 reference, above the 2e-2 bar; std 0.1 keeps it near 0.016."""
    m = rng.normal(0.0, 0.1, size=(b, 2, 6, d)).astype(np.float32)
    if gate_std != 0.1:
        m[:, :, 2] *= np.float32(gate_std / 0.1)
        m[:, :, 5] *= np.float32(gate_std / 0.1)
    return m


# --------------------------------------------------------------------------------------------
# named workloads
# --------------------------------------------------------------------------------------------

SHAPES: Dict[str, BlockShape] = {
    # 32x32 grid + 64 text tokens, hidden 256, 4 heads x 64, MLP 4x, fp32
    "tiny": BlockShape(1, 1, 32, 32, 64, 256, 4, 64, 1024, F32),
    # 1024px: 64x64 grid + 512 text tokens, hidden 3072, 24 heads x 128, bf16
    "m1024": BlockShape(1, 1, 64, 64, 512, 3072, 24, 128, 12288, BF16),
    # 2048px: 128x128 grid + 512 text tokens
    "h2048": BlockShape(1, 1, 128, 128, 512, 3072, 24, 128, 12288, BF16),
    # edit with reference conditioning: target + source 64x64 grids + 512 text tokens
    "edit": BlockShape(1, 2, 64, 64, 512, 3072, 24, 128, 12288, BF16),
    # batched ragged stress: 8 samples of 64x64 + 512 text
    "ragged": BlockShape(8, 1, 64, 64, 512, 3072, 24, 128, 12288, BF16),
    # small bf16 shapes that still span several tiles and ragged tails (parity at oracle speed)
    "small128": BlockShape(2, 1, 16, 20, 40, 256, 2, 128, 1024, BF16),
    "small64": BlockShape(1, 2, 12, 16, 24, 256, 4, 64, 1024, BF16),
    "smallf32": BlockShape(2, 1, 10, 14, 9, 128, 2, 64, 512, F32),
}

_SEED = {"tiny": 1001, "m1024": 1002, "h2048": 1003, "edit": 1004, "ragged": 1005,
         "small128": 2001, "small64": 2002, "smallf32": 2003}


def pixel_image(shape: BlockShape, seed: int) -> np.ndarray:
    """A synthetic RGB image of the token grid's size, planar float32 [G][3][16 H][16 W]: per
    channel a smooth degree-3 polynomial background (values around 0.5) plus N(0, 0.15) pixel
    noise inside 1-3 seeded regions covering ~35% of the image (the textured, high-frequency
    areas), the stand-in for the paper's input images."""
    rng = np.random.default_rng(seed)
    T = 16
    G, h, w = shape.grids, shape.grid_h, shape.grid_w
    Hp, Wp = h * T, w * T
    img = np.empty((G, 3, Hp, Wp), dtype=np.float32)
    u, v = _coords(Hp, Wp)
    basis = np.stack([u ** a * v ** b for a in range(4) for b in range(4 - a)], axis=0).astype(np.float32)
    for g in range(G):
        reg = region_mask(rng, h, w, 0.35, 0.10, 1, 3)
        reg_px = np.repeat(np.repeat(reg, T, axis=0), T, axis=1)
        for c in range(3):
            alpha = rng.normal(0.0, 0.1, size=basis.shape[0]).astype(np.float32)
            field = 0.5 + np.tensordot(alpha, basis, axes=1)
            field += np.where(reg_px, rng.normal(0.0, 0.15, size=(Hp, Wp)), 0.0).astype(np.float32)
            img[g, c] = field
    return img


@dataclasses.dataclass
class StackWorkload:
    """One request in the paper's regime: the selection is computed once, from step 0's latents,
    then each of `steps` sampling steps compresses that step's latents with it, runs `n_blocks`
    blocks on the compressed sequence and decompresses.

    base     Workload of step 0 (shape, x_txt, force, keep, dilate_r; its weights are block 0's)
    x_steps  list of `steps` arrays [G][N][D] (x_steps[0] is base.x_img): each step's latents are
             the previous step's plus N(0, 0.1) changes, stored in the shape's dtype
    weights  list of `n_blocks` weight sets (block_weights)
    mods     [steps][n_blocks][B][2][6][D] float32: the modulation of block l at step t
    """

    base: Workload
    x_steps: List[np.ndarray]
    weights: List[List[Dict[str, np.ndarray]]]
    mods: np.ndarray


def make_stack(name: str, n_blocks: int, steps: int, *, seed: Optional[int] = None,
               shape: Optional[BlockShape] = None, keep_frac: Optional[float] = None) -> StackWorkload:
    base = make_workload(name, seed=seed, shape=shape, keep_frac=keep_frac)
    shp = base.shape
    ss = np.random.SeedSequence((seed if seed is not None else _SEED.get(name, 3000)) + 7919)
    c_w, c_mod, c_x = [np.random.default_rng(s) for s in ss.spawn(3)]
    weights = [base.weights] + [block_weights(c_w, shp.dim, shp.mlp_dim, shp.dtype)
                                for _ in range(n_blocks - 1)]
    mods = np.stack([np.stack([modulation(c_mod, shp.batch, shp.dim) for _ in range(n_blocks)])
                     for _ in range(steps)])
    x_steps = [base.x_img]
    for _ in range(steps - 1):
        x_steps.append(_store(x_steps[-1] + c_x.normal(0.0, 0.1, size=x_steps[-1].shape).astype(np.float32),
                              shp.dtype))
    return StackWorkload(base, x_steps, weights, mods)


def make_workload(name: str, *, with_block: bool = True, keep_frac: Optional[float] = None,
                  seed: Optional[int] = None, shape: Optional[BlockShape] = None,
                  gate_std: float = 0.1) -> Workload:
    """Build the named workload.  `keep_frac` overrides the kept-fine block fraction of every grid
    (used for the dense baseline, keep_frac=1, and the kept-fraction sweep); `gate_std` the
    standard deviation of the adaLN gates."""
    shp = shape or SHAPES[name]
    ss = np.random.SeedSequence(seed if seed is not None else _SEED.get(name, 3000))
    (c_bg, c_noise, c_reg, c_tex, c_txt, c_w, c_mod, c_mask, c_frac) = [
        np.random.default_rng(s) for s in ss.spawn(9)]
    del c_noise  # the background generator draws its own noise; the child is kept for stable order
    h, w, d = shp.grid_h, shp.grid_w, shp.dim
    G, B, NB = shp.grids, shp.batch, shp.n_blocks

    x = np.empty((G, h * w, d), dtype=np.float32)
    for g in range(G):
        x[g] = smooth_background(c_bg, h, w, d)
        if name in ("tiny",):
            reg = square_mask(c_reg, h, w, 12)
        elif name == "h2048":
            reg = region_mask(c_reg, h, w, 0.20, 0.03)
        elif name not in SHAPES or name.startswith("small"):
            reg = region_mask(c_reg, h, w, 0.35, 0.10, 1, 3)
        else:
            reg = region_mask(c_reg, h, w, 0.35, 0.03)
        if name == "h2048":
            tex = octave_noise(c_tex, h, w, d).reshape(h * w, d)
            x[g][reg.reshape(-1)] += tex[reg.reshape(-1)]
        else:
            idx = np.flatnonzero(reg.reshape(-1))
            x[g][idx] += c_tex.standard_normal((idx.size, d), dtype=np.float32)
    x_txt = c_txt.standard_normal((B, shp.text_len, d), dtype=np.float32)

    force = None
    dilate_r = 0
    if name in ("edit", "small64"):
        m = edit_mask(c_mask, h, w, 0.15, 0.02 if name == "edit" else 0.08)
        force = np.repeat(m.reshape(1, -1), G, axis=0).astype(np.uint8)

    fracs = {"tiny": 0.30, "m1024": 0.40, "h2048": 0.25, "edit": 0.35}
    if keep_frac is not None:
        keep = np.full(G, int(round(keep_frac * NB)), dtype=np.int32)
    elif name == "ragged" or name.startswith("small"):
        keep = np.round(c_frac.uniform(0.05, 0.95, size=G) * NB).astype(np.int32)
    else:
        keep = np.full(G, int(round(fracs.get(name, 0.4) * NB)), dtype=np.int32)

    weights = mod = None
    if with_block:
        weights = block_weights(c_w, d, shp.mlp_dim, shp.dtype)
        mod = modulation(c_mod, B, d, gate_std)
    return Workload(name, shp, _store(x, shp.dtype), _store(x_txt, shp.dtype), force, keep,
                    dilate_r, weights, mod)
