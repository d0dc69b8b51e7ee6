"""GPU parity of the whole hot path against the CPU oracle on small seeded workloads (every kernel
is launched through the C ABI).  Sizes span several GEMM / attention tiles and ragged tails while
the oracle still finishes in seconds."""
import numpy as np
import pytest
import torch

from oracle import hilo_oracle as O
from paper_2606_13898_amd import hilo, inputs
from paper_2606_13898_amd.pipeline import DeviceBlock, DeviceStack

from parity_util import (assert_close, assert_update_close, check_compressed, check_selection,
                         float_report, midpoint_tau, oracle_for, to_np)

pytestmark = pytest.mark.gpu

SMALL = ["tiny", "small128", "small64", "smallf32"]


def _block_stages(name, wl, check_z=True, fused=False):
    """Score, select and compress, then the block one half at a time: the selection bit for bit,
    the compressed sequence bit for bit (pooled rows to float32 rounding), each half's update of z
    against the oracle's update, z and y against the oracle (fused: hilo_compress_norm, then
    hilo_attention_normed on the rows it left in the workspace)."""
    dt = wl.shape.dtype
    db = DeviceBlock(wl)
    ref = oracle_for(wl)
    db.score()
    db.select(hilo.TOPK)
    db.compress(norm=fused)
    torch.cuda.synchronize()
    check_selection(db, ref)
    T = int(ref["cu"][-1])
    z0 = to_np(db.z)[:T].copy()
    check_compressed(z0, ref, wl)
    db.attention(normed=fused)
    torch.cuda.synchronize()
    z1 = to_np(db.z)[:T].copy()
    assert_update_close(z1, ref["z1"], z0, ref["Z"], dt, f"{name} attention update z1 - Z")
    if check_z:
        assert_close(z1, ref["z1"], dt, f"{name} z after attention")
    db.mlp()
    torch.cuda.synchronize()
    z2 = to_np(db.z)[:T].copy()
    assert_update_close(z2, ref["z2"], z1, ref["z1"], dt, f"{name} mlp update z2 - z1")
    if check_z:
        assert_close(z2, ref["z2"], dt, f"{name} z after mlp")
    db.decompress()
    torch.cuda.synchronize()
    return db, ref


@pytest.mark.parametrize("name", SMALL)
def test_pipeline_parity(name):
    print(f"[parity] workload={name}", flush=True)
    wl = inputs.make_workload(name)
    dt = wl.shape.dtype
    db, ref = _block_stages(name, wl)
    assert_close(to_np(db.y_img), ref["y_img"], dt, f"{name} y_img")
    assert_close(to_np(db.y_txt), ref["y_txt"], dt, f"{name} y_txt")
    assert np.abs(ref["y_img"]).max() < 8.0


@pytest.mark.parametrize("name", SMALL)
def test_fused_compress_norm(name):
    """The attention half's first row norm in the compress pass (hilo_compress_norm +
    hilo_attention_normed, the benchmark's step): every stage against the oracle, and z, y_img and
    y_txt bit for bit those of hilo_compress + hilo_attention."""
    print(f"[parity] fused compress + norm workload={name}", flush=True)
    wl = inputs.make_workload(name)
    db, ref = _block_stages(f"{name} fused", wl, fused=True)
    T = int(ref["cu"][-1])
    z_f, yi_f, yt_f = db.z[:T].clone(), db.y_img.clone(), db.y_txt.clone()
    db.run(hilo.TOPK, fused=False)
    torch.cuda.synchronize()
    assert int(db.cu[-1]) == T
    assert torch.equal(db.z[:T], z_f), "z differs from the unfused calls"
    assert torch.equal(db.y_img, yi_f), "y_img differs from the unfused calls"
    assert torch.equal(db.y_txt, yt_f), "y_txt differs from the unfused calls"


def test_pipeline_parity_gate_std_0_3():
    """adaLN gates ~ N(0, 0.3): the block's update is ~3x larger next to the residual stream.  The
    output's own bf16 rounding then takes most of the max-abs bar wherever |y| reaches [4, 8), so
    this workload is judged on each half's update (relative L2) and on y's relative L2."""
    print("[parity] workload=small128 gate std 0.3", flush=True)
    wl = inputs.make_workload("small128", gate_std=0.3)
    db, ref = _block_stages("small128 gate 0.3", wl, check_z=False)
    _, rel = float_report(to_np(db.y_img), ref["y_img"])
    print(f"[parity] gate 0.3 y_img rel_l2 {rel:.3g}", flush=True)
    assert rel <= 5e-3


@pytest.mark.parametrize("name", ["tiny", "small128", "small64"])
def test_threshold_selection_matches(name):
    print(f"[parity] threshold workload={name}", flush=True)
    wl = inputs.make_workload(name, with_block=False)
    db = DeviceBlock(wl, with_block=False)
    E = O.score(wl.x_img, wl.shape.grid_h, wl.shape.grid_w)
    tau = midpoint_tau(E, wl.force, wl.shape, wl.dilate_r, wl.keep)
    ref = oracle_for(wl, mode="threshold", tau=tau, with_block=False)
    db.score()
    db.select(hilo.THRESHOLD, tau=tau)
    db.compress()
    db.decompress()
    torch.cuda.synchronize()
    check_selection(db, ref)
    # the midpoint threshold picks exactly the top-k set
    ref_k = oracle_for(wl, mode="topk", with_block=False)
    np.testing.assert_array_equal(ref["idx_map"], ref_k["idx_map"])
    # without the block, decompress(compress(x)) keeps fine patches bit for bit
    y = to_np(db.y_img)
    blk = O.block_of(wl.shape.grid_h, wl.shape.grid_w)
    for g in range(wl.shape.grids):
        fp = ref["fine"][g][blk]
        np.testing.assert_array_equal(y[g][fp], wl.x_img[g][fp])


@pytest.mark.parametrize("keep_frac", [0.0, 1.0])
def test_extreme_keep_fractions(keep_frac):
    """0% kept (every block pooled) and 100% kept (0% compression: the dense block)."""
    print(f"[parity] small128 keep_frac={keep_frac}", flush=True)
    wl = inputs.make_workload("small128", keep_frac=keep_frac)
    db = DeviceBlock(wl)
    ref = oracle_for(wl)
    db.run(hilo.TOPK)
    torch.cuda.synchronize()
    check_selection(db, ref)
    assert_close(to_np(db.y_img), ref["y_img"], "bf16", "y_img")
    if keep_frac == 1.0:
        s = wl.shape
        np.testing.assert_array_equal(to_np(db.idx_map), np.tile(np.arange(s.n_patches), (s.grids, 1)))
        Zd, cud = O.dense_sequence(wl.x_img, wl.x_txt, s.batch, s.images, s.text_len)
        _, z2d = O.block(Zd, cud, s.text_len, s.heads, wl.weights, wl.mod)
        N = s.n_patches
        dense_y = np.stack([z2d[cud[b] + i * N: cud[b] + (i + 1) * N]
                            for b in range(s.batch) for i in range(s.images)])
        assert_close(to_np(db.y_img), dense_y, "bf16", "0% compression vs dense oracle")


def test_force_mask_with_dilation():
    print("[parity] small64 force r=1", flush=True)
    wl = inputs.make_workload("small64")
    db = DeviceBlock(wl)
    ref = oracle_for(wl, r=1)
    db.run(hilo.TOPK, dilate_r=1)
    torch.cuda.synchronize()
    check_selection(db, ref)
    assert_close(to_np(db.y_img), ref["y_img"], "bf16", "y_img r=1")


def test_flat_grid_threshold_keeps_only_forced_blocks():
    print("[parity] flat grid", flush=True)
    shp = inputs.BlockShape(1, 2, 8, 12, 0, 64, 1, 64, 256, "bf16")
    wl = inputs.make_workload("flat", shape=shp, with_block=False, seed=5)
    wl.x_img[:] = 0.5
    wl.force = np.zeros((2, 96), np.uint8)
    wl.force[1, 30] = 1
    db = DeviceBlock(wl, with_block=False)
    ref = oracle_for(wl, mode="threshold", tau=[0.1, 0.1], r=0, with_block=False)
    db.score()
    db.select(hilo.THRESHOLD, tau=[0.1, 0.1], dilate_r=0)
    db.compress()
    db.decompress()
    torch.cuda.synchronize()
    check_selection(db, ref)
    assert to_np(db.counts).tolist() == [[0, 24], [4, 23]]
    # constant blocks pool and broadcast back losslessly
    np.testing.assert_array_equal(to_np(db.y_img), wl.x_img)


def test_constant_blocks_roundtrip_bitwise():
    print("[parity] constant blocks", flush=True)
    shp = inputs.BlockShape(2, 1, 10, 14, 3, 128, 1, 128, 512, "bf16")
    wl = inputs.make_workload("const", shape=shp, with_block=False, seed=6)
    coarse = inputs.to_bf16_values(np.random.default_rng(1).standard_normal((2, 5, 7, 128)).astype(np.float32))
    wl.x_img = np.repeat(np.repeat(coarse, 2, 1), 2, 2).reshape(2, 140, 128).copy()
    wl.keep = np.array([5, 11], np.int32)
    db = DeviceBlock(wl, with_block=False)
    db.score()
    db.select(hilo.TOPK)
    db.compress()
    db.decompress()
    torch.cuda.synchronize()
    np.testing.assert_array_equal(to_np(db.y_img), wl.x_img)
    np.testing.assert_array_equal(to_np(db.y_txt), wl.x_txt)


def test_no_text_tokens():
    print("[parity] no text", flush=True)
    shp = inputs.BlockShape(2, 1, 12, 10, 0, 256, 2, 128, 1024, "bf16")
    wl = inputs.make_workload("notext", shape=shp, seed=8)
    wl.keep = np.array([7, 20], np.int32)
    db = DeviceBlock(wl)
    ref = oracle_for(wl)
    db.run(hilo.TOPK)
    torch.cuda.synchronize()
    check_selection(db, ref)
    assert_close(to_np(db.y_img), ref["y_img"], "bf16", "y_img no text")


def test_run_to_run_determinism():
    print("[parity] determinism small128", flush=True)
    wl = inputs.make_workload("small128")
    db = DeviceBlock(wl)
    outs = []
    for _ in range(2):
        db.run(hilo.TOPK)
        torch.cuda.synchronize()
        outs.append((db.energy.clone(), db.idx_map.clone(), db.z.clone(), db.y_img.clone()))
    for a, b in zip(*outs):
        assert torch.equal(a, b)


# (128, [150, 300, 3]): fewer key steps than workgroups, so every step is its own range and the
# query tiles are cut into 3 and 5 pieces -- the merge's odd, unpaired last contributor
# Many units per workgroup (256 workgroups for head dim 128, 512 for 64): (128, 24 heads, 3 x 1100)
# is 360 query tiles of 256 rows; (64, 8 heads, 8 x 1000) 512 tiles of 128 rows, as many as
# workgroups, so every range boundary falls at a tile's key step 0 or mid-tile alike; (64, 8 heads,
# 9 x 1000) 576 tiles
@pytest.mark.parametrize("hd,lens,heads", [(128, [1, 17, 64, 65, 200], 2), (128, [150, 300, 3], 2),
                                           (64, [3, 130, 31], 2), (128, [1100] * 3, 24),
                                           (64, [1000] * 8, 8), (64, [1000] * 9, 8)])
def test_attention_core_ragged(hd, lens, heads):
    print(f"[parity] attention core hd={hd} heads={heads} lens={lens}", flush=True)
    D = heads * hd
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    T = int(cu[-1])
    rng = np.random.default_rng(hd + len(lens))
    qkv = inputs.to_bf16_values(rng.standard_normal((T, 3 * D)).astype(np.float32))
    want = O.attention_core(qkv, cu, heads)
    # a shape whose longest possible sample covers the longest length
    maxlen = max(lens)
    H = 2
    W = 2 * ((maxlen + 3) // 4)
    shp = hilo.hilo_shape(len(lens), 1, H, W, 0, D, heads, hd, 4 * D, hilo.BF16)
    q = torch.from_numpy(qkv).to(torch.bfloat16).cuda()
    out = torch.zeros(T, D, dtype=torch.bfloat16, device="cuda")
    cut = torch.from_numpy(cu).cuda()
    ws = torch.empty(hilo.hilo_workspace_bytes(shp), dtype=torch.uint8, device="cuda")
    hilo.hilo_attention_core(shp, q, cut, out, ws)
    torch.cuda.synchronize()
    assert_close(to_np(out), want, "bf16", f"attention core hd={hd}")


@pytest.mark.parametrize("shp", [
    # down projection: ~6 tiles, K = 8192 (128 steps) -> tiles cut into K pieces plus a stream-K tail
    inputs.BlockShape(3, 1, 16, 20, 40, 256, 2, 128, 8192, "bf16"),
    # a single 192 x 192 down-projection tile (at most 144 rows, N = 192): every K piece is one
    # step, the fixup sums 128 partial tiles
    inputs.BlockShape(1, 1, 12, 12, 0, 192, 3, 64, 8192, "bf16"),
], ids=["pieces_and_tail", "one_tile_128_pieces"])
def test_mlp_split_k(shp):
    """MLP with a long down-projection K and few output tiles: the projection is split along K
    and finished by the fixup; every row of z is compared with the oracle."""
    print(f"[parity] split-K mlp shape={shp}", flush=True)
    wl = inputs.make_workload("splitk", shape=shp, seed=11)
    db = DeviceBlock(wl)
    ref = oracle_for(wl)
    db.run(hilo.TOPK)
    torch.cuda.synchronize()
    check_selection(db, ref)
    T = int(ref["cu"][-1])
    assert_close(to_np(db.z)[:T], ref["z2"], "bf16", "z after split-K mlp")
    assert_close(to_np(db.y_img), ref["y_img"], "bf16", "y_img split-K")


# On a 256-CU device these reach every schedule of the 192 x 192 GEMM tiling (tests/
# test_gemm_schedule.py models the same plans); every block is kept fine so the row counts are fixed.
@pytest.mark.parametrize("shp", [
    # 12 + 2 row tiles x 19 column tiles = 266 MLP-up tiles of 16 K steps: one wave of whole tiles,
    # then a 10-tile stream-K tail over 14 workgroups whose range boundaries cut tiles (fixup)
    inputs.BlockShape(1, 1, 48, 48, 256, 1024, 8, 128, 3648, "bf16"),
    # 22 + 2 row tiles x 16 = 384 MLP-up tiles: the last wave holds 128 >= 128 tiles, so two waves of
    # whole tiles
    inputs.BlockShape(1, 1, 64, 64, 256, 256, 2, 128, 3072, "bf16"),
    # few tiles and K = 4608 (72 steps): QKV cut into 2 K pieces plus a stream-K tail, the attention
    # output into 6, MLP up into 22 pieces of three or four steps
    inputs.BlockShape(1, 1, 16, 16, 0, 4608, 36, 128, 1024, "bf16"),
], ids=["sk_tail", "whole_waves", "k_pieces"])
def test_gemm_schedules(shp):
    print(f"[parity] 192-tile GEMM schedules shape={shp}", flush=True)
    wl = inputs.make_workload("splitk", shape=shp, seed=5, keep_frac=1.0)
    db = DeviceBlock(wl)
    ref = oracle_for(wl)
    db.run(hilo.TOPK)
    torch.cuda.synchronize()
    check_selection(db, ref)
    T = int(ref["cu"][-1])
    assert_close(to_np(db.z)[:T], ref["z2"], "bf16", "z after block")
    assert_close(to_np(db.y_img), ref["y_img"], "bf16", "y_img")


@pytest.mark.parametrize("name,n_blocks,steps", [("small128", 2, 2), ("small64", 3, 2)])
def test_request_block_stack(name, n_blocks, steps):
    """One request: selection once from step 0, then per step compress -> hilo_blocks (n_blocks
    blocks) -> decompress; every step's outputs against the oracle's request loop."""
    print(f"[parity] request {name} blocks={n_blocks} steps={steps}", flush=True)
    st = inputs.make_stack(name, n_blocks, steps, seed=21)
    ds = DeviceStack(st)
    ds.run(hilo.TOPK)
    torch.cuda.synchronize()
    wl = st.base
    ref = O.request(st.x_steps, wl.x_txt, wl.shape, wl.force, wl.dilate_r, "topk", st.weights, st.mods,
                    keep=wl.keep)
    check_selection(ds.db, ref)
    dt = wl.shape.dtype
    for t in range(steps):
        assert_close(to_np(ds.y_img[t]), ref["y_img"][t], dt, f"{name} step {t} y_img", blocks=n_blocks)
        assert_close(to_np(ds.y_txt[t]), ref["y_txt"][t], dt, f"{name} step {t} y_txt", blocks=n_blocks)


TOKEN_SET = {"overlap": hilo.OVERLAP, "drop": hilo.DROP}


@pytest.mark.parametrize("name,tokens,delta", [
    ("small128", "overlap", False), ("small128", "overlap", True), ("small64", "overlap", True),
    ("small64", "drop", True), ("small64", "drop", False), ("smallf32", "overlap", True),
])
def test_token_sets(name, tokens, delta):
    """Every block's low-frequency token next to the kept fine patches (overlap), or the kept fine
    patches alone (drop), reassembled by broadcast or by the delta form."""
    print(f"[parity] token set {tokens} delta={delta} workload={name}", flush=True)
    wl = inputs.make_workload(name)
    db = DeviceBlock(wl)
    ref = oracle_for(wl, tokens=tokens, delta=delta)
    db.run(hilo.TOPK, tokens=TOKEN_SET[tokens], delta=delta)
    torch.cuda.synchronize()
    check_selection(db, ref)
    dt = wl.shape.dtype
    T = int(ref["cu"][-1])
    assert_close(to_np(db.z)[:T], ref["z2"], dt, f"{name} {tokens} z2")
    assert_close(to_np(db.y_img), ref["y_img"], dt, f"{name} {tokens} y_img")
    assert_close(to_np(db.y_txt), ref["y_txt"], dt, f"{name} {tokens} y_txt")


@pytest.mark.parametrize("shp", [
    inputs.BlockShape(1, 1, 8, 10, 0, 64, 1, 64, 256, "f32"),
    inputs.BlockShape(2, 2, 16, 20, 8, 64, 1, 64, 256, "bf16"),
    inputs.BlockShape(1, 1, 64, 64, 512, 3072, 24, 128, 12288, "bf16"),  # the 1024 px image
], ids=["8x10", "batch2x2_16x20", "1024px"])
def test_pixel_score_and_paper_threshold(shp):
    """Sobel on the RGB image summed per token (bit for bit), then the threshold selects the same
    blocks as the oracle.  The paper cuts its normalised Sobel magnitude map at 0.1; the energy is
    the magnitude squared, so the counterpart on the normalised energy map is 0.1^2 = 0.01 (exact
    where a token's magnitude is uniform; the mean of squares weights strong edges more)."""
    print(f"[parity] pixel score {shp.grid_h}x{shp.grid_w} grids={shp.grids}", flush=True)
    rgb = inputs.pixel_image(shp, 41)
    H, W, G, N = shp.grid_h, shp.grid_w, shp.grids, shp.n_patches
    want = O.score_pixels(rgb, H, W)
    shape = hilo.make_shape(shp)
    rgb_d = torch.from_numpy(rgb).cuda()
    E = torch.empty(G, N, dtype=torch.int64, device="cuda")
    hilo.hilo_score_pixels(shape, rgb_d, E)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(to_np(E), want)
    tau = [0.01] * G
    fine = O.select(want, None, H, W, 0, "threshold", tau=tau)
    idx_map, _, _, counts = O.compact(fine, H, W)
    i32 = dict(dtype=torch.int32, device="cuda")
    im, fi = torch.empty(G, N, **i32), torch.empty(G, N, **i32)
    pi, cnt = torch.empty(G, N // 4, **i32), torch.empty(G, 2, **i32)
    cu, seg = torch.empty(shp.batch + 1, **i32), torch.empty(G, **i32)
    hilo.hilo_select(shape, E, None, 0, hilo.THRESHOLD, tau, None, im, fi, pi, cnt, cu, seg)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(to_np(cnt), counts)
    np.testing.assert_array_equal(to_np(im), idx_map)
    assert 0 < counts[:, 0].sum() < G * N


def _random_shape(i):
    """Case i of a fixed seeded draw of valid block shapes: batch 1-3, one or two grids per sample,
    even grids 4..40 a side, no text or 1..159 text tokens, 1..6 heads of 64 or 128, bf16 or
    float32, kept fraction anywhere in [0, 1], the fused compress + LN pair on half the bf16 cases."""
    rng = np.random.default_rng([7919, i])
    hd = int(rng.choice([64, 128]))
    heads = int(rng.integers(1, 7))
    dim = hd * heads
    shp = inputs.BlockShape(int(rng.integers(1, 4)), int(rng.integers(1, 3)), 2 * int(rng.integers(2, 21)),
                            2 * int(rng.integers(2, 21)), int(rng.choice([0, int(rng.integers(1, 160))])),
                            dim, heads, hd, 4 * dim, str(rng.choice(["bf16", "f32"])))
    return shp, float(rng.uniform(0.0, 1.0)), int(rng.integers(0, 1 << 30)), bool(rng.integers(0, 2))


@pytest.mark.parametrize("i", range(12))
def test_random_shapes(i):
    """The whole path on seeded random shapes (ragged grids, text or none, 1-6 heads, both head
    dims and dtypes): the selection and compressed sequence bit for bit, both updates and z, y
    against the oracle, as on the named workloads."""
    shp, keep, seed, fused = _random_shape(i)
    fused = fused and shp.dtype == "bf16"
    name = f"random{i}"
    print(f"[parity] {name} {shp} keep={keep:.2f} seed={seed} fused={fused}", flush=True)
    wl = inputs.make_workload(name, shape=shp, seed=seed, keep_frac=keep)
    db, ref = _block_stages(name, wl, fused=fused)
    assert_close(to_np(db.y_img), ref["y_img"], shp.dtype, f"{name} y_img")
    if shp.text_len:
        assert_close(to_np(db.y_txt), ref["y_txt"], shp.dtype, f"{name} y_txt")
