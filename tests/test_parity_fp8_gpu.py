"""GPU parity of the FP8 block (all four projections on per-row E4M3 operands) against the oracle's
FP8 block, through the C ABI: the row quantiser bit for bit, the normalised rows' codes up to
float32-versus-float64 rounding of the layer norm, and the block outputs to the bf16 tolerances."""
import numpy as np
import pytest
import torch

from oracle import hilo_oracle as O
from paper_2606_13898_amd import hilo, inputs
from paper_2606_13898_amd.pipeline import DeviceBlock

from parity_util import assert_close, check_selection, float_report, oracle_for, to_np

pytestmark = pytest.mark.gpu


def _rows_for_quantiser(rng, dtype):
    """Rows that reach every branch of the quantiser: ordinary Gaussian rows, an all-zero row, a
    row whose amax is one huge outlier (most codes subnormal or zero), a row of one repeated value
    (every code 448), tiny values, and values exactly halfway between E4M3 neighbours after
    scaling (ties to even)."""
    x = rng.standard_normal((37, 96)).astype(np.float32) * 0.05
    x[3] = 0.0
    x[5] = rng.standard_normal(96).astype(np.float32) * 1e-3
    x[5, 17] = 30.0
    x[7] = -0.75
    x[9] *= 1e-6
    # row 11: amax 448 -> inv 1, so the scaled values are the values themselves; 1.0625 and
    # 1.1875 are ties between neighbouring codes (1.0 / 1.125 and 1.125 / 1.25)
    x[11] = 1.0
    x[11, 0], x[11, 1], x[11, 2], x[11, 3] = 448.0, 1.0625, 1.1875, -1.0625
    if dtype == torch.bfloat16:
        x = torch.from_numpy(x).to(torch.bfloat16).float().numpy()  # values the bf16 input holds
    return x


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
def test_quantize_rows_bitwise(dtype):
    print(f"[parity-fp8] quantize rows dtype={dtype}", flush=True)
    x = _rows_for_quantiser(np.random.default_rng(3), dtype)
    xd = torch.from_numpy(x).to(dtype).cuda()
    codes = torch.empty(x.shape, dtype=torch.uint8, device="cuda")
    scale = torch.empty(x.shape[0], dtype=torch.float32, device="cuda")
    hilo.hilo_quantize_rows(xd, codes, scale)
    torch.cuda.synchronize()
    want_c, want_s = O.quantize_rows(x)
    np.testing.assert_array_equal(codes.cpu().numpy(), want_c)
    np.testing.assert_array_equal(scale.cpu().numpy(), want_s)
    assert (want_c[11, :4] == np.array([0x7e, 0x38, 0x3a, 0xb8], dtype=np.uint8)).all()
    assert (want_c[3] == 0).all() and want_s[3] == 0.0


def _code_order(c):
    """Position of an E4M3 code on the number line (codes of one sign are monotone in magnitude)."""
    c = c.astype(np.int64)
    return np.where(c & 0x80, -(c & 0x7F), c & 0x7F)


def _align(x):
    return -(-x // 256) * 256


def _ws_h(Tmax, D):
    """Bytes of the workspace's first region: bf16 rows, or FP8 codes plus row scales."""
    return max(_align(Tmax * D * 2), _align(Tmax * D) + _align(Tmax * 4))


def _bf16_rows(ws, off, T, C):
    return torch.from_numpy(ws[off:off + T * C * 2].copy()).view(torch.bfloat16).float().numpy().reshape(T, C)


def _codes_and_scales(ws, off, Tmax, T, C):
    codes = ws[off:off + T * C].reshape(T, C)
    soff = off + _align(Tmax * C)
    return codes, ws[soff:soff + 4 * T].view(np.float32)


def _check_projection_exact(db, wl, T, z_in, z_out, x_bf16, codes, scales, wname, bname, gate_idx):
    """One FP8 projection on the device's own operands: the codes of its bf16 input rows bit for
    bit, then z_out = z_in + gate (dequant(x) dequant(W)^T + b) to float32-accumulation accuracy."""
    want_c, want_s = O.quantize_rows(x_bf16.astype(np.float32))
    np.testing.assert_array_equal(codes, want_c)
    np.testing.assert_array_equal(scales, want_s)
    s = wl.shape
    cu = to_np(db.cu)
    x = O.dequant_rows(codes, scales)
    want = np.empty_like(z_in, dtype=np.float64)
    sname = {"w_o": "s_o", "w2": "s2"}[wname]
    for (smp, sig, a, b) in O._segments(cu, s.text_len):
        wc = db.weights8[sig][wname].cpu().numpy()
        ws = db.weights8[sig][sname].cpu().numpy()
        bias = db.weights[sig][bname].float().cpu().numpy().astype(np.float64)
        o = x[a:b] @ O.dequant_rows(wc, ws).T + bias
        want[a:b] = z_in[a:b] + wl.mod[smp, sig, gate_idx] * o
    # float32 accumulation (the MFMA's own rounding stays below ~1.3e-4 of each 64-term chunk's sum
    # of |terms|) against float64: far inside any FP8 effect, and an O(1) error for a wrong code,
    # scale or column
    ma, rel = float_report(z_out, want)
    assert ma <= 5e-3 and rel <= 1e-3, f"{wname} on the device's codes: max_abs {ma:.3g}, rel {rel:.3g}"
    return ma, rel


def _check_h2_codes(db, z1_dev, wl, T):
    """The MLP's FP8 operand rows as the device left them in the workspace (codes [T][D], then the
    row scales at the next 256-byte boundary) against the oracle's quantisation of
    h2 = LN(z1) (1 + scale2) + shift2 formed from the device's own z1: the two differ only where
    float32 and float64 layer norms round a scaled value to different sides of a code boundary."""
    s = wl.shape
    D, Tmax = s.dim, db.T
    ws = db.ws.cpu().numpy()
    codes = ws[:T * D].reshape(T, D)
    off = (Tmax * D + 255) // 256 * 256
    scales = ws[off:off + 4 * T].view(np.float32)
    cu = to_np(db.cu)
    h2 = np.empty((T, D), dtype=np.float64)
    for (smp, sig, a, b) in O._segments(cu, s.text_len):
        h2[a:b] = O.layer_norm(z1_dev[a:b].astype(np.float64)) * (1.0 + wl.mod[smp, sig, 4]) + wl.mod[smp, sig, 3]
    want_c, want_s = O.quantize_rows(h2.astype(np.float32))
    np.testing.assert_allclose(scales, want_s, rtol=1e-5)
    same = codes == want_c
    frac = same.mean()
    assert frac >= 0.995, f"only {frac:.4f} of the h2 codes match"
    step = np.abs(_code_order(codes[~same]) - _code_order(want_c[~same]))
    assert (step <= 1).all(), "a differing code is not a neighbour of the oracle's"
    return frac


@pytest.mark.parametrize("name", ["small128", "small64"])
def test_fp8_block_parity(name):
    print(f"[parity-fp8] block workload={name}", flush=True)
    wl = inputs.make_workload(name)
    db = DeviceBlock(wl)
    ref = oracle_for(wl, fp8=True)
    ref16 = oracle_for(wl)
    db.prepare_fp8()
    for k in range(2):  # weight codes and scales bit for bit
        for name_w, name_s in (("w_qkv", "s_qkv"), ("w_o", "s_o"), ("w1", "s1"), ("w2", "s2")):
            want_c, want_s = O.quantize_rows(np.asarray(wl.weights[k][name_w], dtype=np.float32))
            np.testing.assert_array_equal(db.weights8[k][name_w].cpu().numpy(), want_c)
            np.testing.assert_array_equal(db.weights8[k][name_s].cpu().numpy(), want_s)
    db.score()
    db.select(hilo.TOPK)
    db.compress()
    torch.cuda.synchronize()
    check_selection(db, ref)
    T = int(ref["cu"][-1])
    Z = ref["Z"][:T]
    z0 = to_np(db.z)[:T].copy()
    db.attention(fp8=True)
    torch.cuda.synchronize()
    z1 = to_np(db.z)[:T].copy()
    assert_close(z1, ref["z1"], "fp8", f"{name} z after FP8 attention")
    s_ = wl.shape
    Tmax, D, F = db.T, s_.dim, s_.mlp_dim
    ws = db.ws.cpu().numpy()
    hsz = _ws_h(Tmax, D)
    a_codes, a_scales = _codes_and_scales(ws, hsz, Tmax, T, D)  # in the QKV region, free after attention
    _check_projection_exact(db, wl, T, z0, z1, _bf16_rows(ws, 0, T, D), a_codes, a_scales, "w_o", "b_o", 2)
    db.mlp(fp8=True)
    torch.cuda.synchronize()
    z2 = to_np(db.z)[:T]
    assert_close(z2, ref["z2"], "fp8", f"{name} z after FP8 mlp")
    ws = db.ws.cpu().numpy()
    # the hidden rows' codes and scales are the last two regions of the FP8 workspace
    hid_off = hilo.hilo_workspace_bytes_fp8(db.shape) - _align(Tmax * F) - _align(Tmax * 4)
    h_codes, h_scales = _codes_and_scales(ws, hid_off, Tmax, T, F)
    _check_projection_exact(db, wl, T, z1, z2, _bf16_rows(ws, hsz, T, F), h_codes, h_scales, "w2", "b2", 5)
    frac = _check_h2_codes(db, z1, wl, T)
    # the device follows the FP8 block, not the bf16 one: on each half's update of z the FP8 and
    # bf16 oracles differ by ~3% (relative L2); the device is well inside that
    for tag, got, want8, want16 in (("attention", z1 - Z, ref["z1"] - Z, ref16["z1"] - Z),
                                    ("mlp", z2 - z1, ref["z2"] - ref["z1"], ref16["z2"] - ref16["z1"])):
        _, e8 = float_report(got, want8)
        _, gap = float_report(want8, want16)
        print(f"[parity-fp8] {name} {tag} update: rel to FP8 oracle {e8:.3g}, FP8 vs bf16 oracle {gap:.3g}",
              flush=True)
        assert e8 < 0.4 * gap, f"{tag}: device update is not closer to the FP8 oracle ({e8:.3g} vs {gap:.3g})"
    db.decompress()
    torch.cuda.synchronize()
    assert_close(to_np(db.y_img), ref["y_img"], "fp8", f"{name} y_img")
    assert_close(to_np(db.y_txt), ref["y_txt"], "fp8", f"{name} y_txt")
    print(f"[parity-fp8] {name}: h2 codes equal {frac:.5f}", flush=True)


# The schedules of the FP8 256 x 256 tiling on a 256-CU device (every block kept fine, so the row
# counts are fixed).  With K = dim <= 8192 an FP8 projection has at most 64 K steps of 128, so a
# problem below one wave of tiles always runs whole tiles; the two larger problems reach the
# stream-K tail (partials in the bf16 fragment layout, finished by the fixup) and the rule that
# prefers two waves of whole tiles.
@pytest.mark.parametrize("shp", [
    # 17 row tiles x 16 column tiles = 272 MLP-up tiles: one wave plus a 16-tile stream-K tail
    inputs.BlockShape(1, 1, 64, 64, 256, 256, 2, 128, 4096, "bf16"),
    # 17 x 24 = 408 MLP-up tiles: two waves of whole tiles
    inputs.BlockShape(1, 1, 64, 64, 256, 256, 2, 128, 6144, "bf16"),
    # K = 4608 in 36 steps of 128, few tiles: whole tiles; MLP up N = 1152 ends in a 128-column tile;
    # MLP down has K = 1152, 9 steps of 128
    inputs.BlockShape(1, 1, 16, 16, 0, 4608, 36, 128, 1152, "bf16"),
], ids=["sk_tail", "whole_waves", "long_k"])
def test_fp8_gemm_schedules(shp):
    print(f"[parity-fp8] 256-tile FP8 schedules shape={shp}", flush=True)
    wl = inputs.make_workload("splitk", shape=shp, seed=5, keep_frac=1.0)
    db = DeviceBlock(wl)
    ref = oracle_for(wl, fp8=True)
    db.run(hilo.TOPK, fp8=True)
    torch.cuda.synchronize()
    check_selection(db, ref)
    T = int(ref["cu"][-1])
    assert_close(to_np(db.z)[:T], ref["z2"], "fp8", "z after FP8 block")
    assert_close(to_np(db.y_img), ref["y_img"], "fp8", "y_img")


def test_fp8_full_size_sampled():
    """The 1024 px workload (2766 tokens at 40% kept, dim 3072, MLP 12288) in the benchmark's launch
    configuration, block outputs on a seeded sample of rows."""
    from test_parity_full_gpu import _sample_rows

    print("[parity-fp8] full size m1024", flush=True)
    wl = inputs.make_workload("m1024")
    s = wl.shape
    db = DeviceBlock(wl)
    db.run(hilo.TOPK, fp8=True)
    torch.cuda.synchronize()
    front = oracle_for(wl, with_block=False)
    check_selection(db, front)
    rows = _sample_rows(front["counts"], front["cu"], front["seg"], s.images, s.text_len, per_seg=4)
    q8 = O.quantize_fp8_weights(wl.weights)
    _, z2 = O.block(front["Z"], front["cu"], s.text_len, s.heads, wl.weights, wl.mod, rows, q8)
    got = to_np(db.z)[rows]
    ma, rel = assert_close(got, z2, "fp8", "m1024 FP8 z at sampled rows")
    print(f"[parity-fp8] m1024: {rows.size} rows, max_abs {ma:.3g}, rel_l2 {rel:.3g}", flush=True)
