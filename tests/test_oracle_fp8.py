"""FP8 E4M3 codes and per-row quantisation of the oracle, pinned by hand-worked bit patterns."""
import numpy as np
import pytest

from oracle import hilo_oracle as O
from paper_2606_13898_amd import inputs


def test_e4m3_decoding_of_hand_worked_codes():
    # 0x38 = 0 0111 000 = 1.0; 0x30 = 0.5; 0x7e = 0 1111 110 = 1.75 * 2^8 = 448; 0x77 = 1.875 * 2^7
    # = 240; 0x01 = 2^-9 (smallest subnormal); 0x08 = 2^-6 (smallest normal); 0xb8 = -1.0
    codes = np.array([0x38, 0x30, 0x7e, 0x77, 0x01, 0x08, 0xb8, 0x00, 0x3a], dtype=np.uint8)
    np.testing.assert_array_equal(O.e4m3_value(codes), [1.0, 0.5, 448.0, 240.0, 2.0 ** -9, 2.0 ** -6, -1.0, 0.0, 1.25])
    assert np.isnan(O.e4m3_value(np.array([0x7f], dtype=np.uint8)))[0]


def test_quantize_row_with_max_448_keeps_exact_values_and_rounds_ties_to_even():
    # amax = 448 -> inv = 1: values encode directly.  1.0625 lies halfway between 1.0 (mantissa 000)
    # and 1.125 (001): even -> 1.0; 1.1875 halfway between 1.125 (001) and 1.25 (010): even -> 1.25
    x = np.array([[448.0, -448.0, 1.0, 0.5, 240.0, 1.0625, 1.1875, 0.0]], dtype=np.float32)
    codes, scale = O.quantize_rows(x)
    np.testing.assert_array_equal(codes[0], [0x7e, 0xfe, 0x38, 0x30, 0x77, 0x38, 0x3a, 0x00])
    assert scale[0] == np.float32(1.0)


def test_quantize_zero_row_and_scaled_row():
    codes, scale = O.quantize_rows(np.zeros((1, 8), dtype=np.float32))
    assert (codes == 0).all() and scale[0] == 0
    # row [2, 1, 0.5]: amax 2 -> inv 224, values 448, 224, 112 -> codes 0x7e, 0x76 (1.75 * 2^7), 0x6e
    codes, scale = O.quantize_rows(np.array([[2.0, 1.0, 0.5]], dtype=np.float32))
    np.testing.assert_array_equal(codes[0], [0x7e, 0x76, 0x6e])
    assert scale[0] == np.float32(2.0 / 448.0)
    np.testing.assert_allclose(O.dequant_rows(codes, scale)[0], [2.0, 1.0, 0.5], rtol=1e-6)


def test_quantisation_error_is_within_half_an_e4m3_step():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((16, 256)).astype(np.float32)
    codes, scale = O.quantize_rows(x)
    err = np.abs(O.dequant_rows(codes, scale) - x) / np.abs(x).max(axis=1, keepdims=True)
    assert err.max() <= 2.0 ** -4 / 2 * 448 / 256 + 1e-6  # half a step at the top binade, relative to amax


def test_fp8_block_stays_close_to_the_bf16_block():
    shp = inputs.BlockShape(1, 1, 8, 10, 4, 256, 2, 128, 1024, "bf16")
    wl = inputs.make_workload("smallx", shape=shp, seed=51)
    a = O.pipeline(wl.x_img, wl.x_txt, shp, None, 0, "topk", keep=wl.keep, weights=wl.weights, mod=wl.mod)
    b = O.pipeline(wl.x_img, wl.x_txt, shp, None, 0, "topk", keep=wl.keep, weights=wl.weights, mod=wl.mod, fp8=True)
    d = np.abs(b["y_img"] - a["y_img"]).max()
    assert 0 < d < 0.1


def test_fp8_product_of_exactly_representable_rows_is_the_plain_product():
    # rows whose amax is 448 and whose entries are E4M3 values quantise to themselves (scale 1), so
    # the FP8 product is the exact product; a row scaled by 2^-3 keeps exact codes with scale 2^-3
    rng = np.random.default_rng(5)
    vals = O.e4m3_value(np.arange(0x00, 0x7f, dtype=np.uint8))
    h = rng.choice(vals, size=(3, 16)) * rng.choice([-1.0, 1.0], size=(3, 16))
    w = rng.choice(vals, size=(5, 16)) * rng.choice([-1.0, 1.0], size=(5, 16))
    h[:, 0], w[:, 0] = 448.0, 448.0
    h[2] *= 0.125
    got = O._fp8_matmul(h.astype(np.float32), O.quantize_rows(w.astype(np.float32)))
    np.testing.assert_array_equal(got, h @ w.T)


def test_fp8_block_quantises_all_four_projections():
    # zero the output and down projection weights of one stream's FP8 codes only: the FP8 block's
    # update then differs from the one with full codes, so those projections do read FP8 weights
    shp = inputs.BlockShape(1, 1, 8, 10, 4, 256, 2, 128, 1024, "bf16")
    wl = inputs.make_workload("smallx", shape=shp, seed=52)
    res = O.pipeline(wl.x_img, wl.x_txt, shp, None, 0, "topk", keep=wl.keep, with_block=False)
    q = O.quantize_fp8_weights(wl.weights)
    assert set(q[0]) == {"w_qkv", "w_o", "w1", "w2"}
    z1, z2 = O.block(res["Z"], res["cu"], shp.text_len, shp.heads, wl.weights, wl.mod, fp8=q)
    for name in ("w_o", "w2"):
        q0 = [dict(d) for d in q]
        for d in q0:
            d[name] = (np.zeros_like(d[name][0]), d[name][1])
        y1, y2 = O.block(res["Z"], res["cu"], shp.text_len, shp.heads, wl.weights, wl.mod, fp8=q0)
        assert np.abs(y2 - z2).max() > 1e-4, name
        if name == "w_o":
            # with the output projection zeroed the attention half adds the gated bias only
            Z = res["Z"]
            for (s_, sig, a, b) in O._segments(res["cu"], shp.text_len):
                np.testing.assert_allclose(y1[a:b], Z[a:b] + wl.mod[s_, sig, 2] * np.asarray(wl.weights[sig]["b_o"], np.float64), atol=1e-12)


def test_pow2_exponent_is_the_least_power_of_two_scale():
    # against a brute-force search over k of the defining inequality 448 * 2^k >= amax
    rng = np.random.default_rng(7)
    amax = np.concatenate([np.float32([448.0, 449.0, 224.0, 0.875, 1.0, 3.0e-30, 1.0e30]),
                           np.exp2(rng.uniform(-60, 60, 200)).astype(np.float32)])
    k = O.pow2_exponent(amax)
    for a, kk in zip(amax.astype(np.float64), k):
        want = next(j for j in range(-140, 140) if 448.0 * 2.0 ** j >= a)
        assert kk == max(want, -127), (a, kk, want)
    assert O.pow2_exponent(np.float32([0.0]))[0] == 0
    # hand-worked: 448 -> 0, 449 -> 1 (448 < 449 <= 896), 224 -> -1, 1.0 -> -8 (448 / 256 = 1.75 >= 1)
    np.testing.assert_array_equal(k[:5], [0, 1, -1, -9, -8])


def test_pow2_quantisation_of_representable_rows_is_exact():
    # entries that are E4M3 values times 2^j with the row's max code 448: codes come back exactly and
    # the exponent is j; a row of zeros gives zero codes
    rng = np.random.default_rng(8)
    vals = O.e4m3_value(np.arange(0x00, 0x7f, dtype=np.uint8))
    base = rng.choice(vals, size=(4, 32)) * rng.choice([-1.0, 1.0], size=(4, 32))
    base[:, 3] = 448.0
    j = np.array([0, -5, 7, -20])
    x = (base * np.exp2(j)[:, None]).astype(np.float32)
    codes, k = O.quantize_rows_pow2(x)
    np.testing.assert_array_equal(k, j)
    np.testing.assert_array_equal(O.dequant_rows_pow2(codes, k), x.astype(np.float64))
    codes, k = O.quantize_rows_pow2(np.zeros((1, 8), dtype=np.float32))
    assert (codes == 0).all() and k[0] == 0


def test_pow2_quantisation_error_is_within_half_an_e4m3_step():
    # a normal E4M3 code is off by at most half its step, 2^-4 of its magnitude; below 2^-6 (in code
    # units) the subnormal step 2^-9 bounds the absolute error
    rng = np.random.default_rng(9)
    x = (rng.standard_normal((32, 128)) * np.exp2(rng.uniform(-10, 10, (32, 1)))).astype(np.float32)
    codes, k = O.quantize_rows_pow2(x)
    y = x.astype(np.float64) * np.exp2(-k.astype(np.float64))[:, None]
    assert np.abs(y).max() <= 448.0
    err = np.abs(O.e4m3_value(codes) - y)
    assert (err <= np.maximum(2.0 ** -4 * np.abs(y), 2.0 ** -10) + 1e-12).all()


def test_fp8_scores_of_representable_q_and_k_equal_the_plain_attention():
    # q and k rows that quantise exactly (E4M3 values times a power of two, max code 448 per head)
    # give the FP8-score attention exactly the float64 attention
    rng = np.random.default_rng(10)
    vals = O.e4m3_value(np.arange(0x00, 0x60, dtype=np.uint8))
    heads, hd, n = 2, 64, 12
    q = rng.choice(vals, size=(n, heads * hd)) * rng.choice([-1.0, 1.0], size=(n, heads * hd))
    k = rng.choice(vals, size=(n, heads * hd)) * rng.choice([-1.0, 1.0], size=(n, heads * hd))
    for hh in range(heads):
        q[:, hh * hd] = 448.0
        k[:, hh * hd + 1] = -448.0
    q *= 2.0 ** -9
    k *= 2.0 ** -8
    v = rng.standard_normal((n, heads * hd))
    np.testing.assert_allclose(O._attend_fp8(q, k, v, heads), O._attend(q, k, v, heads), rtol=0, atol=1e-12)


def test_attend_codes_is_the_fp8_attention_after_quantisation():
    rng = np.random.default_rng(11)
    heads, hd, n = 2, 128, 20
    q, k, v = (rng.standard_normal((n, heads * hd)) for _ in range(3))
    qc = np.empty((n, heads * hd), np.uint8); kc = np.empty_like(qc)
    qe = np.empty((n, heads), np.int64); ke = np.empty_like(qe)
    for hh in range(heads):
        cols = slice(hh * hd, (hh + 1) * hd)
        qc[:, cols], qe[:, hh] = O.quantize_rows_pow2(q[:, cols].astype(np.float32))
        kc[:, cols], ke[:, hh] = O.quantize_rows_pow2(k[:, cols].astype(np.float32))
    np.testing.assert_array_equal(O.attend_codes(qc, qe, kc, ke, v, heads), O._attend_fp8(q, k, v, heads))
    # and the FP8 scores stay close to the exact ones.  Rounding to E4M3 leaves a relative error of
    # RMS ~2^-4 / sqrt(3) ~ 3.6% per operand entry, so for unit-variance q and k a score (its
    # variance 1) moves by ~sqrt(2) * 3.6% ~ 5% RMS, and the softmax-weighted mean of v moves by a
    # fraction of that relative to its own size: the relative L2 stays well under 10%
    a, b = O._attend_fp8(q, k, v, heads), O._attend(q, k, v, heads)
    rel = np.linalg.norm(a - b) / np.linalg.norm(b)
    assert 0 < rel < 0.1
