"""The C-ABI library on the host: it loads, exports every declared entry point, and validates its
arguments before touching a device (CPU only; no kernel is launched here)."""
import ctypes
import math
import os
import re

import pytest
import torch

from paper_2606_13898_amd import hilo

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hilo.h")

pytestmark = pytest.mark.skipif(not os.path.exists(hilo.LIB_PATH), reason="libhilo.so not built")


def declared_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(hilo_[a-z_0-9]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    L = hilo.lib()
    names = declared_symbols()
    assert len(names) >= 15
    for n in names:
        assert hasattr(L, n), n


def test_version_and_status_strings():
    assert hilo.hilo_abi_version() == 6
    for st in range(7):
        assert hilo.status_str(st)
    assert hilo.status_str(99) == "unknown status"


def good_shape(dtype=hilo.BF16):
    return hilo.hilo_shape(2, 1, 8, 10, 5, 256, 2, 128, 1024, dtype)


def test_max_tokens_and_workspace():
    s = good_shape()
    assert hilo.hilo_max_tokens(s) == 2 * (80 + 20 + 5)  # every patch fine plus a pooled token per block
    T = 210
    part = 256 * 3 * 256 * 256 * 4  # GEMM partial tiles: 3 slots of 256 x 256 fp32 per CU, at most 256 CUs
    want = max(-(-T * 256 * 2 // 256) * 256 + -(-T * 768 * 2 // 256) * 256,
               -(-T * 256 * 2 // 256) * 256 + -(-T * 1024 * 2 // 256) * 256) + part
    assert hilo.hilo_workspace_bytes(s) == want
    f = good_shape(hilo.F32)
    assert hilo.hilo_workspace_bytes(f) == max(-(-T * 256 * 4 // 256) * 256 + -(-T * 768 * 4 // 256) * 256,
                                               -(-T * 256 * 4 // 256) * 256 + -(-T * 1024 * 4 // 256) * 256)
    bad = good_shape()
    bad.grid_h = 7
    assert hilo.hilo_max_tokens(bad) == -1
    assert hilo.hilo_workspace_bytes(bad) == 0


FAKE = 0x1000  # never dereferenced: validation rejects or the missing device stops the call


def call_score(shape, x=FAKE, e=FAKE):
    return hilo.lib().hilo_score(ctypes.byref(shape), x, e, None)


def call_select(shape, mode=hilo.TOPK, tau=None, keep=None, r=0, ptrs=FAKE):
    G = shape.batch * shape.images if shape.batch > 0 and shape.images > 0 else 1
    t = (ctypes.c_double * G)(*(tau or [0.1] * G))
    k = (ctypes.c_int32 * G)(*(keep or [1] * G))
    return hilo.lib().hilo_select(ctypes.byref(shape), FAKE, None, r, mode, t, k,
                                  ptrs, FAKE, FAKE, FAKE, FAKE, FAKE, None)


@pytest.mark.parametrize("field,value,status", [
    ("grid_h", 7, 2), ("grid_w", 0, 2), ("batch", 0, 2), ("dim", 100, 2), ("dim", 8256, 2),
    ("text_len", -1, 2), ("dtype", 5, 3),
])
def test_shape_validation(field, value, status):
    s = good_shape()
    setattr(s, field, value)
    assert call_score(s) == status


def test_block_shape_validation():
    L = hilo.lib()
    s = good_shape()
    s.heads = 3  # 3 * 128 != 256
    aw = (hilo.hilo_attn_w * 2)(*[hilo.hilo_attn_w(FAKE, FAKE, FAKE, FAKE)] * 2)
    assert L.hilo_attention(ctypes.byref(s), FAKE, FAKE, aw, FAKE, FAKE, 1 << 40, None) == 2
    s = good_shape()
    s.head_dim, s.heads = 32, 8
    assert L.hilo_attention(ctypes.byref(s), FAKE, FAKE, aw, FAKE, FAKE, 1 << 40, None) == 3
    s = good_shape()
    s.mlp_dim = 1000
    mw = (hilo.hilo_mlp_w * 2)(*[hilo.hilo_mlp_w(FAKE, FAKE, FAKE, FAKE)] * 2)
    assert L.hilo_mlp(ctypes.byref(s), FAKE, FAKE, mw, FAKE, FAKE, 1 << 40, None) == 2


def test_null_pointers():
    s = good_shape()
    assert call_score(s, x=None) == 1
    assert call_score(s, e=None) == 1
    assert hilo.lib().hilo_score(None, FAKE, FAKE, None) == 1
    assert call_select(s, ptrs=None) == 1
    L = hilo.lib()
    aw = (hilo.hilo_attn_w * 2)(hilo.hilo_attn_w(FAKE, FAKE, FAKE, FAKE), hilo.hilo_attn_w(FAKE, None, FAKE, FAKE))
    assert L.hilo_attention(ctypes.byref(s), FAKE, FAKE, aw, FAKE, FAKE, 1 << 40, None) == 1
    assert L.hilo_decompress(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, None, None, None) == 1
    assert L.hilo_compress(ctypes.byref(s), FAKE, None, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None) == 1


def test_fused_compress_norm_validation():
    """hilo_compress_norm / hilo_attention_normed: block shape, pointers and workspace checked
    before anything is enqueued (status codes as hilo_compress and hilo_attention)."""
    L = hilo.lib()
    s = good_shape()
    need = hilo.hilo_workspace_bytes(s)
    aw = (hilo.hilo_attn_w * 2)(*[hilo.hilo_attn_w(FAKE, FAKE, FAKE, FAKE)] * 2)

    def cn(shape, mod=FAKE, ws=FAKE, nbytes=1 << 40, x_txt=FAKE):
        return L.hilo_compress_norm(ctypes.byref(shape), FAKE, x_txt, FAKE, FAKE, FAKE, FAKE, FAKE, mod,
                                    FAKE, ws, nbytes, None)

    bad = good_shape()
    bad.heads = 3  # not a block shape: heads * head_dim != dim
    assert cn(bad) == 2
    grid = good_shape()
    grid.grid_w = 9  # odd grid
    assert cn(grid) == 2
    assert cn(s, mod=None) == 1
    assert cn(s, ws=None) == 1
    assert cn(s, x_txt=None) == 1  # text_len > 0 needs the text rows
    assert cn(s, nbytes=100) == 5
    assert L.hilo_attention_normed(ctypes.byref(bad), FAKE, FAKE, aw, FAKE, FAKE, 1 << 40, None) == 2
    assert L.hilo_attention_normed(ctypes.byref(s), FAKE, FAKE, aw, None, FAKE, 1 << 40, None) == 1
    assert L.hilo_attention_normed(ctypes.byref(s), FAKE, FAKE, aw, FAKE, FAKE, 100, None) == 5
    if not torch.cuda.is_available():
        assert cn(s, nbytes=need) == 6
        assert L.hilo_attention_normed(ctypes.byref(s), FAKE, FAKE, aw, FAKE, FAKE, need, None) == 6


def test_fused_compress_norm_fp8_validation():
    """The FP8 block's pair: an FP8 block shape, pointers and the FP8 workspace checked first."""
    L = hilo.lib()
    s = good_shape()
    need = hilo.hilo_workspace_bytes_fp8(s)
    aw8 = (hilo.hilo_attn_w_fp8 * 2)(*[hilo.hilo_attn_w_fp8(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE)] * 2)

    def cn(shape, mod=FAKE, nbytes=1 << 40):
        return L.hilo_compress_norm_fp8(ctypes.byref(shape), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, mod,
                                        FAKE, FAKE, nbytes, None)

    odd = good_shape()
    odd.dim, odd.heads = 384, 3  # a block shape, but not a multiple of 256
    assert cn(odd) == 2
    f32 = good_shape(hilo.F32)
    assert cn(f32) == 3
    assert cn(s, mod=None) == 1
    assert cn(s, nbytes=100) == 5
    assert L.hilo_attention_fp8_normed(ctypes.byref(odd), FAKE, FAKE, aw8, FAKE, FAKE, 1 << 40, None) == 2
    assert L.hilo_attention_fp8_normed(ctypes.byref(s), FAKE, FAKE, aw8, FAKE, FAKE, 100, None) == 5
    if not torch.cuda.is_available():
        assert cn(s, nbytes=need) == 6
        assert L.hilo_attention_fp8_normed(ctypes.byref(s), FAKE, FAKE, aw8, FAKE, FAKE, need, None) == 6


def test_select_parameter_validation():
    s = good_shape()
    NB = 8 * 10 // 4
    assert call_select(s, mode=7) == 4
    assert call_select(s, r=-1) == 4
    assert call_select(s, keep=[NB + 1, 0]) == 4
    assert call_select(s, keep=[-1, 0]) == 4
    assert call_select(s, mode=hilo.THRESHOLD, tau=[math.nan, 0.1]) == 4
    assert call_select(s, mode=hilo.THRESHOLD, tau=[math.inf, 0.1]) == 4


def test_workspace_too_small():
    s = good_shape()
    need = hilo.hilo_workspace_bytes(s)
    aw = (hilo.hilo_attn_w * 2)(*[hilo.hilo_attn_w(FAKE, FAKE, FAKE, FAKE)] * 2)
    assert hilo.lib().hilo_attention(ctypes.byref(s), FAKE, FAKE, aw, FAKE, FAKE, 100, None) == 5
    mw = (hilo.hilo_mlp_w * 2)(*[hilo.hilo_mlp_w(FAKE, FAKE, FAKE, FAKE)] * 2)
    assert hilo.lib().hilo_mlp(ctypes.byref(s), FAKE, FAKE, mw, FAKE, FAKE, need - 1, None) == 5


@pytest.mark.skipif(torch.cuda.is_available(), reason="checks the no-device path")
def test_valid_calls_without_a_device_report_device_error():
    s = good_shape()
    assert call_score(s) == 6
    assert call_select(s) == 6
    assert call_select(s, mode=hilo.THRESHOLD, tau=[0.1, 0.2]) == 6
    aw = (hilo.hilo_attn_w * 2)(*[hilo.hilo_attn_w(FAKE, FAKE, FAKE, FAKE)] * 2)
    assert hilo.lib().hilo_attention(ctypes.byref(s), FAKE, FAKE, aw, FAKE, FAKE, 1 << 40, None) == 6
    assert hilo.lib().hilo_attention_core(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, 1 << 40, None) == 6
    assert hilo.lib().hilo_attention_core(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, 10, None) == 5


def test_profile_api():
    n = hilo.hilo_profile_kinds()
    assert n >= 10
    names = [hilo.hilo_profile_name(k) for k in range(n)]
    assert "attention_core" in names and "score" in names
    hilo.hilo_profile_enable(True)
    ms, cnt = hilo.hilo_profile_read(0)
    assert ms == 0.0 and cnt == 0
    hilo.hilo_profile_enable(False)
    with pytest.raises(hilo.HiloError):
        hilo.hilo_profile_read(n)


def test_binding_refuses_host_tensors():
    s = good_shape()
    with pytest.raises(ValueError):
        hilo.hilo_score(s, torch.zeros(4), torch.zeros(4))


def test_blocks_validation():
    """hilo_blocks checks every block's pointers and the count before enqueuing anything."""
    s = good_shape()
    L = hilo.lib()
    need = hilo.hilo_workspace_bytes(s)
    n = 3
    aw = (hilo.hilo_attn_w * (2 * n))(*[hilo.hilo_attn_w(FAKE, FAKE, FAKE, FAKE)] * (2 * n))
    mw = (hilo.hilo_mlp_w * (2 * n))(*[hilo.hilo_mlp_w(FAKE, FAKE, FAKE, FAKE)] * (2 * n))
    assert L.hilo_blocks(ctypes.byref(s), FAKE, FAKE, aw, mw, FAKE, -1, FAKE, need, None) == 4
    assert L.hilo_blocks(ctypes.byref(s), None, FAKE, aw, mw, FAKE, n, FAKE, need, None) == 1
    assert L.hilo_blocks(ctypes.byref(s), FAKE, FAKE, None, mw, FAKE, n, FAKE, need, None) == 1
    assert L.hilo_blocks(ctypes.byref(s), FAKE, FAKE, aw, mw, None, n, FAKE, need, None) == 1
    assert L.hilo_blocks(ctypes.byref(s), FAKE, FAKE, aw, mw, FAKE, n, FAKE, need - 1, None) == 5
    bad_aw = (hilo.hilo_attn_w * (2 * n))(*[hilo.hilo_attn_w(FAKE, FAKE, FAKE, FAKE)] * (2 * n))
    bad_aw[5] = hilo.hilo_attn_w(FAKE, FAKE, None, FAKE)  # last block's text stream
    assert L.hilo_blocks(ctypes.byref(s), FAKE, FAKE, bad_aw, mw, FAKE, n, FAKE, need, None) == 1
    bad_mw = (hilo.hilo_mlp_w * (2 * n))(*[hilo.hilo_mlp_w(FAKE, FAKE, FAKE, FAKE)] * (2 * n))
    bad_mw[2] = hilo.hilo_mlp_w(FAKE, FAKE, FAKE, None)
    assert L.hilo_blocks(ctypes.byref(s), FAKE, FAKE, aw, bad_mw, FAKE, n, FAKE, need, None) == 1
    s.heads, s.head_dim = 8, 32  # a head size the attention kernels do not take
    assert L.hilo_blocks(ctypes.byref(s), FAKE, FAKE, aw, mw, FAKE, n, FAKE, need, None) == 3


def test_select_tokens_validation():
    s = good_shape()
    L = hilo.lib()
    G = 2
    keep = (ctypes.c_int32 * G)(1, 2)
    args = lambda tset: (ctypes.byref(s), FAKE, None, 0, hilo.TOPK, None, keep, tset, FAKE, FAKE, FAKE, FAKE,
                         FAKE, FAKE, None)
    assert L.hilo_select_tokens(*args(3)) == 4
    assert L.hilo_select_tokens(*args(-1)) == 4
    assert L.hilo_decompress_delta(ctypes.byref(s), FAKE, None, FAKE, FAKE, FAKE, FAKE, FAKE, None, None) == 1
    assert L.hilo_decompress_delta(ctypes.byref(s), FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE, None, None) == 1


def test_fp8_validation():
    """The FP8 block takes bf16 shapes with dim % 256 == 0 (whole heads of q and k in each 256-column
    tile of the QKV projection), mlp_dim % 128 == 0 and every weight pointer, scales included; the
    row quantiser takes float32 / bf16 rows of a multiple of 4 columns."""
    L = hilo.lib()
    s = good_shape()
    need = hilo.hilo_workspace_bytes(s)
    aw = (hilo.hilo_attn_w_fp8 * 2)(*[hilo.hilo_attn_w_fp8(*[FAKE] * 6)] * 2)
    mw = (hilo.hilo_mlp_w_fp8 * 2)(*[hilo.hilo_mlp_w_fp8(*[FAKE] * 6)] * 2)
    need8 = hilo.hilo_workspace_bytes_fp8(s)
    assert need8 > need  # one more region on top: the attention output, later the hidden rows' codes
    T, F, D = hilo.hilo_max_tokens(s), s.mlp_dim, s.dim
    up = lambda x: -(-x // 256) * 256  # noqa: E731
    assert need8 == need + max(up(T * F) + up(T * 4), up(T * D * 2))
    f = good_shape(hilo.F32)
    assert L.hilo_attention_fp8(ctypes.byref(f), FAKE, FAKE, aw, FAKE, FAKE, 1 << 40, None) == 3
    assert L.hilo_mlp_fp8(ctypes.byref(f), FAKE, FAKE, mw, FAKE, FAKE, 1 << 40, None) == 3
    odd = hilo.hilo_shape(2, 1, 8, 10, 5, 192, 3, 64, 1024, hilo.BF16)  # 192 is not a multiple of 128
    assert L.hilo_attention_fp8(ctypes.byref(odd), FAKE, FAKE, aw, FAKE, FAKE, 1 << 40, None) == 2
    assert L.hilo_mlp_fp8(ctypes.byref(odd), FAKE, FAKE, mw, FAKE, FAKE, 1 << 40, None) == 2
    odd_d = hilo.hilo_shape(2, 1, 8, 10, 5, 384, 3, 128, 1024, hilo.BF16)  # 384 is not a multiple of 256
    assert L.hilo_attention_fp8(ctypes.byref(odd_d), FAKE, FAKE, aw, FAKE, FAKE, 1 << 40, None) == 2
    assert L.hilo_attention_core_fp8(ctypes.byref(odd_d), FAKE, FAKE, FAKE, FAKE, 1 << 40, None) == 2
    assert hilo.hilo_workspace_bytes_fp8(odd_d) == 0
    core8 = L.hilo_attention_core_fp8
    assert core8(ctypes.byref(f), FAKE, FAKE, FAKE, FAKE, 1 << 40, None) == 3
    assert core8(ctypes.byref(s), None, FAKE, FAKE, FAKE, 1 << 40, None) == 1
    assert core8(ctypes.byref(s), FAKE, FAKE, FAKE, None, 1 << 40, None) == 1
    assert core8(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, 10, None) == 5
    odd_f = hilo.hilo_shape(2, 1, 8, 10, 5, 256, 2, 128, 1088, hilo.BF16)  # mlp_dim 1088: K of MLP down
    assert L.hilo_mlp_fp8(ctypes.byref(odd_f), FAKE, FAKE, mw, FAKE, FAKE, 1 << 40, None) == 2
    assert hilo.hilo_workspace_bytes_fp8(odd_f) == 0
    bad_aw = (hilo.hilo_attn_w_fp8 * 2)(*[hilo.hilo_attn_w_fp8(*[FAKE] * 6)] * 2)
    bad_aw[1] = hilo.hilo_attn_w_fp8(FAKE, FAKE, FAKE, FAKE, None, FAKE)  # text stream without W_o scales
    assert L.hilo_attention_fp8(ctypes.byref(s), FAKE, FAKE, bad_aw, FAKE, FAKE, need8, None) == 1
    bad_mw = (hilo.hilo_mlp_w_fp8 * 2)(*[hilo.hilo_mlp_w_fp8(*[FAKE] * 6)] * 2)
    bad_mw[0] = hilo.hilo_mlp_w_fp8(FAKE, None, FAKE, FAKE, FAKE, FAKE)
    assert L.hilo_mlp_fp8(ctypes.byref(s), FAKE, FAKE, bad_mw, FAKE, FAKE, need8, None) == 1
    assert L.hilo_attention_fp8(ctypes.byref(s), FAKE, FAKE, aw, FAKE, FAKE, 100, None) == 5
    assert L.hilo_attention_fp8(ctypes.byref(s), FAKE, FAKE, aw, FAKE, FAKE, need8 - 1, None) == 5
    assert L.hilo_mlp_fp8(ctypes.byref(s), FAKE, FAKE, mw, FAKE, FAKE, need8 - 1, None) == 5
    assert L.hilo_attention_fp8(ctypes.byref(s), None, FAKE, aw, FAKE, FAKE, need, None) == 1
    q = L.hilo_quantize_rows
    assert q(2, FAKE, 4, 8, FAKE, FAKE, None) == 3      # dtype
    assert q(hilo.BF16, FAKE, 4, 6, FAKE, FAKE, None) == 2   # cols % 4
    assert q(hilo.BF16, FAKE, -1, 8, FAKE, FAKE, None) == 2
    assert q(hilo.BF16, FAKE, 4, 0, FAKE, FAKE, None) == 2
    assert q(hilo.BF16, FAKE, 1 << 31, 8, FAKE, FAKE, None) == 2
    assert q(hilo.BF16, FAKE, 4, 8, None, FAKE, None) == 1
    assert q(hilo.F32, FAKE, 0, 8, FAKE, FAKE, None) == 0    # nothing to do
    if not torch.cuda.is_available():
        assert q(hilo.F32, FAKE, 4, 8, FAKE, FAKE, None) == 6
        assert L.hilo_attention_fp8(ctypes.byref(s), FAKE, FAKE, aw, FAKE, FAKE, need8, None) == 6
        assert L.hilo_mlp_fp8(ctypes.byref(s), FAKE, FAKE, mw, FAKE, FAKE, need8, None) == 6
        assert core8(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, need8, None) == 6
