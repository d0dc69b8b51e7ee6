"""Python binding of libhilo.so: argument marshalling only.

Every function here has the name of its C entry point (include/hilo.h), takes torch tensors that
already live on the GPU, passes their device pointers and the current HIP stream to the library,
and raises HiloError on a non-zero status.  All arithmetic happens in the library's kernels; there
is no fallback of any kind -- without the built library every call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libhilo.so")

F32, BF16 = 0, 1
THRESHOLD, TOPK = 0, 1
PARTITION, OVERLAP, DROP = 0, 1, 2  # hilo_token_set
DTYPES = {"f32": F32, "bf16": BF16}
TORCH_DTYPES = {F32: torch.float32, BF16: torch.bfloat16}


class HiloError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__(f"{fn} failed with status {status}: {status_str(status)}")


class hilo_shape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("batch", "images", "grid_h", "grid_w", "text_len", "dim", "heads", "head_dim",
                 "mlp_dim", "dtype")]


class hilo_attn_w(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("w_qkv", "b_qkv", "w_o", "b_o")]


class hilo_mlp_w(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("w1", "b1", "w2", "b2")]


class hilo_attn_w_fp8(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("w_qkv", "s_qkv", "b_qkv", "w_o", "s_o", "b_o")]


class hilo_mlp_w_fp8(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("w1", "s1", "b1", "w2", "s2", "b2")]


_lib = None

_P = ctypes.c_void_p
_SIG = {
    "hilo_score": [ctypes.POINTER(hilo_shape), _P, _P, _P],
    "hilo_score_pixels": [ctypes.POINTER(hilo_shape), _P, _P, _P],
    "hilo_select": [ctypes.POINTER(hilo_shape), _P, _P, ctypes.c_int32, ctypes.c_int32,
                    ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int32),
                    _P, _P, _P, _P, _P, _P, _P],
    "hilo_select_tokens": [ctypes.POINTER(hilo_shape), _P, _P, ctypes.c_int32, ctypes.c_int32,
                           ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int32),
                           ctypes.c_int32, _P, _P, _P, _P, _P, _P, _P],
    "hilo_compress": [ctypes.POINTER(hilo_shape), _P, _P, _P, _P, _P, _P, _P, _P, _P],
    "hilo_compress_norm": [ctypes.POINTER(hilo_shape), _P, _P, _P, _P, _P, _P, _P, _P, _P, _P,
                           ctypes.c_size_t, _P],
    "hilo_attention_normed": [ctypes.POINTER(hilo_shape), _P, _P, ctypes.POINTER(hilo_attn_w), _P, _P,
                              ctypes.c_size_t, _P],
    "hilo_decompress_delta": [ctypes.POINTER(hilo_shape), _P, _P, _P, _P, _P, _P, _P, _P, _P],
    "hilo_attention": [ctypes.POINTER(hilo_shape), _P, _P, ctypes.POINTER(hilo_attn_w), _P, _P,
                       ctypes.c_size_t, _P],
    "hilo_mlp": [ctypes.POINTER(hilo_shape), _P, _P, ctypes.POINTER(hilo_mlp_w), _P, _P,
                 ctypes.c_size_t, _P],
    "hilo_compress_norm_fp8": [ctypes.POINTER(hilo_shape), _P, _P, _P, _P, _P, _P, _P, _P, _P, _P,
                               ctypes.c_size_t, _P],
    "hilo_attention_fp8_normed": [ctypes.POINTER(hilo_shape), _P, _P, ctypes.POINTER(hilo_attn_w_fp8), _P,
                                  _P, ctypes.c_size_t, _P],
    "hilo_attention_fp8": [ctypes.POINTER(hilo_shape), _P, _P, ctypes.POINTER(hilo_attn_w_fp8), _P, _P,
                           ctypes.c_size_t, _P],
    "hilo_mlp_fp8": [ctypes.POINTER(hilo_shape), _P, _P, ctypes.POINTER(hilo_mlp_w_fp8), _P, _P,
                     ctypes.c_size_t, _P],
    "hilo_quantize_rows": [ctypes.c_int32, _P, ctypes.c_int64, ctypes.c_int64, _P, _P, _P],
    "hilo_blocks": [ctypes.POINTER(hilo_shape), _P, _P, ctypes.POINTER(hilo_attn_w),
                    ctypes.POINTER(hilo_mlp_w), _P, ctypes.c_int32, _P, ctypes.c_size_t, _P],
    "hilo_decompress": [ctypes.POINTER(hilo_shape), _P, _P, _P, _P, _P, _P, _P],
    "hilo_attention_core": [ctypes.POINTER(hilo_shape), _P, _P, _P, _P, ctypes.c_size_t, _P],
    "hilo_attention_core_noalloc": [ctypes.POINTER(hilo_shape), _P, _P, _P, _P],
    "hilo_attention_core_fp8": [ctypes.POINTER(hilo_shape), _P, _P, _P, _P, ctypes.c_size_t, _P],
    "hilo_workspace_bytes": [ctypes.POINTER(hilo_shape)],
    "hilo_workspace_bytes_fp8": [ctypes.POINTER(hilo_shape)],
    "hilo_max_tokens": [ctypes.POINTER(hilo_shape)],
    "hilo_status_str": [ctypes.c_int32],
    "hilo_abi_version": [],
    "hilo_profile_enable": [ctypes.c_int32],
    "hilo_profile_read": [ctypes.c_int32, ctypes.POINTER(ctypes.c_double),
                          ctypes.POINTER(ctypes.c_int64)],
    "hilo_profile_kinds": [],
    "hilo_profile_name": [ctypes.c_int32],
}
_RES = {"hilo_workspace_bytes": ctypes.c_size_t, "hilo_workspace_bytes_fp8": ctypes.c_size_t, "hilo_max_tokens": ctypes.c_int64,
        "hilo_status_str": ctypes.c_char_p, "hilo_profile_name": ctypes.c_char_p}


def lib() -> ctypes.CDLL:
    """Load libhilo.so (built in-tree by paper_2606_13898_amd.build); raise if it is missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2606_13898_amd.build`"
                              " (there is no fallback path)")
        L = ctypes.CDLL(LIB_PATH)
        for name, args in _SIG.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = _RES.get(name, ctypes.c_int32)
        _lib = L
    return _lib


def make_shape(s) -> hilo_shape:
    """hilo_shape from anything with the BlockShape attributes (dtype 'f32'/'bf16' or 0/1)."""
    dt = s.dtype if isinstance(s.dtype, int) else DTYPES[s.dtype]
    return hilo_shape(s.batch, s.images, s.grid_h, s.grid_w, s.text_len, s.dim, s.heads,
                      s.head_dim, s.mlp_dim, dt)


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("libhilo takes device tensors only")
    if not t.is_contiguous():
        raise ValueError("libhilo takes contiguous tensors only")
    return t.data_ptr()


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _check(fn: str, st: int):
    if st != 0:
        raise HiloError(fn, st)


def status_str(st: int) -> str:
    return lib().hilo_status_str(int(st)).decode()


def hilo_abi_version() -> int:
    return lib().hilo_abi_version()


def hilo_max_tokens(shape: hilo_shape) -> int:
    return lib().hilo_max_tokens(ctypes.byref(shape))


def hilo_workspace_bytes_fp8(shape: hilo_shape) -> int:
    return int(lib().hilo_workspace_bytes_fp8(ctypes.byref(shape)))


def hilo_workspace_bytes(shape: hilo_shape) -> int:
    return lib().hilo_workspace_bytes(ctypes.byref(shape))


def hilo_score(shape, x_img, energy, stream=None):
    _check("hilo_score", lib().hilo_score(ctypes.byref(shape), _ptr(x_img), _ptr(energy),
                                          _stream(stream)))


def hilo_score_pixels(shape, rgb, energy, stream=None):
    _check("hilo_score_pixels", lib().hilo_score_pixels(ctypes.byref(shape), _ptr(rgb), _ptr(energy),
                                                        _stream(stream)))


def hilo_select(shape, energy, force, dilate_r: int, mode: int, tau: Optional[Sequence[float]],
                keep: Optional[Sequence[int]], idx_map, fine_idx, pool_idx, counts, cu_seqlens,
                seg_off, stream=None):
    G = shape.batch * shape.images
    tau_arr = (ctypes.c_double * G)(*[float(t) for t in tau]) if tau is not None else None
    keep_arr = (ctypes.c_int32 * G)(*[int(k) for k in keep]) if keep is not None else None
    _check("hilo_select", lib().hilo_select(
        ctypes.byref(shape), _ptr(energy), _ptr(force), int(dilate_r), int(mode), tau_arr, keep_arr,
        _ptr(idx_map), _ptr(fine_idx), _ptr(pool_idx), _ptr(counts), _ptr(cu_seqlens),
        _ptr(seg_off), _stream(stream)))


def hilo_select_tokens(shape, energy, force, dilate_r: int, mode: int, tau: Optional[Sequence[float]],
                       keep: Optional[Sequence[int]], token_set: int, idx_map, fine_idx, pool_idx, counts,
                       cu_seqlens, seg_off, stream=None):
    G = shape.batch * shape.images
    tau_arr = (ctypes.c_double * G)(*[float(t) for t in tau]) if tau is not None else None
    keep_arr = (ctypes.c_int32 * G)(*[int(k) for k in keep]) if keep is not None else None
    _check("hilo_select_tokens", lib().hilo_select_tokens(
        ctypes.byref(shape), _ptr(energy), _ptr(force), int(dilate_r), int(mode), tau_arr, keep_arr,
        int(token_set), _ptr(idx_map), _ptr(fine_idx), _ptr(pool_idx), _ptr(counts), _ptr(cu_seqlens),
        _ptr(seg_off), _stream(stream)))


def hilo_decompress_delta(shape, z, x_img, idx_map, counts, cu_seqlens, seg_off, y_img, y_txt, stream=None):
    _check("hilo_decompress_delta", lib().hilo_decompress_delta(
        ctypes.byref(shape), _ptr(z), _ptr(x_img), _ptr(idx_map), _ptr(counts), _ptr(cu_seqlens),
        _ptr(seg_off), _ptr(y_img), _ptr(y_txt), _stream(stream)))


def hilo_compress(shape, x_img, x_txt, fine_idx, pool_idx, counts, cu_seqlens, seg_off, z,
                  stream=None):
    _check("hilo_compress", lib().hilo_compress(
        ctypes.byref(shape), _ptr(x_img), _ptr(x_txt), _ptr(fine_idx), _ptr(pool_idx),
        _ptr(counts), _ptr(cu_seqlens), _ptr(seg_off), _ptr(z), _stream(stream)))


def hilo_compress_norm(shape, x_img, x_txt, fine_idx, pool_idx, counts, cu_seqlens, seg_off, mod, z,
                       workspace, stream=None):
    _check("hilo_compress_norm", lib().hilo_compress_norm(
        ctypes.byref(shape), _ptr(x_img), _ptr(x_txt), _ptr(fine_idx), _ptr(pool_idx),
        _ptr(counts), _ptr(cu_seqlens), _ptr(seg_off), _ptr(mod), _ptr(z), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream)))


def attn_weights(ws: Sequence[dict]):
    arr = (hilo_attn_w * 2)()
    for k in range(2):
        arr[k] = hilo_attn_w(_ptr(ws[k]["w_qkv"]), _ptr(ws[k]["b_qkv"]), _ptr(ws[k]["w_o"]),
                             _ptr(ws[k]["b_o"]))
    return arr


def mlp_weights(ws: Sequence[dict]):
    arr = (hilo_mlp_w * 2)()
    for k in range(2):
        arr[k] = hilo_mlp_w(_ptr(ws[k]["w1"]), _ptr(ws[k]["b1"]), _ptr(ws[k]["w2"]),
                            _ptr(ws[k]["b2"]))
    return arr


def hilo_attention(shape, z, cu_seqlens, w, mod, workspace, stream=None):
    _check("hilo_attention", lib().hilo_attention(
        ctypes.byref(shape), _ptr(z), _ptr(cu_seqlens), w, _ptr(mod), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream)))


def hilo_attention_normed(shape, z, cu_seqlens, w, mod, workspace, stream=None):
    _check("hilo_attention_normed", lib().hilo_attention_normed(
        ctypes.byref(shape), _ptr(z), _ptr(cu_seqlens), w, _ptr(mod), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream)))


def hilo_mlp(shape, z, cu_seqlens, w, mod, workspace, stream=None):
    _check("hilo_mlp", lib().hilo_mlp(
        ctypes.byref(shape), _ptr(z), _ptr(cu_seqlens), w, _ptr(mod), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream)))


def hilo_quantize_rows(x, codes, scale, stream=None):
    """Per-row E4M3 codes (uint8 [rows][cols]) and float32 scales [rows] of x (float32 or bf16)."""
    dt = {torch.float32: F32, torch.bfloat16: BF16}.get(x.dtype, -1)
    rows, cols = (x.shape[0], x.shape[1]) if x.dim() == 2 else (-1, -1)
    _check("hilo_quantize_rows", lib().hilo_quantize_rows(
        dt, _ptr(x), rows, cols, _ptr(codes), _ptr(scale), _stream(stream)))


def quantize_fp8_weights(ws: Sequence[dict], stream=None):
    """Per stream, the FP8 codes and scales of the four projection weights (hilo_quantize_rows) next
    to the bf16 biases: the weight dicts hilo_attention_fp8 / hilo_mlp_fp8 take (keys w_qkv, s_qkv,
    b_qkv, w_o, s_o, b_o, w1, s1, b1, w2, s2, b2)."""
    out = []
    for w in ws:
        d = dict(w)
        for name, sname in (("w_qkv", "s_qkv"), ("w_o", "s_o"), ("w1", "s1"), ("w2", "s2")):
            src = w[name]
            codes = torch.empty(src.shape, dtype=torch.uint8, device=src.device)
            scale = torch.empty(src.shape[0], dtype=torch.float32, device=src.device)
            hilo_quantize_rows(src, codes, scale, stream)
            d[name], d[sname] = codes, scale
        out.append(d)
    return out


def attn_weights_fp8(ws: Sequence[dict]):
    arr = (hilo_attn_w_fp8 * 2)()
    for k in range(2):
        arr[k] = hilo_attn_w_fp8(_ptr(ws[k]["w_qkv"]), _ptr(ws[k]["s_qkv"]), _ptr(ws[k]["b_qkv"]),
                                 _ptr(ws[k]["w_o"]), _ptr(ws[k]["s_o"]), _ptr(ws[k]["b_o"]))
    return arr


def mlp_weights_fp8(ws: Sequence[dict]):
    arr = (hilo_mlp_w_fp8 * 2)()
    for k in range(2):
        arr[k] = hilo_mlp_w_fp8(_ptr(ws[k]["w1"]), _ptr(ws[k]["s1"]), _ptr(ws[k]["b1"]),
                                _ptr(ws[k]["w2"]), _ptr(ws[k]["s2"]), _ptr(ws[k]["b2"]))
    return arr


def hilo_attention_fp8(shape, z, cu_seqlens, w, mod, workspace, stream=None):
    _check("hilo_attention_fp8", lib().hilo_attention_fp8(
        ctypes.byref(shape), _ptr(z), _ptr(cu_seqlens), w, _ptr(mod), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream)))


def hilo_compress_norm_fp8(shape, x_img, x_txt, fine_idx, pool_idx, counts, cu_seqlens, seg_off, mod, z,
                           workspace, stream=None):
    _check("hilo_compress_norm_fp8", lib().hilo_compress_norm_fp8(
        ctypes.byref(shape), _ptr(x_img), _ptr(x_txt), _ptr(fine_idx), _ptr(pool_idx),
        _ptr(counts), _ptr(cu_seqlens), _ptr(seg_off), _ptr(mod), _ptr(z), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream)))


def hilo_attention_fp8_normed(shape, z, cu_seqlens, w, mod, workspace, stream=None):
    _check("hilo_attention_fp8_normed", lib().hilo_attention_fp8_normed(
        ctypes.byref(shape), _ptr(z), _ptr(cu_seqlens), w, _ptr(mod), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream)))


def hilo_mlp_fp8(shape, z, cu_seqlens, w, mod, workspace, stream=None):
    _check("hilo_mlp_fp8", lib().hilo_mlp_fp8(
        ctypes.byref(shape), _ptr(z), _ptr(cu_seqlens), w, _ptr(mod), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream)))


def stack_weights(blocks: Sequence[Sequence[dict]]):
    """Host arrays [n_blocks][2] of attention and MLP weight pointers for hilo_blocks."""
    n = len(blocks)
    aw = (hilo_attn_w * (2 * n))()
    mw = (hilo_mlp_w * (2 * n))()
    for l, ws in enumerate(blocks):
        for k in range(2):
            aw[2 * l + k] = hilo_attn_w(_ptr(ws[k]["w_qkv"]), _ptr(ws[k]["b_qkv"]), _ptr(ws[k]["w_o"]),
                                        _ptr(ws[k]["b_o"]))
            mw[2 * l + k] = hilo_mlp_w(_ptr(ws[k]["w1"]), _ptr(ws[k]["b1"]), _ptr(ws[k]["w2"]),
                                       _ptr(ws[k]["b2"]))
    return aw, mw


def hilo_blocks(shape, z, cu_seqlens, aw, mw, mod, n_blocks: int, workspace, stream=None):
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check("hilo_blocks", lib().hilo_blocks(
        ctypes.byref(shape), _ptr(z), _ptr(cu_seqlens), aw, mw, _ptr(mod), n_blocks, _ptr(workspace),
        ws_bytes, _stream(stream)))


def hilo_decompress(shape, z, idx_map, cu_seqlens, seg_off, y_img, y_txt, stream=None):
    _check("hilo_decompress", lib().hilo_decompress(
        ctypes.byref(shape), _ptr(z), _ptr(idx_map), _ptr(cu_seqlens), _ptr(seg_off),
        _ptr(y_img), _ptr(y_txt), _stream(stream)))


def hilo_attention_core(shape, qkv, cu_seqlens, out, workspace=None, stream=None):
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check("hilo_attention_core", lib().hilo_attention_core(
        ctypes.byref(shape), _ptr(qkv), _ptr(cu_seqlens), _ptr(out), _ptr(workspace), ws_bytes,
        _stream(stream)))


def hilo_attention_core_fp8(shape, qkv8, cu_seqlens, out, workspace, stream=None):
    ws_bytes = workspace.numel() * workspace.element_size()
    _check("hilo_attention_core_fp8", lib().hilo_attention_core_fp8(
        ctypes.byref(shape), _ptr(qkv8), _ptr(cu_seqlens), _ptr(out), _ptr(workspace), ws_bytes,
        _stream(stream)))


def hilo_attention_core_noalloc(shape, qkv, cu_seqlens, out, stream=None):
    _check("hilo_attention_core_noalloc", lib().hilo_attention_core_noalloc(
        ctypes.byref(shape), _ptr(qkv), _ptr(cu_seqlens), _ptr(out), _stream(stream)))


def hilo_profile_enable(on: bool):
    _check("hilo_profile_enable", lib().hilo_profile_enable(1 if on else 0))


def hilo_profile_read(kind: int):
    ms = ctypes.c_double()
    n = ctypes.c_int64()
    _check("hilo_profile_read", lib().hilo_profile_read(int(kind), ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value


def hilo_profile_kinds() -> int:
    return lib().hilo_profile_kinds()


def hilo_profile_name(kind: int) -> str:
    return lib().hilo_profile_name(int(kind)).decode()
