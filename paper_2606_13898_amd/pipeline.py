"""Device buffers for one compressed-block problem and the six library calls in order.

torch is used here for device memory and streams only; every step is a libhilo kernel.
"""
from __future__ import annotations

from typing import Optional, Sequence

import numpy as np
import torch

from . import hilo
from .inputs import StackWorkload, Workload


def _dev(a: np.ndarray, dtype: torch.dtype, device) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a)).to(dtype).to(device)


class DeviceBlock:
    """All inputs, outputs and scratch of one workload, resident on `device`."""

    def __init__(self, wl: Workload, device: str = "cuda", with_block: bool = True):
        s = wl.shape
        self.wl = wl
        self.shape = hilo.make_shape(s)
        self.dtype = hilo.TORCH_DTYPES[self.shape.dtype]
        G, N, NB, B, D, L = s.grids, s.n_patches, s.n_blocks, s.batch, s.dim, s.text_len
        self.T = hilo.hilo_max_tokens(self.shape)
        if self.T < 0:
            raise ValueError(f"invalid shape {s}")
        self.x_img = _dev(wl.x_img, self.dtype, device)
        self.x_txt = _dev(wl.x_txt, self.dtype, device)
        self.force = _dev(wl.force, torch.uint8, device) if wl.force is not None else None
        i32, i64 = torch.int32, torch.int64
        self.energy = torch.empty(G, N, dtype=i64, device=device)
        self.idx_map = torch.empty(G, N, dtype=i32, device=device)
        self.fine_idx = torch.empty(G, N, dtype=i32, device=device)
        self.pool_idx = torch.empty(G, NB, dtype=i32, device=device)
        self.counts = torch.empty(G, 2, dtype=i32, device=device)
        self.cu = torch.empty(B + 1, dtype=i32, device=device)
        self.seg = torch.empty(G, dtype=i32, device=device)
        self.z = torch.empty(self.T, D, dtype=torch.float32, device=device)
        self.y_img = torch.empty(G, N, D, dtype=self.dtype, device=device)
        self.y_txt = torch.empty(B, L, D, dtype=self.dtype, device=device) if L > 0 else None
        self.with_block = with_block
        if with_block:
            self.weights = [{k: _dev(v, self.dtype, device) for k, v in w.items()} for w in wl.weights]
            self.mod = _dev(wl.mod, torch.float32, device)
            # sized for the FP8 block too when the shape allows it (it needs the hidden rows' codes)
            nbytes = max(hilo.hilo_workspace_bytes(self.shape), hilo.hilo_workspace_bytes_fp8(self.shape))
            self.ws = torch.empty(nbytes, dtype=torch.uint8, device=device)
            self.aw = hilo.attn_weights(self.weights)
            self.mw = hilo.mlp_weights(self.weights)

    def attach_block(self, weights, mod: torch.Tensor):
        """Run the block with the given device weights (two stream dicts) and modulation
        [B][2][6][D] instead of the workload's own (benchmarks reuse one weight set across shapes)."""
        self.weights = weights
        self.mod = mod
        nbytes = max(hilo.hilo_workspace_bytes(self.shape), hilo.hilo_workspace_bytes_fp8(self.shape))
        self.ws = torch.empty(nbytes, dtype=torch.uint8, device=mod.device)
        self.aw = hilo.attn_weights(weights)
        self.mw = hilo.mlp_weights(weights)
        self.with_block = True

    # -- the six steps ---------------------------------------------------------------------
    def score(self, stream=None):
        hilo.hilo_score(self.shape, self.x_img, self.energy, stream)

    def select(self, mode: int = hilo.TOPK, keep: Optional[Sequence[int]] = None,
               tau: Optional[Sequence[float]] = None, dilate_r: Optional[int] = None, stream=None,
               tokens: int = hilo.PARTITION):
        keep = self.wl.keep if (keep is None and mode == hilo.TOPK) else keep
        r = self.wl.dilate_r if dilate_r is None else dilate_r
        if tokens == hilo.PARTITION:
            hilo.hilo_select(self.shape, self.energy, self.force, r, mode, tau, keep, self.idx_map,
                             self.fine_idx, self.pool_idx, self.counts, self.cu, self.seg, stream)
        else:
            hilo.hilo_select_tokens(self.shape, self.energy, self.force, r, mode, tau, keep, tokens,
                                    self.idx_map, self.fine_idx, self.pool_idx, self.counts, self.cu,
                                    self.seg, stream)

    def compress(self, stream=None, norm: bool = False, fp8: bool = False):
        """S3; with norm (a block attached) also the attention half's first row norm, whose rows
        land in the workspace for attention(normed=True) (fp8: in the FP8 block's form)."""
        if norm and fp8:
            hilo.hilo_compress_norm_fp8(self.shape, self.x_img, self.x_txt, self.fine_idx, self.pool_idx,
                                        self.counts, self.cu, self.seg, self.mod, self.z, self.ws, stream)
        elif norm:
            hilo.hilo_compress_norm(self.shape, self.x_img, self.x_txt, self.fine_idx, self.pool_idx,
                                    self.counts, self.cu, self.seg, self.mod, self.z, self.ws, stream)
        else:
            hilo.hilo_compress(self.shape, self.x_img, self.x_txt, self.fine_idx, self.pool_idx,
                               self.counts, self.cu, self.seg, self.z, stream)

    def prepare_fp8(self, stream=None):
        """FP8 codes and per-output-channel scales of the four projection weights (once; weights
        are static)."""
        if getattr(self, "weights8", None) is None:
            self.weights8 = hilo.quantize_fp8_weights(self.weights, stream)
            self.aw8 = hilo.attn_weights_fp8(self.weights8)
            self.mw8 = hilo.mlp_weights_fp8(self.weights8)

    def attention(self, stream=None, fp8: bool = False, normed: bool = False):
        if fp8:
            self.prepare_fp8(stream)
            if normed:
                hilo.hilo_attention_fp8_normed(self.shape, self.z, self.cu, self.aw8, self.mod, self.ws, stream)
            else:
                hilo.hilo_attention_fp8(self.shape, self.z, self.cu, self.aw8, self.mod, self.ws, stream)
        elif normed:
            hilo.hilo_attention_normed(self.shape, self.z, self.cu, self.aw, self.mod, self.ws, stream)
        else:
            hilo.hilo_attention(self.shape, self.z, self.cu, self.aw, self.mod, self.ws, stream)

    def mlp(self, stream=None, fp8: bool = False):
        if fp8:
            self.prepare_fp8(stream)
            hilo.hilo_mlp_fp8(self.shape, self.z, self.cu, self.mw8, self.mod, self.ws, stream)
        else:
            hilo.hilo_mlp(self.shape, self.z, self.cu, self.mw, self.mod, self.ws, stream)

    def decompress(self, stream=None, delta: bool = False):
        if delta:
            hilo.hilo_decompress_delta(self.shape, self.z, self.x_img, self.idx_map, self.counts, self.cu,
                                       self.seg, self.y_img, self.y_txt, stream)
        else:
            hilo.hilo_decompress(self.shape, self.z, self.idx_map, self.cu, self.seg, self.y_img,
                                 self.y_txt, stream)

    def run(self, mode: int = hilo.TOPK, keep=None, tau=None, dilate_r=None, stream=None,
            tokens: int = hilo.PARTITION, delta: bool = False, fp8: bool = False, fused: bool = True):
        """One pass of the whole hot path: score, select, compress, attention, MLP, decompress
        (fp8: all four projections on FP8 operands; fused: the attention half's first row norm in
        the compress pass, hilo_compress_norm + hilo_attention_normed, or their FP8 counterparts)."""
        self.score(stream)
        self.select(mode, keep, tau, dilate_r, stream, tokens)
        norm = fused and self.with_block
        if norm and fp8:
            self.prepare_fp8(stream)
        self.compress(stream, norm, fp8)
        if self.with_block:
            self.attention(stream, fp8, norm)
            self.mlp(stream, fp8)
        self.decompress(stream, delta)


class DeviceStack:
    """One request of the paper's regime on the device: the selection once (from step 0's
    latents), then per sampling step compress -> n_blocks blocks (hilo_blocks) -> decompress."""

    def __init__(self, st: StackWorkload, device: str = "cuda"):
        self.st = st
        self.db = DeviceBlock(st.base, device, with_block=False)
        db = self.db
        self.x_steps = [_dev(x, db.dtype, device) for x in st.x_steps]
        self.weights = [[{k: _dev(v, db.dtype, device) for k, v in w.items()} for w in ws] for ws in st.weights]
        self.aw, self.mw = hilo.stack_weights(self.weights)
        self.mods = _dev(st.mods, torch.float32, device)  # [steps][n_blocks][B][2][6][D]
        self.n_blocks = len(st.weights)
        self.ws = torch.empty(hilo.hilo_workspace_bytes(db.shape), dtype=torch.uint8, device=device)
        self.y_img = [torch.empty_like(db.y_img) for _ in st.x_steps]
        self.y_txt = [torch.empty_like(db.y_txt) if db.y_txt is not None else None for _ in st.x_steps]

    def select(self, mode: int = hilo.TOPK, stream=None):
        db = self.db
        db.x_img = self.x_steps[0]
        db.score(stream)
        db.select(mode, stream=stream)

    def step(self, t: int, stream=None):
        db = self.db
        hilo.hilo_compress(db.shape, self.x_steps[t], db.x_txt, db.fine_idx, db.pool_idx, db.counts,
                           db.cu, db.seg, db.z, stream)
        hilo.hilo_blocks(db.shape, db.z, db.cu, self.aw, self.mw, self.mods[t], self.n_blocks, self.ws,
                         stream)
        hilo.hilo_decompress(db.shape, db.z, db.idx_map, db.cu, db.seg, self.y_img[t], self.y_txt[t],
                             stream)

    def run(self, mode: int = hilo.TOPK, stream=None):
        self.select(mode, stream)
        for t in range(len(self.x_steps)):
            self.step(t, stream)
