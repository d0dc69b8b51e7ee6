"""The allocation-free attention core (hilo_attention_core_noalloc, scratch inside the library)
against hilo_attention_core with a caller workspace, through the C ABI: the same kernels on the
same inputs, so the outputs must agree bit for bit.  Two calls in a row share the scratch, the
second with a smaller input; head dims 128 and 64."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2606_13898_amd import hilo, inputs

pytestmark = pytest.mark.gpu


def _case(lens, heads, hd, seed):
    D = heads * hd
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    T = int(cu[-1])
    rng = np.random.default_rng(seed)
    qkv = torch.from_numpy(inputs.to_bf16_values(rng.standard_normal((T, 3 * D)).astype(np.float32)))
    maxlen = max(lens)
    shp = hilo.hilo_shape(len(lens), 1, 2, 2 * ((maxlen + 3) // 4), 0, D, heads, hd, 4 * D, hilo.BF16)
    return shp, qkv.to(torch.bfloat16).cuda(), torch.from_numpy(cu).cuda(), T, D


@pytest.mark.parametrize("hd,first,second", [
    (128, [700, 1300, 9], [5, 200]),
    (64, [3, 130, 31, 900], [64]),
])
def test_noalloc_core_matches_workspace_core(hd, first, second):
    for k, lens in enumerate((first, second)):
        print(f"[no-alloc] hd={hd} call {k} lens={lens}", flush=True)
        shp, qkv, cu, T, D = _case(lens, 2, hd, 100 * hd + k)
        want = torch.zeros(T, D, dtype=torch.bfloat16, device="cuda")
        got = torch.full((T, D), float("nan"), dtype=torch.bfloat16, device="cuda")
        ws = torch.empty(hilo.hilo_workspace_bytes(shp), dtype=torch.uint8, device="cuda")
        hilo.hilo_attention_core(shp, qkv, cu, want, ws)
        hilo.hilo_attention_core_noalloc(shp, qkv, cu, got)
        torch.cuda.synchronize()
        assert torch.isfinite(want.float()).all()
        assert torch.equal(got, want), f"call {k}: max diff {(got.float() - want.float()).abs().max().item()}"


def test_noalloc_core_validates_before_enqueueing():
    L = hilo.lib()
    FAKE = ctypes.c_void_p(256)
    shp = hilo.hilo_shape(1, 1, 2, 8, 0, 256, 2, 128, 1024, hilo.BF16)
    assert L.hilo_attention_core_noalloc(ctypes.byref(shp), None, FAKE, FAKE, None) == 1
    bad = hilo.hilo_shape(1, 1, 2, 8, 0, 256, 2, 96, 1024, hilo.BF16)  # 2 * 96 != 256
    assert L.hilo_attention_core_noalloc(ctypes.byref(bad), FAKE, FAKE, FAKE, None) == 2
