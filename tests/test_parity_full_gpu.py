"""GPU parity at the full workload sizes, in the launch configuration the benchmark times.

Selection outputs (energies, index maps, counts, offsets) are compared bit for bit on every patch;
the compressed sequence on every row; the block outputs on a seeded sample of rows (image fine,
image pooled and text rows of every sample), which the oracle computes row by row (each sampled
row still attends to every row of its sample)."""
import numpy as np
import pytest
import torch

from oracle import hilo_oracle as O
from paper_2606_13898_amd import hilo, inputs
from paper_2606_13898_amd.pipeline import DeviceBlock

from parity_util import assert_close, assert_update_close, check_compressed, check_selection, oracle_for, to_np

pytestmark = pytest.mark.gpu


def _sample_rows(counts, cu, seg, images, L, per_seg=6, seed=0):
    rng = np.random.default_rng(seed)
    rows = []
    B = len(cu) - 1
    for s in range(B):
        for i in range(images):
            g = s * images + i
            nf, npool = counts[g]
            if nf:
                rows += list(seg[g] + rng.choice(nf, min(per_seg, nf), replace=False))
            if npool:
                rows += list(seg[g] + nf + rng.choice(npool, min(per_seg, npool), replace=False))
        if L:
            rows += list(cu[s + 1] - L + rng.choice(L, min(per_seg, L), replace=False))
    return np.array(sorted(set(int(r) for r in rows)))


@pytest.mark.parametrize("name,r", [("m1024", 0), ("edit", 0), ("edit", 1), ("h2048", 0), ("ragged", 0)],
                         ids=["m1024", "edit", "edit_r1", "h2048", "ragged"])
def test_full_size_parity_sampled(name, r):
    """(edit, r = 1): the edit mask dilated by one patch before it forces blocks fine."""
    print(f"[parity-full] workload={name} dilate_r={r}", flush=True)
    wl = inputs.make_workload(name)
    s = wl.shape
    db = DeviceBlock(wl)
    db.score()
    db.select(hilo.TOPK, dilate_r=r)
    db.compress()
    torch.cuda.synchronize()
    front = oracle_for(wl, r=r, with_block=False)
    check_selection(db, front)
    T = int(front["cu"][-1])
    check_compressed(to_np(db.z)[:T], front, wl)
    print(f"[parity-full] {name}: selection bit-exact, compressed rows exact, tokens {T}", flush=True)
    rows = _sample_rows(front["counts"], front["cu"], front["seg"], s.images, s.text_len)
    z0_dev = to_np(db.z)[rows].astype(np.float64)
    db.attention()
    torch.cuda.synchronize()
    z1_dev = to_np(db.z)[rows].astype(np.float64)
    db.mlp()
    torch.cuda.synchronize()
    z2_dev = to_np(db.z)[rows].astype(np.float64)
    db.decompress()
    torch.cuda.synchronize()
    z1, z2 = O.block(front["Z"], front["cu"], s.text_len, s.heads, wl.weights, wl.mod, rows)
    assert np.abs(z2).max() < 8.0
    # each half's own update of the sampled rows, the residual stream taken out
    assert_update_close(z1_dev, z1, z0_dev, front["Z"][rows], "bf16", f"{name} attention update")
    assert_update_close(z2_dev, z2, z1_dev, z1, "bf16", f"{name} mlp update")
    # y at every patch whose compressed row was sampled, and text rows
    y = to_np(db.y_img)
    got, want = [], []
    row_pos = {r: k for k, r in enumerate(rows)}
    for g in range(s.grids):
        rr = front["seg"][g] + front["idx_map"][g]
        sel = np.flatnonzero(np.isin(rr, rows))
        got.append(y[g][sel])
        want.append(z2[[row_pos[int(r)] for r in rr[sel]]])
    if s.text_len:
        yt = to_np(db.y_txt)
        for b in range(s.batch):
            lo = int(front["cu"][b + 1]) - s.text_len
            for t in range(s.text_len):
                if lo + t in row_pos:
                    got.append(yt[b][t:t + 1])
                    want.append(z2[row_pos[lo + t]][None])
    got, want = np.concatenate(got), np.concatenate(want)
    ma, rel = assert_close(got, want, "bf16", f"{name} y at sampled rows")
    print(f"[parity-full] {name}: {got.shape[0]} output rows, max_abs {ma:.3g}, rel_l2 {rel:.3g}",
          flush=True)
