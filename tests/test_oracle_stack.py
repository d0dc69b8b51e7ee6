"""The oracle's block stack and request loop (several blocks per sampling step, several steps per
selection), pinned by identities of the method rather than by re-running the same code."""
import numpy as np

from oracle import hilo_oracle as O
from paper_2606_13898_amd import inputs


def _shape():
    return inputs.BlockShape(2, 1, 6, 8, 5, 32, 2, 16, 64, "f32")


def test_zero_gates_make_the_stack_the_identity():
    shp = _shape()
    st = inputs.make_stack("smallx", 3, 1, shape=shp, seed=5)
    mods = st.mods[0].copy()
    mods[:, :, :, 2] = 0.0  # gate1
    mods[:, :, :, 5] = 0.0  # gate2
    res = O.pipeline(st.base.x_img, st.base.x_txt, shp, None, 0, "topk", keep=st.base.keep,
                     with_block=False)
    z = O.stack(res["Z"], res["cu"], shp.text_len, shp.heads, st.weights, mods)
    np.testing.assert_array_equal(z, res["Z"])


def test_one_block_one_step_request_is_the_single_block_pipeline():
    shp = _shape()
    st = inputs.make_stack("smallx", 1, 1, shape=shp, seed=6)
    req = O.request(st.x_steps, st.base.x_txt, shp, None, 0, "topk", st.weights, st.mods, keep=st.base.keep)
    one = O.pipeline(st.base.x_img, st.base.x_txt, shp, None, 0, "topk", keep=st.base.keep,
                     weights=st.weights[0], mod=st.mods[0][0])
    np.testing.assert_array_equal(req["y_img"][0], one["y_img"])
    np.testing.assert_array_equal(req["y_txt"][0], one["y_txt"])


def test_zero_compression_request_equals_the_dense_stack_every_step():
    """All blocks kept fine: every step's compressed sequence is the dense sequence, so the stack
    output equals the stack run on the uncompressed tokens (the 0% identity, for L blocks)."""
    shp = _shape()
    st = inputs.make_stack("smallx", 2, 3, shape=shp, seed=7, keep_frac=1.0)
    req = O.request(st.x_steps, st.base.x_txt, shp, None, 0, "topk", st.weights, st.mods, keep=st.base.keep)
    N = shp.grid_h * shp.grid_w
    for t, x in enumerate(st.x_steps):
        Zd, cud = O.dense_sequence(x, st.base.x_txt, shp.batch, shp.images, shp.text_len)
        zd = Zd
        for l in range(2):
            _, zd = O.block(zd, cud, shp.text_len, shp.heads, st.weights[l], st.mods[t][l])
        for s in range(shp.batch):
            np.testing.assert_array_equal(req["y_img"][t][s], zd[cud[s]:cud[s] + N])


def test_selection_is_computed_once_and_later_steps_compress_their_own_latents():
    shp = _shape()
    st = inputs.make_stack("smallx", 1, 2, shape=shp, seed=8)
    req = O.request(st.x_steps, st.base.x_txt, shp, None, 0, "topk", st.weights, st.mods, keep=st.base.keep)
    sel0 = O.select(O.score(st.x_steps[0], shp.grid_h, shp.grid_w), None, shp.grid_h, shp.grid_w, 0,
                    "topk", keep=st.base.keep)
    np.testing.assert_array_equal(req["fine"], sel0)
    # the fine rows of step 1 are step 1's patches (fine_idx from step 0's selection)
    _, fine_idx, _, counts = O.compact(sel0, shp.grid_h, shp.grid_w)
    for g in range(shp.grids):
        nf = int(counts[g][0])
        rows = req["Z"][1][req["seg"][g]:req["seg"][g] + nf]
        np.testing.assert_array_equal(rows, st.x_steps[1][g][fine_idx[g][:nf]].astype(np.float64))
    assert not np.array_equal(st.x_steps[0], st.x_steps[1])
