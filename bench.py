#!/usr/bin/env python3
"""Benchmark of the HiLo-Token compressed DiT block on one MI355X.

One step = one pass of the whole hot path over one batch: score, select, compress, attention,
MLP, decompress (six C-ABI calls, all kernels on the GPU), inputs resident in HBM.  Consecutive
steps read different copies of the step's inputs (latents and text tokens, more than 512 MB in
all) and alternate between two copies of the block's weights, so no step finds its operands in the
256 MB last-level cache (MALL) from an earlier step.  Prints ONE JSON line with the step latency,
throughput, the dense (uncompressed) block for the speedup, per-kernel times from HIP events with
their roofline fractions, the other workloads and a kept-fraction sweep, and the CPU oracle timed
on a bounded sample.

    python bench.py [--steps K] [--warmup W] [--workload m1024] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "compressed DiT-block latency (ms) + attn TFLOP/s at 64×64 grid; speedup vs dense"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_FP8_TFLOPS = 5000.0    # MI355X dense fp8 MFMA
PEAK_F32_TFLOPS = 157.3     # MI355X fp32 vector
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
# vector-ALU issue peak: 256 CUs x 4 SIMDs, one wave64 instruction per SIMD every 4 cycles (16 lanes
# per cycle: fp32 157.3 TFLOP/s counts the packed two-wide FMA), 2.4 GHz
PEAK_VALU_INSTS_PER_S = 256 * 4 * 2.4e9 / 4

DESCR = {
    "m1024": "one MMDiT-style DiT block at 1024px: 64x64 latent grid + 512 text tokens, D=3072, "
             "24 heads x 128, MLP 12288, bf16; 3-5 texture regions (~35% area); top-k keeps 40% of "
             "2x2 blocks fine",
    "h2048": "one DiT block at 2048px: 128x128 grid + 512 text tokens, D=3072, 24x128 heads, bf16; "
             "multi-octave texture on ~20% area; top-k keeps 25% fine",
    "edit": "edit with reference: two 64x64 grids + 512 text tokens, D=3072, bf16; 15% edit mask "
            "forced fine; top-k keeps 35% per grid",
    "ragged": "batch of 8 samples of 64x64 + 512 text tokens, D=3072, bf16; kept fraction per "
              "sample U[5%,95%]",
}


def kernel_work(shape, counts, cu):
    """Algorithmic work per launch of every kernel kind: (amount, unit, peak)."""
    import numpy as np

    s = shape
    es = 2 if s.dtype == "bf16" else 4
    G, N, D, F, B, L = s.grids, s.n_patches, s.dim, s.mlp_dim, s.batch, s.text_len
    nc = int(cu[-1])
    n_img = int(counts.sum())
    seqs = np.diff(cu).astype(np.int64)
    mfma = PEAK_BF16_TFLOPS if s.dtype == "bf16" else PEAK_F32_TFLOPS
    gemm = lambda n_out, k: (2.0 * nc * n_out * k / 1e12, "TFLOP", mfma)
    return {
        "score": ((G * N * D * es + 8 * G * N) / 1e9, "GB", PEAK_HBM_GBS),
        # the step's compress pass also writes the attention half's normalised rows (hilo_compress_norm)
        "compress": ((G * N * D * es + n_img * D * 4 + B * L * D * (es + 4) + nc * D * es) / 1e9, "GB",
                     PEAK_HBM_GBS),
        "rownorm_attn": (nc * D * (4 + es) / 1e9, "GB", PEAK_HBM_GBS),
        "gemm_qkv": gemm(3 * D, D),
        "attention_core": (4.0 * float((seqs ** 2).sum()) * D / 1e12, "TFLOP", mfma),
        "gemm_o": gemm(D, D),
        "rownorm_mlp": (nc * D * (4 + es) / 1e9, "GB", PEAK_HBM_GBS),
        "gemm_fc1": gemm(F, D),
        "gemm_fc2": gemm(D, F),
        "decompress": ((n_img * D * 4 + G * N * D * es + B * L * D * (4 + es)) / 1e9, "GB", PEAK_HBM_GBS),
    }


def source_digest(paths):
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def traffic_for(kind):
    """HBM bytes per launch measured with rocprofv3 counters (profiles/traffic.json), or None when
    the counters are missing or the kernel source changed since they were taken."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        tab = json.load(f)
    ent = tab.get("kernels", {}).get(kind)
    if not ent:
        return None
    if source_digest(ent["sources"]) != ent["source_digest"]:
        return None
    return ent["bytes_per_launch"]


def valu_for(kind):
    """Vector-ALU wave instructions per launch measured with rocprofv3 (SQ_INSTS_VALU, the counter
    pass of profiles/traffic.json), or None when missing or the kernel source changed since."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        ent = json.load(f).get("kernels", {}).get(kind)
    if not ent or "valu_insts_per_launch" not in ent or source_digest(ent["sources"]) != ent["source_digest"]:
        return None
    return ent["valu_insts_per_launch"]


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(wl):
    """The oracle, untuned, on one full step of the same workload (bounded: ~10-30 s), its BLAS
    threads set to the cores this process may run on."""
    import threadpoolctl

    from oracle import hilo_oracle as O

    cores = len(os.sched_getaffinity(0))
    with threadpoolctl.threadpool_limits(limits=cores, user_api="blas"):
        info = threadpoolctl.threadpool_info()
        threads = max([i.get("num_threads", 1) for i in info if i.get("user_api") == "blas"] or [1])
        t0 = time.perf_counter()
        O.pipeline(wl.x_img, wl.x_txt, wl.shape, wl.force, wl.dilate_r, "topk", keep=wl.keep,
                   weights=wl.weights, mod=wl.mod)
        dt = time.perf_counter() - t0
    return {"value": round(dt * 1e3, 1), "unit": "ms", "cores": int(threads), "kind": "oracle",
            "sample": f"one full step (score..decompress) of the {wl.name} workload in float64 "
                      f"numpy (matrix products on BLAS with {threads} threads, "
                      f"{cores} cores in this process's affinity)",
            "cpu_model": cpu_model(), "affinity_cores": cores}


class Rotation:
    """Copies of a step's inputs for MALL-proof timing: R copies of (x_img, x_txt) totalling more
    than `min_bytes`, and two copies of the block weights; step k reads input copy k % R and weight
    copy k % 2."""

    def __init__(self, db, min_bytes=512 << 20, weight_sets=None):
        import math

        per = db.x_img.numel() * db.x_img.element_size()
        if db.x_txt is not None:
            per += db.x_txt.numel() * db.x_txt.element_size()
        self.R = max(3, math.ceil(min_bytes / per))
        self.xs = [(db.x_img, db.x_txt)] + [
            (db.x_img.clone(), db.x_txt.clone() if db.x_txt is not None else None) for _ in range(self.R - 1)]
        self.bytes = per * self.R
        self.ws = weight_sets if weight_sets is not None else ([(db.aw, db.mw)] if db.with_block else [])

    @staticmethod
    def weight_sets(db):
        from paper_2606_13898_amd import hilo

        w2 = [{k: v.clone() for k, v in w.items()} for w in db.weights]
        return [(db.aw, db.mw), (hilo.attn_weights(w2), hilo.mlp_weights(w2))], w2

    def use(self, db, k):
        db.x_img, db.x_txt = self.xs[k % self.R]
        if self.ws:
            db.aw, db.mw = self.ws[k % len(self.ws)]


def timed(stream, steps, fn):
    """Runs fn(k) for k < steps with an event between consecutive calls: (mean ms, sorted ms)."""
    import numpy as np
    import torch

    evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    evs[0].record(stream)
    for k in range(steps):
        fn(k)
        evs[k + 1].record(stream)
    torch.cuda.synchronize()
    return evs[0].elapsed_time(evs[-1]) / steps, np.sort([evs[k].elapsed_time(evs[k + 1]) for k in range(steps)])


def kernel_profile(steps, fn, work):
    """The same calls again with the library's event pairs around every kernel: per kernel kind the
    mean duration and, where the algorithmic work is known, the achieved rate and roofline fraction."""
    import torch

    from paper_2606_13898_amd import hilo

    hilo.hilo_profile_enable(True)
    for k in range(steps):
        fn(k)
    torch.cuda.synchronize()
    kinds = {hilo.hilo_profile_name(k): hilo.hilo_profile_read(k) for k in range(hilo.hilo_profile_kinds())}
    hilo.hilo_profile_enable(False)
    kern = {}
    for name, (tot, n) in kinds.items():
        if n == 0:
            continue
        avg = tot / n
        ent = {"ms": round(avg, 4), "launches_per_step": n // steps}
        if name in work:
            amt, unit, peak = work[name]
            ach = amt / (avg * 1e-3)  # GB/s or TFLOP/s
            ent.update(achieved=round(ach, 1), unit=unit + "/s", peak=peak,
                       frac=round(ach / peak, 4), work_per_launch=f"{amt:.4g} {unit}")
        kern[name] = ent
    return kern


BLOCK_KERNELS = ("rownorm_attn", "gemm_qkv", "attention_core", "gemm_o", "rownorm_mlp", "gemm_fc1", "gemm_fc2")


def block_flops(shape, seqlens):
    """Algorithmic FLOPs of the block on packed samples of the given lengths: the four projections
    (2 n D (3D + D + F + F)) and the attention core (4 n^2 D per sample)."""
    import numpy as np

    n = np.asarray(seqlens, dtype=np.float64)
    D, F = shape.dim, shape.mlp_dim
    return float(2.0 * n.sum() * D * (4 * D + 2 * F) + 4.0 * (n ** 2).sum() * D)


def dense_block_ms(db, rot, steps, warmup, stream, dilate_r=None):
    """The block (attention + MLP) on the uncompressed sequence: every block kept fine (the dense
    token order), timed per step around the two calls.  As in the compressed step, the attention
    half's first row norm runs in the compress pass before it (hilo_compress_norm), outside the
    block's time in both."""
    import torch

    from paper_2606_13898_amd import hilo

    s = db.wl.shape
    db.score()
    db.select(hilo.TOPK, keep=[s.n_blocks] * s.grids, dilate_r=dilate_r)
    for k in range(warmup):
        rot.use(db, k)
        db.compress(norm=True)
        db.attention(normed=True)
        db.mlp()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for k, (a, b) in enumerate(ev):
        rot.use(db, k)
        db.compress(norm=True)
        a.record(stream)
        db.attention(normed=True)
        db.mlp()
        b.record(stream)
    torch.cuda.synchronize()
    n = int(db.cu.cpu().numpy()[-1])
    return sum(a.elapsed_time(b) for a, b in ev) / steps, n, db.cu.cpu().numpy()


def config_leg(name, base, rot_w, steps, warmup, stream, dilate_r=0):
    """Another workload at full size (its own seeded latents, grids, masks and keep rule; the m1024
    block weights, since their values do not change the timing): step and block latency, the dense
    block, tokens and FLOPs, and the per-kernel roofline fractions."""
    import numpy as np
    import torch

    from paper_2606_13898_amd import hilo, inputs
    from paper_2606_13898_amd.pipeline import DeviceBlock

    wl = inputs.make_workload(name, with_block=False)
    s = wl.shape
    db = DeviceBlock(wl, with_block=False)
    g = torch.Generator(device="cuda")
    g.manual_seed(77)
    mod = torch.randn(s.batch, 2, 6, s.dim, generator=g, device="cuda") * 0.1
    db.attach_block(base.weights, mod)
    rot = Rotation(db, weight_sets=rot_w)

    def step(k):
        rot.use(db, k)
        db.run(hilo.TOPK, dilate_r=dilate_r)

    for k in range(warmup):
        step(k)
    ms, per = timed(stream, steps, step)
    cu = db.cu.cpu().numpy()
    counts = db.counts.cpu().numpy()
    kern = kernel_profile(steps, step, kernel_work(s, counts, cu))
    t_blk = sum(kern[k]["ms"] for k in BLOCK_KERNELS if k in kern)
    # the Sobel score is bound by the vector ALU (its exact fixed-point energy), not by HBM: its
    # instruction count at the issue peak is the floor it is measured against as well
    nv = valu_for("score")
    if "score" in kern and nv:
        floor = nv / PEAK_VALU_INSTS_PER_S * 1e3
        kern["score"]["alu"] = {"bound": "alu", "valu_insts_per_launch": nv,
                                "peak": "%.4g wave64 instructions/s" % PEAK_VALU_INSTS_PER_S,
                                "floor_ms": round(floor, 4), "frac": round(floor / kern["score"]["ms"], 4)}
    dense_ms, nd, cud = dense_block_ms(db, rot, steps, warmup, stream, dilate_r)
    nc = int(cu[-1])
    f_c, f_d = block_flops(s, np.diff(cu)), block_flops(s, np.diff(cud))
    out = {"workload": f"{name}: {DESCR[name]}" + (f"; mask dilated by r = {dilate_r}" if dilate_r else ""),
           "ms_per_step": round(ms, 4), "ms_per_step_median": round(float(per[len(per) // 2]), 4),
           "block_ms": round(t_blk, 4), "dense_block_ms": round(dense_ms, 4),
           "compressed_tokens": nc, "dense_tokens": nd, "token_ratio": round(nd / nc, 3),
           "flop_ratio": round(f_d / f_c, 3),
           "speedup_vs_dense": round(dense_ms / ms, 3), "block_speedup_vs_dense": round(dense_ms / t_blk, 3),
           "compressed_tokens_per_s": round(nc / (ms * 1e-3), 1),
           "kernels": {k: {kk: v[kk] for kk in ("ms", "achieved", "unit", "frac") if kk in v} for k, v in kern.items()}}
    del db, rot
    torch.cuda.empty_cache()
    return out


def sweep_leg(db, rot, steps, warmup, stream, keeps):
    """The kept-fraction sweep on one 64x64 sample (Sec. 3.3 reports the speedup as a function of the
    mask ratio): for each number of kept blocks the whole step, the block alone, tokens and FLOPs,
    against the dense block (every block kept)."""
    import numpy as np
    import torch

    from paper_2606_13898_amd import hilo

    s = db.wl.shape
    rows = []
    for keep in keeps:
        kk = [keep] * s.grids

        def step(k):
            rot.use(db, k)
            db.run(hilo.TOPK, keep=kk)

        for k in range(warmup):
            step(k)
        ms, _ = timed(stream, steps, step)
        blk = []
        for k in range(steps):
            rot.use(db, k)
            db.score()
            db.select(hilo.TOPK, keep=kk)
            db.compress(norm=True)
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            db.attention(normed=True)
            db.mlp()
            b.record(stream)
            blk.append((a, b))
        torch.cuda.synchronize()
        blk_ms = sum(a.elapsed_time(b) for a, b in blk) / steps
        cu = db.cu.cpu().numpy()
        rows.append({"kept_fraction": round(keep / s.n_blocks, 3), "kept_blocks": keep,
                     "tokens": int(cu[-1]), "ms_per_step": round(ms, 4), "block_ms": round(blk_ms, 4),
                     "flops": block_flops(s, np.diff(cu))})
    dense = rows[-1] if keeps[-1] == s.n_blocks else None
    for r in rows:
        if dense:
            r["token_ratio"] = round(dense["tokens"] / r["tokens"], 3)
            r["flop_ratio"] = round(dense["flops"] / r["flops"], 3)
            r["block_speedup_vs_dense"] = round(dense["block_ms"] / r["block_ms"], 3)
            r["step_speedup_vs_dense_block"] = round(dense["block_ms"] / r["ms_per_step"], 3)
        r["flops"] = f"{r['flops']:.4g}"
    db.run(hilo.TOPK)  # leave the buffers as the default step left them
    torch.cuda.synchronize()
    return rows


def pixel_leg(db, steps, warmup, stream):
    """The paper's own selector input: Sobel on the RGB image at 16x the token grid (1024 x 1024
    pixels for the 64 x 64 grid), summed per token (hilo_score_pixels), then the threshold.  The
    paper cuts its normalised Sobel magnitude map at 0.1; the energy is the magnitude squared, so
    its counterpart is 0.01 on the normalised energy map.  The image is synthetic
    (inputs.pixel_image).  HBM-bound: one read of the image plus the 8-byte energies."""
    import numpy as np
    import torch

    from paper_2606_13898_amd import hilo, inputs

    s = db.wl.shape
    G, N = s.grids, s.n_patches
    rgb = torch.from_numpy(inputs.pixel_image(s, 5)).cuda()
    E = torch.empty(G, N, dtype=torch.int64, device="cuda")
    for _ in range(warmup):
        hilo.hilo_score_pixels(db.shape, rgb, E)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(steps):
        hilo.hilo_score_pixels(db.shape, rgb, E)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    nbytes = rgb.numel() * 4 + E.numel() * 8
    gbs = nbytes / (ms * 1e-3) / 1e9
    db.energy.copy_(E)
    db.select(hilo.THRESHOLD, tau=[0.01] * G)
    counts = db.counts.cpu().numpy()
    res = {"ms": round(ms, 4), "image": f"{G}x3x{16 * s.grid_h}x{16 * s.grid_w} float32",
           "achieved": round(gbs, 1), "unit": "GB/s", "peak": 8000.0, "frac": round(gbs / 8000.0, 4),
           "work_per_launch": f"{nbytes / 1e9:.4g} GB",
           "kept_fine_fraction_energy_tau_0.01": round(float(counts[:, 0].sum()) / (G * N), 4)}
    db.run(hilo.TOPK)  # leave the buffers as the default step left them
    torch.cuda.synchronize()
    return res


def token_set_leg(db, rot, steps, warmup, stream, dense_ms):
    """The whole step with the other token sets (same selection rule): overlap -- every block's
    pooled token kept next to the fine patches, the paper's own token set (Sec. 2.3) -- and drop --
    the fine patches alone (Sec. 3.2) -- both reassembled in the delta form; partition with the
    delta form for comparison."""
    import torch

    from paper_2606_13898_amd import hilo

    res = {}
    for name, tokens in (("overlap", hilo.OVERLAP), ("drop", hilo.DROP), ("partition", hilo.PARTITION)):
        def step(k):
            rot.use(db, k)
            db.run(hilo.TOPK, tokens=tokens, delta=True)

        for k in range(warmup):
            step(k)
        ms, _ = timed(stream, steps, step)
        nc = int(db.cu.cpu().numpy()[-1])
        ent = {"ms_per_step": round(ms, 4), "compressed_tokens": nc, "decompress": "delta"}
        if dense_ms:
            ent["speedup_vs_dense"] = round(dense_ms / ms, 3)
        res[name] = ent
    db.run(hilo.TOPK)  # leave the buffers as the default step left them
    torch.cuda.synchronize()
    return res


def fp8_leg(db, rot, steps, warmup, stream, work, bf16_ms):
    """The step with all four projections and the attention's score product in FP8 (per-row E4M3
    operands: one scale per token for the activations, one per output channel for the weights, one
    power-of-two scale per (token, head) for q and k; Sec. 3.3 combines the compression with FP8
    quantisation): step latency, the projections' rates against the fp8 MFMA peak, the attention
    core (FP8 scores, bf16 P V), the two passes that quantise the attention and GELU outputs, and how
    far the block's update of the compressed tokens moves from the bf16 step's (relative L2 over
    all rows)."""
    import numpy as np
    import torch

    from paper_2606_13898_amd import hilo

    db.prepare_fp8()
    db.score()
    db.select(hilo.TOPK)
    db.compress()
    z0 = db.z.clone()
    db.attention()
    db.mlp()
    z16 = db.z.clone()
    db.compress()
    db.attention(fp8=True)
    db.mlp(fp8=True)
    torch.cuda.synchronize()
    nc = int(db.cu.cpu().numpy()[-1])
    upd16 = (z16 - z0)[:nc].double()
    upd8 = (db.z - z0)[:nc].double()
    rel = float(torch.linalg.norm(upd8 - upd16) / torch.linalg.norm(upd16))

    def step(k):
        db.x_img, db.x_txt = rot.xs[k % rot.R]
        db.run(hilo.TOPK, fp8=True)

    for k in range(warmup):
        step(k)
    ms, per_step = timed(stream, steps, step)

    hilo.hilo_profile_enable(True)
    for k in range(steps):
        step(k)
    torch.cuda.synchronize()
    kern = {}
    for k in range(hilo.hilo_profile_kinds()):
        name = hilo.hilo_profile_name(k)
        tot, n = hilo.hilo_profile_read(k)
        if n and name in ("rownorm_attn", "gemm_qkv", "attention_core", "quantize_attn", "gemm_o", "rownorm_mlp",
                          "gemm_fc1", "quantize_mlp", "gemm_fc2"):
            avg = tot / n
            ent = {"ms": round(avg, 4)}
            if name.startswith("gemm"):
                ach = work[name][0] / (avg * 1e-3)
                ent.update(achieved=round(ach, 1), unit="TFLOP/s", peak=PEAK_FP8_TFLOPS,
                           frac=round(ach / PEAK_FP8_TFLOPS, 4))
            elif name == "attention_core":  # half its FLOPs on the fp8 rate (scores), half on bf16 (P V)
                ach = work[name][0] / (avg * 1e-3)
                ent.update(achieved=round(ach, 1), unit="TFLOP/s", note="scores FP8, P V bf16")
            kern[name] = ent
    hilo.hilo_profile_enable(False)
    db.run(hilo.TOPK)  # leave the buffers as the default step left them
    torch.cuda.synchronize()
    res = {"ms_per_step": round(ms, 4), "ms_per_step_median": round(float(per_step[len(per_step) // 2]), 4),
           "projections_in_fp8": ["qkv", "attention_output", "mlp_up", "mlp_down"],
           "attention_in_fp8": "scores q k^T (E4M3 q and k, power-of-two scale per token and head); P V bf16",
           "kernels": kern,
           "timing": "latents rotated as in the main step; one FP8 weight set (quantised once)",
           "block_update_rel_l2_vs_bf16": round(rel, 5)}
    if bf16_ms:
        res["speedup_vs_bf16_step"] = round(bf16_ms / ms, 3)
    return res


def stack_leg(db, wl, n_blocks, steps, stream, reps=3):
    """The paper's regime (Sec. 2.3, Sec. 3.3): one request = the selection once, then for each
    sampling step: compress that step's latents, run `n_blocks` blocks on the compressed tokens
    (hilo_blocks), decompress.  Against it: the same blocks on the uncompressed tokens every step
    (no selection, compression or decompression).  Every block has its own random-init weights
    (N(0, 0.02), bf16, generated on the device) and modulation; each step's latents are the
    previous step's plus N(0, 0.1) changes."""
    import torch

    from paper_2606_13898_amd import hilo

    s = wl.shape
    D, F, B, NB = s.dim, s.mlp_dim, s.batch, s.n_blocks
    dt = db.dtype
    g = torch.Generator(device="cuda")
    g.manual_seed(4242)

    def rnd(*shape, std=0.02, dtype=dt):
        return (torch.randn(*shape, generator=g, device="cuda", dtype=torch.float32) * std).to(dtype)

    weights = [[{"w_qkv": rnd(3 * D, D), "b_qkv": rnd(3 * D), "w_o": rnd(D, D), "b_o": rnd(D),
                 "w1": rnd(F, D), "b1": rnd(F), "w2": rnd(D, F), "b2": rnd(D)} for _ in range(2)]
               for _ in range(n_blocks)]
    aw, mw = hilo.stack_weights(weights)
    mods = rnd(steps, n_blocks, B, 2, 6, D, std=0.1, dtype=torch.float32)
    xs = [db.x_img]
    for _ in range(steps - 1):
        xs.append((xs[-1].float() + rnd(*xs[-1].shape, std=0.1, dtype=torch.float32)).to(dt))
    ws = db.ws

    def request(keep):
        db.x_img = xs[0]
        db.score()
        db.select(hilo.TOPK, keep=keep)
        for t in range(steps):
            hilo.hilo_compress(db.shape, xs[t], db.x_txt, db.fine_idx, db.pool_idx, db.counts, db.cu,
                               db.seg, db.z)
            hilo.hilo_blocks(db.shape, db.z, db.cu, aw, mw, mods[t], n_blocks, ws)
            hilo.hilo_decompress(db.shape, db.z, db.idx_map, db.cu, db.seg, db.y_img, db.y_txt)

    def dense_blocks():
        for t in range(steps):
            hilo.hilo_compress(db.shape, xs[t], db.x_txt, db.fine_idx, db.pool_idx, db.counts, db.cu,
                               db.seg, db.z)  # every block fine: the dense token order, untimed
            e0.record(stream)
            hilo.hilo_blocks(db.shape, db.z, db.cu, aw, mw, mods[t], n_blocks, ws)
            e1.record(stream)
            torch.cuda.synchronize()
            times.append(e0.elapsed_time(e1))

    x0 = db.x_img
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    request(wl.keep)  # warm-up
    torch.cuda.synchronize()
    req = []
    for _ in range(reps):
        e0.record(stream)
        request(wl.keep)
        e1.record(stream)
        torch.cuda.synchronize()
        req.append(e0.elapsed_time(e1))
    nc = int(db.cu.cpu().numpy()[-1])
    db.score()
    db.select(hilo.TOPK, keep=[NB] * s.grids)
    times = []
    dense_blocks()  # warm-up
    times = []
    for _ in range(reps):
        dense_blocks()
    db.x_img = x0
    nd = int(db.cu.cpu().numpy()[-1])
    req_ms = sorted(req)[len(req) // 2]
    dense_ms = sorted(times)[len(times) // 2] * steps  # median step, times the steps of a request
    del weights, aw, mw, mods, xs
    return {"blocks": n_blocks, "sampling_steps": steps, "requests_timed": reps,
            "request_ms": round(req_ms, 3), "dense_request_ms": round(dense_ms, 3),
            "speedup_vs_dense": round(dense_ms / req_ms, 3), "token_ratio": round(nd / nc, 3),
            "compressed_tokens": nc, "dense_tokens": nd,
            "ms_per_block": round(req_ms / (steps * n_blocks), 4),
            "dense_ms_per_block": round(dense_ms / (steps * n_blocks), 4)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="m1024", choices=sorted(DESCR))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--no-stack", action="store_true",
                    help="skip the request leg (selection once, then per sampling step compress -> "
                         "a stack of blocks -> decompress, against the same stack on the dense tokens)")
    ap.add_argument("--no-token-sets", action="store_true",
                    help="skip the token-set leg (the step with every block's pooled token kept next "
                         "to the fine patches, and with the fine patches alone)")
    ap.add_argument("--no-pixel-score", action="store_true",
                    help="skip the pixel-space scorer leg (Sobel on the 16x-resolution RGB image)")
    ap.add_argument("--no-fp8", action="store_true",
                    help="skip the step with FP8 projections")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the other workloads (2048 px, edit with r = 0 and 1, ragged batch of 8)")
    ap.add_argument("--no-sweep", action="store_true",
                    help="skip the kept-fraction sweep (0, 25, 50, 75, 100% of the blocks on one sample)")
    ap.add_argument("--stack-blocks", type=int, default=8)
    ap.add_argument("--stack-steps", type=int, default=8)
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="only run one plain device-to-device copy of this many MiB (the known-size "
                         "kernel that calibrates the HBM traffic counters) and exit")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the compressed block runs on a single MI355X; "
              "multi-GPU runs are not part of this build", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    if args.copy_mib:
        a = torch.ones(args.copy_mib << 20, dtype=torch.uint8, device="cuda")
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copied_bytes": a.numel()}))
        return

    from paper_2606_13898_amd import hilo, inputs
    from paper_2606_13898_amd.pipeline import DeviceBlock

    hilo.lib()  # fail loudly if the library is not built
    torch.cuda.set_device(0)
    wl = inputs.make_workload(args.workload)
    s = wl.shape
    db = DeviceBlock(wl)
    stream = torch.cuda.current_stream()
    weight_sets, _w2 = Rotation.weight_sets(db)
    rot = Rotation(db, weight_sets=weight_sets)
    sec_steps, sec_warm = min(args.steps, 10), min(args.warmup, 3)

    def step(k):
        rot.use(db, k)
        db.run(hilo.TOPK)

    for k in range(args.warmup):
        step(k)
    torch.cuda.synchronize()
    # one event between consecutive steps: the mean over the K steps is the value, the per-step
    # durations give the median and the 10th / 90th percentiles
    t0 = time.perf_counter()
    ms, per_step = timed(stream, args.steps, step)
    wall = (time.perf_counter() - t0) * 1e3 / args.steps
    pct = lambda q: float(per_step[min(len(per_step) - 1, int(round(q * (len(per_step) - 1))))])
    counts = db.counts.cpu().numpy()
    cu = db.cu.cpu().numpy()
    nc = int(cu[-1])

    # per-kernel durations: the same steps again with the library's event pairs around each kernel
    work = kernel_work(s, counts, cu)
    kern = kernel_profile(args.steps, step, work)
    dom = max((k for k in kern if k in work), key=lambda k: kern[k]["ms"])
    d = kern[dom]
    roof = {"kernel": dom, "bound": "mfma" if d["unit"] == "TFLOP/s" else "hbm",
            "achieved": d["achieved"], "peak": d["peak"], "unit": d["unit"], "frac": d["frac"],
            "traffic": traffic_for(dom)}
    t_blk = sum(kern[k]["ms"] for k in BLOCK_KERNELS if k in kern)
    # the Sobel score is bound by the vector ALU (its exact fixed-point energy), not by HBM: its
    # instruction count at the issue peak is the floor it is measured against as well
    nv = valu_for("score")
    if "score" in kern and nv:
        floor = nv / PEAK_VALU_INSTS_PER_S * 1e3
        kern["score"]["alu"] = {"bound": "alu", "valu_insts_per_launch": nv,
                                "peak": "%.4g wave64 instructions/s" % PEAK_VALU_INSTS_PER_S,
                                "floor_ms": round(floor, 4), "frac": round(floor / kern["score"]["ms"], 4)}

    # the box's plain device copy, for the memory-bound kernels' fractions (read + write bytes)
    cp_a = torch.empty(256 << 20, dtype=torch.uint8, device="cuda")
    cp_b = torch.empty_like(cp_a)
    for _ in range(3):
        cp_b.copy_(cp_a)
    cp_ms, _ = timed(stream, 10, lambda k: cp_b.copy_(cp_a))
    copy_ref = {"bytes_per_copy": 2 * cp_a.numel(), "gbs": round(2 * cp_a.numel() / (cp_ms * 1e-3) / 1e9, 1)}
    del cp_a, cp_b

    # the same block on the uncompressed sequence (every block kept fine)
    dense = None
    if not args.no_dense:
        dense_ms, n_dense, cud = dense_block_ms(db, rot, args.steps, args.warmup, stream)
        dense = {"block_ms": round(dense_ms, 4), "tokens": n_dense,
                 "flop_ratio": round(block_flops(s, np.diff(cud)) / block_flops(s, np.diff(cu)), 3)}
        db.run(hilo.TOPK)

    sweep = None
    if not args.no_sweep and s.batch == 1 and s.images == 1:
        NB = s.n_blocks
        sweep = sweep_leg(db, rot, sec_steps, sec_warm, stream, [0, NB // 4, NB // 2, 3 * NB // 4, NB])

    token_sets = None
    if not args.no_token_sets:
        token_sets = token_set_leg(db, rot, sec_steps, sec_warm, stream, dense["block_ms"] if dense else None)

    pixel = None
    if not args.no_pixel_score:
        pixel = pixel_leg(db, sec_steps, sec_warm, stream)

    fp8 = None
    if not args.no_fp8 and s.dtype == "bf16" and s.dim % 128 == 0 and s.mlp_dim % 128 == 0:
        fp8 = fp8_leg(db, rot, sec_steps, sec_warm, stream, work, ms)

    stack = None
    if not args.no_stack:
        stack = stack_leg(db, wl, args.stack_blocks, args.stack_steps, stream)

    configs = None
    if not args.no_configs and args.workload == "m1024":
        configs = {}
        for name, r in (("h2048", 0), ("edit", 0), ("edit", 1), ("ragged", 0)):
            key = name + (f"_r{r}" if r else "")
            configs[key] = config_leg(name, db, weight_sets, sec_steps, sec_warm, stream, r)

    attn = kern.get("attention_core", {})
    out = {
        "metric": METRIC,
        "value": round(ms, 4),
        "unit": "ms",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "wall_ms_per_step": round(wall, 4),
        "ms_per_step_median": round(pct(0.5), 4),
        "ms_per_step_p10": round(pct(0.1), 4),
        "ms_per_step_p90": round(pct(0.9), 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": s.dtype,
        "data": "synthetic (seeded latents, random-init weights of the block's shape)",
        "config": {"workload": f"{args.workload}: {DESCR[args.workload]}",
                   "batch": s.batch, "images": s.images, "grid": f"{s.grid_h}x{s.grid_w}",
                   "text_tokens": s.text_len, "dim": s.dim, "heads": s.heads,
                   "head_dim": s.head_dim, "mlp_dim": s.mlp_dim,
                   "compressed_tokens": nc, "dense_tokens": s.max_tokens},
        "timing": {"input_copies": rot.R, "input_bytes_rotated": rot.bytes, "weight_copies": len(weight_sets),
                   "note": "step k reads input copy k % input_copies and weight copy k % weight_copies"},
        "block_ms": round(t_blk, 4),
        "attn_tflops": attn.get("achieved"),
        "compressed_tokens_per_s": round(nc / (ms * 1e-3), 1),
        "represented_tokens_per_s": round(s.max_tokens / (ms * 1e-3), 1),
        "roofline": roof,
        "kernels": kern,
        "hbm_copy_reference": copy_ref,
    }
    if dense:
        out["dense"] = dense
        out["speedup_vs_dense"] = round(dense["block_ms"] / ms, 3)
        out["block_speedup_vs_dense"] = round(dense["block_ms"] / t_blk, 3) if t_blk else None
        out["token_ratio"] = round(dense["tokens"] / nc, 3)
        out["flop_ratio"] = dense["flop_ratio"]
    if sweep:
        out["kept_fraction_sweep"] = sweep
    if configs:
        out["configs"] = configs
    if token_sets:
        out["token_sets"] = token_sets
    if pixel:
        out["pixel_score"] = pixel
    if fp8:
        out["fp8"] = fp8
    if stack:
        out["stack"] = stack
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
