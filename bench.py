#!/usr/bin/env python3
"""Benchmark of the HiLo-Token compressed DiT block on one MI355X.

One step = one pass of the whole hot path over one batch: score, select, compress, attention,
MLP, decompress (six C-ABI calls, all kernels on the GPU), inputs resident in HBM.  Prints ONE JSON
line with the step latency, throughput, the dense (uncompressed) block for the speedup, per-kernel
times from HIP events with their roofline fractions, and the CPU oracle timed on a bounded sample.

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
        "compress": ((G * N * D * es + n_img * D * 4 + B * L * D * (es + 4)) / 1e9, "GB", PEAK_HBM_GBS),
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


def cpu_baseline(wl):
    """The oracle, untuned, on one full step of the same workload (bounded: ~10-30 s)."""
    import threadpoolctl

    from oracle import hilo_oracle as O

    info = threadpoolctl.threadpool_info()
    threads = max([i.get("num_threads", 1) for i in info if i.get("user_api") == "blas"] or [1])
    t0 = time.perf_counter()
    O.pipeline(wl.x_img, wl.x_txt, wl.shape, wl.force, wl.dilate_r, "topk", keep=wl.keep,
               weights=wl.weights, mod=wl.mod)
    dt = time.perf_counter() - t0
    return {"value": round(dt * 1e3, 1), "unit": "ms", "cores": int(threads), "kind": "oracle",
            "sample": f"one full step (score..decompress) of the {wl.name} workload in float64 "
                      f"numpy, BLAS threads={threads}"}


def pixel_leg(db, steps, warmup, stream):
    """The paper's own selector input: Sobel on the RGB image at 16x the token grid (1024 x 1024
    pixels for the 64 x 64 grid), summed per token (hilo_score_pixels), then its threshold 0.1 on
    the normalised map.  The image is synthetic (inputs.pixel_image).  HBM-bound: one read of the
    image plus the 8-byte energies."""
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
    db.select(hilo.THRESHOLD, tau=[0.1] * G)
    counts = db.counts.cpu().numpy()
    res = {"ms": round(ms, 4), "image": f"{G}x3x{16 * s.grid_h}x{16 * s.grid_w} float32",
           "achieved": round(gbs, 1), "unit": "GB/s", "peak": 8000.0, "frac": round(gbs / 8000.0, 4),
           "work_per_launch": f"{nbytes / 1e9:.4g} GB",
           "kept_fine_fraction_tau_0.1": round(float(counts[:, 0].sum()) / (G * N), 4)}
    db.run(hilo.TOPK)  # leave the buffers as the default step left them
    torch.cuda.synchronize()
    return res


def token_set_leg(db, steps, warmup, stream, dense_ms):
    """The whole step with the other token sets (same selection rule): overlap -- every block's
    pooled token kept next to the fine patches, the paper's own token set (Sec. 2.3) -- and drop --
    the fine patches alone (Sec. 3.2) -- both reassembled in the delta form; partition with the
    delta form for comparison."""
    import torch

    from paper_2606_13898_amd import hilo

    res = {}
    for name, tokens in (("overlap", hilo.OVERLAP), ("drop", hilo.DROP), ("partition", hilo.PARTITION)):
        for _ in range(warmup):
            db.run(hilo.TOPK, tokens=tokens, delta=True)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(steps):
            db.run(hilo.TOPK, tokens=tokens, delta=True)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        nc = int(db.cu.cpu().numpy()[-1])
        ent = {"ms_per_step": round(ms, 4), "compressed_tokens": nc, "decompress": "delta"}
        if dense_ms:
            ent["speedup_vs_dense"] = round(dense_ms / ms, 3)
        res[name] = ent
    db.run(hilo.TOPK)  # leave the buffers as the default step left them
    torch.cuda.synchronize()
    return res


def fp8_leg(db, steps, warmup, stream, work, bf16_ms):
    """The step with all four projections in FP8 (per-row E4M3 operands: one scale per token for the
    activations, one per output channel for the weights; Sec. 3.3 combines the compression with FP8
    quantisation): step latency, the projections' rates against the fp8 MFMA peak, the two passes
    that quantise the attention and GELU outputs, and how far the block's update of the compressed
    tokens moves from the bf16 step's (relative L2 over all rows)."""
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

    for _ in range(warmup):
        db.run(hilo.TOPK, fp8=True)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    evs[0].record(stream)
    for k in range(steps):
        db.run(hilo.TOPK, fp8=True)
        evs[k + 1].record(stream)
    torch.cuda.synchronize()
    ms = evs[0].elapsed_time(evs[-1]) / steps
    per_step = np.sort([evs[k].elapsed_time(evs[k + 1]) for k in range(steps)])

    hilo.hilo_profile_enable(True)
    for _ in range(steps):
        db.run(hilo.TOPK, fp8=True)
    torch.cuda.synchronize()
    kern = {}
    for k in range(hilo.hilo_profile_kinds()):
        name = hilo.hilo_profile_name(k)
        tot, n = hilo.hilo_profile_read(k)
        if n and name in ("rownorm_attn", "gemm_qkv", "quantize_attn", "gemm_o", "rownorm_mlp", "gemm_fc1",
                          "quantize_mlp", "gemm_fc2"):
            avg = tot / n
            ent = {"ms": round(avg, 4)}
            if name.startswith("gemm"):
                ach = work[name][0] / (avg * 1e-3)
                ent.update(achieved=round(ach, 1), unit="TFLOP/s", peak=PEAK_FP8_TFLOPS,
                           frac=round(ach / PEAK_FP8_TFLOPS, 4))
            kern[name] = ent
    hilo.hilo_profile_enable(False)
    db.run(hilo.TOPK)  # leave the buffers as the default step left them
    torch.cuda.synchronize()
    res = {"ms_per_step": round(ms, 4), "ms_per_step_median": round(float(per_step[len(per_step) // 2]), 4),
           "projections_in_fp8": ["qkv", "attention_output", "mlp_up", "mlp_down"], "kernels": kern,
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

    def step():
        db.run(hilo.TOPK)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # one event between consecutive steps: the mean over the K steps is the value, the per-step
    # durations give the median and the 10th / 90th percentiles
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    t0 = time.perf_counter()
    evs[0].record(stream)
    for k in range(args.steps):
        step()
        evs[k + 1].record(stream)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3 / args.steps
    ms = evs[0].elapsed_time(evs[-1]) / args.steps
    per_step = np.sort([evs[k].elapsed_time(evs[k + 1]) for k in range(args.steps)])
    pct = lambda q: float(per_step[min(len(per_step) - 1, int(round(q * (len(per_step) - 1))))])
    counts = db.counts.cpu().numpy()
    cu = db.cu.cpu().numpy()
    nc = int(cu[-1])

    # per-kernel durations: the same steps again with the library's event pairs around each kernel
    hilo.hilo_profile_enable(True)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    kinds = {hilo.hilo_profile_name(k): hilo.hilo_profile_read(k) for k in range(hilo.hilo_profile_kinds())}
    hilo.hilo_profile_enable(False)
    work = kernel_work(s, counts, cu)
    kern = {}
    for name, (tot, n) in kinds.items():
        if n == 0:
            continue
        avg = tot / n
        ent = {"ms": round(avg, 4), "launches_per_step": n // args.steps}
        if name in work:
            amt, unit, peak = work[name]
            ach = amt / (avg * 1e-3)  # GB/s or TFLOP/s
            ent.update(achieved=round(ach, 1), unit=unit + "/s", peak=peak,
                       frac=round(ach / peak, 4), work_per_launch=f"{amt:.4g} {unit}")
        kern[name] = ent
    dom = max((k for k in kern if k in work), key=lambda k: kern[k]["ms"])
    d = kern[dom]
    roof = {"kernel": dom, "bound": "mfma" if d["unit"] == "TFLOP/s" else "hbm",
            "achieved": d["achieved"], "peak": d["peak"], "unit": d["unit"], "frac": d["frac"],
            "traffic": traffic_for(dom)}
    t_blk = sum(kern[k]["ms"] for k in ("rownorm_attn", "gemm_qkv", "attention_core", "gemm_o",
                                        "rownorm_mlp", "gemm_fc1", "gemm_fc2") if k in kern)

    # the same block on the uncompressed sequence (every block kept fine)
    dense = None
    if not args.no_dense:
        NB = s.n_blocks
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(args.steps)]
        db.score()
        db.select(hilo.TOPK, keep=[NB] * s.grids)
        for _ in range(args.warmup):
            db.compress()
            db.attention()
            db.mlp()
        for a, b in ev:
            db.compress()
            a.record(stream)
            db.attention()
            db.mlp()
            b.record(stream)
        torch.cuda.synchronize()
        dense_ms = sum(a.elapsed_time(b) for a, b in ev) / args.steps
        n_dense = int(db.cu.cpu().numpy()[-1])
        dense = {"block_ms": round(dense_ms, 4), "tokens": n_dense}

    token_sets = None
    if not args.no_token_sets:
        token_sets = token_set_leg(db, args.steps, args.warmup, stream,
                                   dense["block_ms"] if dense else None)

    pixel = None
    if not args.no_pixel_score:
        pixel = pixel_leg(db, args.steps, args.warmup, stream)

    fp8 = None
    if not args.no_fp8 and s.dtype == "bf16" and s.dim % 128 == 0 and s.mlp_dim % 128 == 0:
        fp8 = fp8_leg(db, args.steps, args.warmup, stream, work, ms)

    stack = None
    if not args.no_stack:
        stack = stack_leg(db, wl, args.stack_blocks, args.stack_steps, stream)

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
        "block_ms": round(t_blk, 4),
        "attn_tflops": attn.get("achieved"),
        "compressed_tokens_per_s": round(nc / (ms * 1e-3), 1),
        "represented_tokens_per_s": round(s.max_tokens / (ms * 1e-3), 1),
        "roofline": roof,
        "kernels": kern,
    }
    if dense:
        out["dense"] = dense
        out["speedup_vs_dense"] = round(dense["block_ms"] / ms, 3)
        out["block_speedup_vs_dense"] = round(dense["block_ms"] / t_blk, 3) if t_blk else None
        out["token_ratio"] = round(dense["tokens"] / nc, 3)
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
