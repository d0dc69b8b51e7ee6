#!/usr/bin/env python3
"""HBM traffic and MFMA utilisation per launch of every kernel kind of the bench, from rocprofv3
counters.

Two counter passes over a short bench run (FETCH_SIZE, then WRITE_SIZE: bytes between the L2 and
memory, per dispatch) and the same two passes over one plain device copy of known size, which
calibrates each counter (calibrated bytes = counter / (counter of the copy / bytes the copy moves)).
The result, profiles/traffic.json, is what bench.py reports as roofline.traffic; each entry carries
a digest of the kernel sources it was measured on, and bench.py drops it once they change.

A fifth pass reads the matrix-core counters: SQ_VALU_MFMA_BUSY_CYCLES (summed over the SIMDs: 32
busy cycles per 32x32x16 bf16 MFMA, 16 per 16x16x32), GRBM_GUI_ACTIVE (summed over the 8 XCDs:
divided by 8 it is the dispatch's length in GPU cycles), SQ_INSTS_MFMA and SQ_INSTS_VALU.  MFMA
utilisation = busy cycles / (SIMDs x GUI cycles / 8), written to profiles/mfma_m1024.md.

    python traffic.py commands OUTDIR        # print the five rocprofv3 commands (run them on the GPU)
    python traffic.py summarize OUTDIR       # write profiles/traffic.json, traffic_m1024.md, mfma_m1024.md
"""
from __future__ import annotations

import collections
import csv
import json
import os
import sys

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from bench import source_digest  # noqa: E402

COPY_MIB = 256
BENCH = ("python3 {root}/bench.py --steps 2 --warmup 1 --no-dense --no-cpu-baseline --no-fp8 --no-stack "
         "--no-token-sets --no-pixel-score --no-configs --no-sweep")
COPY = "python3 {root}/bench.py --copy-mib %d" % COPY_MIB
COUNTERS = ("FETCH_SIZE", "WRITE_SIZE")
MFMA_COUNTERS = "SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_MFMA SQ_INSTS_VALU SQ_BUSY_CYCLES GRBM_GUI_ACTIVE"
SIMDS = 256 * 4      # MI355X: 256 compute units of 4 SIMDs
XCDS = 8

CSRC = "paper_2606_13898_amd/csrc/"
HDRS = [CSRC + "common.h", CSRC + "kernels.h"]
SOURCES = {
    "score": [CSRC + "select.hip"], "select": [CSRC + "select.hip"], "layout": [CSRC + "select.hip"],
    "compress": [CSRC + "pack.hip"], "decompress": [CSRC + "pack.hip"],
    "rownorm_attn": [CSRC + "pack.hip"], "rownorm_mlp": [CSRC + "pack.hip"],
    "gemm_qkv": [CSRC + "gemm.hip"], "gemm_o": [CSRC + "gemm.hip"], "gemm_fc1": [CSRC + "gemm.hip"],
    "gemm_fc2": [CSRC + "gemm.hip"], "attention_core": [CSRC + "attention.hip"],
}
ROLES = {"0": "gemm_qkv", "1": "gemm_o", "2": "gemm_fc1", "3": "gemm_fc2"}


def commands(out):
    cmds = []
    for cnt in COUNTERS:
        for tag, prog in (("bench", BENCH), ("copy", COPY)):
            cmds.append(f"timeout -s KILL 120 rocprofv3 --pmc {cnt} --output-format csv "
                        f"-d {out}/{cnt} -o {tag} -- {prog.format(root=ROOT)}")
    cmds.append(f"timeout -s KILL 120 rocprofv3 --pmc {MFMA_COUNTERS} --output-format csv "
                f"-d {out}/MFMA -o bench -- {BENCH.format(root=ROOT)}")
    return cmds


def load_multi(path):
    """{dispatch id: (kernel name, duration ns, {counter: value})} of a multi-counter pass."""
    per = collections.OrderedDict()
    with open(path) as f:
        for r in csv.DictReader(f):
            key = int(r["Dispatch_Id"])
            ent = per.setdefault(key, [r["Kernel_Name"], int(r["End_Timestamp"]) - int(r["Start_Timestamp"]), {}])
            ent[2][r["Counter_Name"]] = ent[2].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    return per


def summarize_mfma(out):
    path = os.path.join(out, "MFMA", "bench_counter_collection.csv")
    if not os.path.exists(path):
        return None
    agg = collections.defaultdict(lambda: collections.defaultdict(float))
    n = collections.Counter()
    state = {}
    for _, (name, dur, cs) in load_multi(path).items():
        k = kind_of(name, state)
        if k is None or not is_main(name):
            continue
        n[k] += 1 if primary(name) else 0
        agg[k]["dur_ns"] += dur
        for c, v in cs.items():
            agg[k][c] += v
    rows = {}
    for k, a in agg.items():
        c = n[k]
        gui = a["GRBM_GUI_ACTIVE"] / c / XCDS
        rows[k] = {"us": a["dur_ns"] / c / 1e3, "clock_ghz": gui / (a["dur_ns"] / c),
                   "mfma_busy": a["SQ_VALU_MFMA_BUSY_CYCLES"] / c / (SIMDS * gui) if gui else 0.0,
                   "mfma_insts": a["SQ_INSTS_MFMA"] / c, "valu_insts": a["SQ_INSTS_VALU"] / c}
    lines = ["# MFMA utilisation per call, m1024 workload (rocprofv3 SQ_VALU_MFMA_BUSY_CYCLES)", "",
             "MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (%d SIMDs x GRBM_GUI_ACTIVE / %d): the share of the "
             "dispatch's GPU cycles the matrix cores were busy (the counter adds 32 cycles per "
             "32x32x16 and 16 per 16x16x32 bf16 MFMA over all SIMDs; GRBM_GUI_ACTIVE adds the "
             "dispatch's cycles over the %d XCDs).  Main kernels only (the GEMM fixups and the "
             "attention merge issue no MFMA)." %
             (SIMDS, XCDS, XCDS), "",
             "Command:", "", "    " + commands(out)[-1], "",
             "| kind | us | clock GHz | MFMA busy | MFMA insts | VALU insts | VALU per MFMA |",
             "|---|---:|---:|---:|---:|---:|---:|"]
    for k, r in sorted(rows.items(), key=lambda kv: -kv[1]["us"]):
        vpm = r["valu_insts"] / r["mfma_insts"] if r["mfma_insts"] else float("nan")
        lines.append(f"| {k} | {r['us']:.1f} | {r['clock_ghz']:.2f} | {100 * r['mfma_busy']:.1f}% | "
                     f"{r['mfma_insts']:.4g} | {r['valu_insts']:.4g} | {vpm:.2f} |")
    with open(os.path.join(ROOT, "profiles", "mfma_m1024.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    return rows


def load(out, cnt, tag):
    """[(dispatch id, kernel name, value)] in dispatch order, values summed per dispatch."""
    path = os.path.join(out, cnt, f"{tag}_counter_collection.csv")
    per = collections.OrderedDict()
    with open(path) as f:
        for r in csv.DictReader(f):
            key = int(r["Dispatch_Id"])
            name = r["Kernel_Name"]
            per.setdefault(key, [name, 0.0])[1] += float(r["Counter_Value"])
    return [(d, n, v) for d, (n, v) in sorted(per.items())]


def gemm_role(base):
    """Projection of a GEMM kernel from its template arguments: k_gemm_fix<BM, BN, WM, WN, EPI, ROLE,
    F8>, k_gemm_big<BM, BN, EPI, ROLE, F8>."""
    args = [a.strip() for a in base[base.index("<") + 1:base.rindex(">")].split(",")]
    return ROLES[args[3] if base.startswith("hilo::k_gemm_big") else args[5]]


def kind_of(name, state):
    """Bench kernel kind of a dispatch; rownorm launches alternate attention / MLP per step."""
    base = name.split("(")[0].replace("void ", "").strip()
    if "k_gemm_fix<" in base or "k_gemm_big<" in base:
        return gemm_role(base)
    if "k_attn" in base:
        return "attention_core"
    if "k_compress_norm<" in base:
        state["fused"] = True  # the attention half's row norm runs in the compress pass
        return "compress"
    if "k_rownorm" in base:
        if state.get("fused"):
            return "rownorm_mlp"
        state["rownorm"] = state.get("rownorm", 0) + 1
        return "rownorm_attn" if state["rownorm"] % 2 == 1 else "rownorm_mlp"
    if "k_score_bf16<" in base:
        return "score"
    for k in ("k_score", "k_select", "k_layout", "k_compress", "k_decompress"):
        if k + "<" in base or base.endswith(k):
            return k[2:]
    return None


def is_main(name):
    """A kernel that does a call's MFMA work (not a GEMM fixup or the attention merge)."""
    return "k_gemm_fix" not in name and "k_attn_fix" not in name


def primary(name):
    """The kernel of each kind's call whose dispatch count is the number of calls: its main kernel."""
    return is_main(name)


def summarize(out):
    factor = {}
    for cnt in COUNTERS:
        copy = load(out, cnt, "copy")
        big = max(copy, key=lambda r: r[2])
        factor[cnt] = big[2] * 1024.0 / (COPY_MIB << 20)   # counter KiB per byte actually moved
    tot = collections.defaultdict(lambda: {"FETCH_SIZE": 0.0, "WRITE_SIZE": 0.0})
    calls = collections.Counter()
    for cnt in COUNTERS:
        state = {}
        for _, name, v in load(out, cnt, "bench"):
            k = kind_of(name, state)
            if k is None:
                continue
            tot[k][cnt] += v * 1024.0 / factor[cnt]
            if cnt == "FETCH_SIZE" and primary(name):
                calls[k] += 1
    kernels = {}
    for k, t in tot.items():
        n = calls[k]
        if not n or k not in SOURCES:
            continue
        srcs = SOURCES[k] + HDRS
        kernels[k] = {"bytes_per_launch": round((t["FETCH_SIZE"] + t["WRITE_SIZE"]) / n),
                      "fetch_bytes_per_launch": round(t["FETCH_SIZE"] / n),
                      "write_bytes_per_launch": round(t["WRITE_SIZE"] / n),
                      "launches_measured": n, "sources": srcs, "source_digest": source_digest(srcs)}
    # vector-ALU instructions per launch (the counter pass), for the kernels bound by the vector ALU
    mf = summarize_mfma(out)
    for k, e in kernels.items():
        if mf and k in mf:
            e["valu_insts_per_launch"] = round(mf[k]["valu_insts"])
    res = {"workload": "m1024", "calibration": {"copy_bytes": COPY_MIB << 20,
                                                "fetch_counter_per_byte": factor["FETCH_SIZE"],
                                                "write_counter_per_byte": factor["WRITE_SIZE"]},
           "commands": commands(out), "kernels": kernels}
    os.makedirs(os.path.join(ROOT, "profiles"), exist_ok=True)
    with open(os.path.join(ROOT, "profiles", "traffic.json"), "w") as f:
        json.dump(res, f, indent=1)
    lines = ["# HBM traffic per call, m1024 workload (rocprofv3 FETCH_SIZE / WRITE_SIZE)", "",
             "Counters calibrated on one %d MiB device copy: FETCH_SIZE reads %.3f, WRITE_SIZE %.3f "
             "of the bytes the copy moves; every figure below is divided by that factor." %
             (COPY_MIB, factor["FETCH_SIZE"], factor["WRITE_SIZE"]), "",
             "Commands (then `python traffic.py summarize %s`):" % out, ""]
    lines += ["    " + c for c in commands(out)[:4]]
    lines += ["", "| kind | read MB | write MB | total MB |", "|---|---:|---:|---:|"]
    for k, e in sorted(kernels.items(), key=lambda kv: -kv[1]["bytes_per_launch"]):
        lines.append(f"| {k} | {e['fetch_bytes_per_launch'] / 1e6:.1f} | "
                     f"{e['write_bytes_per_launch'] / 1e6:.1f} | {e['bytes_per_launch'] / 1e6:.1f} |")
    with open(os.path.join(ROOT, "profiles", "traffic_m1024.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    print(json.dumps({k: v["bytes_per_launch"] for k, v in kernels.items()}, indent=1))
    if mf:
        print(json.dumps({k: round(100 * v["mfma_busy"], 1) for k, v in mf.items()}, indent=1))


if __name__ == "__main__":
    if len(sys.argv) != 3 or sys.argv[1] not in ("commands", "summarize"):
        print(__doc__)
        sys.exit(2)
    if sys.argv[1] == "commands":
        print("\n".join(commands(sys.argv[2])))
    else:
        summarize(sys.argv[2])
