"""Benchmark of the Ball Sparse Attention layer hot path on one MI355X.

One step = ball-tree ordering of a 65536-point cloud, ordering of its Q/K/V rows and
gate logits, the layer forward pass and the layer backward pass (all on the GPU, all
through the C ABI). Inputs are seeded synthetic data already resident in HBM: a
32-component Gaussian mixture cloud, Q/K/V ~ N(0,1) in bf16, 8 heads of dim 64, ball
256, compression blocks of 16, selection blocks of 32, top-16, groups of 16.

Prints one JSON line (rank 0, N=1). Usage: python bench.py [--steps K] [--warmup W]
[--variant bsa|group_cmp|g1]. The default is the regular layer; group_cmp is the variant
with MLP query coarsening (Eq. 13-14) and group compression (Eq. 15); g1 selects blocks per
token (Eq. 6-8 without the grouping of Eq. 10-12).
"""
from __future__ import annotations

import argparse
import dataclasses
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

MFMA_BF16_PEAK = 2.5e15     # MI355X dense bf16 MFMA, FLOP/s
HBM_PEAK = 8.0e12           # MI355X HBM3E, B/s


VARIANTS = {
    "bsa": {},
    "group_cmp": {"q_coarsen": 1, "group_compression": 1},
    "g1": {},          # per-token selection: the workload with group size 1
}


def algorithmic_flops(cfg, variant="bsa"):
    """Work the method must do (not the dense work it avoids), per step.

    Per head: ball 4 N m d; MLP 2 (N/l)(l d d + d d) per tensor (K and V, plus Q for the
    group-compression variant); compressed attention 4 N (N/l) d (group compression:
    4 (N/l)(N/l) d); scoring 2 (N/g)(N/l) d; selection 4 N k* l' d. Backward: 2.5x each
    attention term (5 vs 2 matrix products), 2x the MLP, nothing for scoring.
    """
    B, H, N, d = cfg.batch, cfg.heads, cfg.n_pad, cfg.head_dim
    m, l, ls, k, g = cfg.ball, cfg.cmp_block, cfg.slc_block, cfg.topk, cfg.group
    gc = variant == "group_cmp"
    per = {
        "ball": 4.0 * N * m * d,
        "mlp": (3 if gc else 2) * 2.0 * (N / l) * (l * d * d + d * d),
        "cmp": 4.0 * (N / l if gc else N) * (N / l) * d,
        "score": 2.0 * (N / g) * (N / l) * d,
        "slc": 4.0 * N * k * ls * d,
    }
    fwd = {n: v * B * H for n, v in per.items()}
    bwd = {"ball": 2.5 * fwd["ball"], "mlp": 2 * fwd["mlp"], "cmp": 2.5 * fwd["cmp"], "score": 0.0,
           "slc": 2.5 * fwd["slc"]}
    return fwd, bwd


# phases that share the chip with a concurrent branch: forward ball + compressed attention
# beside top-k selection + selection attention where the two run as separate launches (the
# forward of the shared ball + compressed launch runs on one stream); the backward dQ chain
# beside the compression and selection dK/dV passes
CONCURRENT_PHASES = ["fwd.ball", "fwd.cmp", "fwd.select", "fwd.slc", "bwd.dq_ball", "bwd.dq_cmp", "bwd.dq_slc",
                     "bwd.mlp", "bwd.slc_csr", "bwd.slc_kv"]


def concurrent_phases(phase_ms):
    """The phases of CONCURRENT_PHASES that shared the chip in this run."""
    shared_fwd = phase_ms.get("fwd.ball_cmp", 0.0) > 0
    return [p for p in CONCURRENT_PHASES if not (shared_fwd and p.startswith("fwd."))]


def phase_flops(cfg, variant="bsa"):
    """Algorithmic FLOPs of each timed phase (same totals as algorithmic_flops).

    Backward split: the key-major kernels compute the recomputed scores, dP, dK and dV
    (4 products, 8 d FLOP per query-key pair); the query-major kernels are credited only
    with dQ (2 d), their recomputation of scores and dP being overhead of the split.
    """
    B, H, N, d = cfg.batch, cfg.heads, cfg.n_pad, cfg.head_dim
    m, l, ls, k, g = cfg.ball, cfg.cmp_block, cfg.slc_block, cfg.topk, cfg.group
    gc = variant == "group_cmp"
    pairs = {"ball": N * m, "cmp": (N // l if gc else N) * (N // l), "slc": N * k * ls}
    mlp = (3 if gc else 2) * 2.0 * (N / l) * (l * d * d + d * d) * B * H
    f = {"fwd.compress": mlp, "fwd.select": 2.0 * (N / g) * (N / l) * d * B * H, "bwd.mlp": 2 * mlp}
    for br, kv in (("ball", "kv_ball"), ("cmp", "kv_cmp"), ("slc", "slc_kv")):
        f[f"fwd.{br}"] = 4.0 * pairs[br] * d * B * H
        f[f"bwd.dq_{br}"] = 2.0 * pairs[br] * d * B * H
        f[f"bwd.{kv}"] = 8.0 * pairs[br] * d * B * H
    f["bwd.kv"] = f["bwd.kv_ball"] + f["bwd.kv_cmp"]   # both key-major passes in one launch
    f["fwd.ball_cmp"] = f["fwd.ball"] + f["fwd.cmp"]   # both forward passes in one launch
    return f


def phase_bytes(cfg, variant="bsa"):
    """Compulsory HBM bytes of each timed phase: every tensor the phase must read or write
    once (bf16 storage, float32 gradients and compressed-branch output, 16 bytes of packed
    row terms per query row and branch in the backward). Intermediate partial sums and the
    re-reads that tiling causes are not counted: they are what the counters measure on top.
    The selection phases count K and V once (every block is selected by some group)."""
    B, H, N, d = cfg.batch, cfg.heads, cfg.n_pad, cfg.head_dim
    l, ls, k, g = cfg.cmp_block, cfg.slc_block, cfg.topk, cfg.group
    e = 2 if cfg.dtype == "bf16" else 4
    R = B * H * N                 # token rows
    Rc = B * H * (N // l)         # compressed rows
    Rg = B * H * (N // g)         # query groups
    gc = variant == "group_cmp"
    Rq = Rc if gc else R          # query rows of the compressed branch
    x = R * d * e                 # one token tensor in the storage type
    xc = Rc * d * e
    sel = Rg * k * 4
    out = {
        "tree": B * N * (3 * 4 + 4),
        "permute": 3 * 2 * x + 2 * B * N * 3 * 4,
        "fwd.compress": (3 if gc else 2) * (x + Rc * d * (4 + 4 + e)),
        "fwd.select": x + 3 * 2 * Rc * d + sel,
        "fwd.ball": 4 * x + 4 * R,
        "fwd.cmp": Rq * d * e + 2 * xc + R * d * 4 + 4 * R,
        "fwd.slc": 4 * x + sel + 4 * R,
        "fwd.gate": 2 * x + R * d * 4 + x + B * N * 12,
        "bwd.gate": x + 2 * x + R * d * 4 + 4 * 3 * R + 3 * 16 * R,
        "bwd.kv_ball": 4 * x + 16 * R + 2 * R * d * 4,
        "bwd.dq_ball": 4 * x + 16 * R + R * d * 4,
        "bwd.kv_cmp": 2 * Rq * d * e + 2 * xc + 16 * Rq + 2 * Rc * d * 4,
        "bwd.dq_cmp": 2 * Rq * d * e + 2 * xc + 16 * Rq + 2 * Rq * d * 4,
        "bwd.dq_slc": 4 * x + sel + 16 * R + 2 * R * d * 4,
        "bwd.slc_kv": 4 * x + sel + 16 * R + 4 * R * d * 4,
        "bwd.slc_csr": 4 * sel,
        "bwd.mlp": (3 if gc else 2) * (2 * x + 2 * R * d * 4 + 3 * Rc * d * 4),
    }
    # the key-major passes in one launch: Q and dO once (unless the compressed pass reads
    # the coarse queries)
    out["bwd.kv"] = out["bwd.kv_ball"] + out["bwd.kv_cmp"] - (0 if gc else 2 * x)
    out["fwd.ball_cmp"] = out["fwd.ball"] + out["fwd.cmp"] - (0 if gc else x)
    return out


# the phases of each attention branch, forward and backward; where the ball and
# compressed key-major passes share one launch (phase bwd.kv) that launch is its own entry
# and the two branches' entries hold their forward and dQ phases
BRANCH_PHASES = {"ball": ("fwd.ball", "bwd.kv_ball", "bwd.dq_ball"),
                 "cmp": ("fwd.cmp", "bwd.kv_cmp", "bwd.dq_cmp"),
                 "ball_cmp_fwd": ("fwd.ball_cmp",),
                 "ball_cmp_kv": ("bwd.kv",),
                 "slc": ("fwd.slc", "bwd.slc_csr", "bwd.slc_kv", "bwd.dq_slc")}


def gathered_bytes(cfg):
    """Selection K/V bytes gathered per pass if no gather hits a cache: every group reads
    its k* blocks of l' keys and values."""
    B, H, N, d = cfg.batch, cfg.heads, cfg.n_pad, cfg.head_dim
    e = 2 if cfg.dtype == "bf16" else 4
    return B * H * (N // cfg.group) * cfg.topk * cfg.slc_block * d * e * 2


def rooflines(cfg, variant, ms):
    """Per phase and per branch: algorithmic TFLOP/s, fraction of the bf16 MFMA peak, and
    fraction of the attainable roofline min(peak, I * HBM) at the phase's compulsory
    intensity I (FLOP per byte)."""
    pf, pb = phase_flops(cfg, variant), phase_bytes(cfg, variant)
    out = {}
    for n, t in ms.items():
        if n not in pf or t <= 0:
            continue
        inten = pf[n] / pb[n]
        att = min(MFMA_BF16_PEAK, inten * HBM_PEAK)
        ach = pf[n] / (t * 1e-3)
        out[n] = {"tflops": round(ach / 1e12, 1), "frac_peak": round(ach / MFMA_BF16_PEAK, 4),
                  "flop_per_byte": round(inten, 1), "attainable_tflops": round(att / 1e12, 1),
                  "frac_attainable": round(ach / att, 4), "bound": "mfma" if att >= MFMA_BF16_PEAK else "hbm",
                  "hbm_gbps_compulsory": round(pb[n] / (t * 1e-3) / 1e9, 1)}
    branches = {}
    for br, names in BRANCH_PHASES.items():
        names = [n for n in names if ms.get(n, 0.0) > 0.0]   # phases that ran
        if not names:
            continue
        t = sum(ms[n] for n in names)
        f = sum(pf.get(n, 0.0) for n in names)
        byt = sum(pb[n] for n in names)
        att = min(MFMA_BF16_PEAK, f / byt * HBM_PEAK)
        ach = f / (t * 1e-3)
        branches[br] = {"ms": round(t, 4), "tflops": round(ach / 1e12, 1), "frac_peak": round(ach / MFMA_BF16_PEAK, 4),
                        "flop_per_byte": round(f / byt, 1), "attainable_tflops": round(att / 1e12, 1),
                        "frac_attainable": round(ach / att, 4)}
    if "slc" in branches and ms.get("fwd.slc", 0.0) > 0.0:
        # the selection's gathers: g FLOP per gathered byte if every gather came from HBM
        gb = gathered_bytes(cfg)
        fs = pf["fwd.slc"]
        branches["slc"]["fwd_gathered_gb"] = round(gb / 1e9, 2)
        branches["slc"]["fwd_gather_tbps"] = round(gb / (ms["fwd.slc"] * 1e-3) / 1e12, 2)
        branches["slc"]["fwd_attainable_tflops_hbm_gathers"] = round(fs / gb * HBM_PEAK / 1e12, 1)
    return out, branches


# single-launch phases whose work is a dense bf16 contraction (roofline candidates)
PHASES = ("tree", "permute", "fwd.compress", "fwd.select", "fwd.ball", "fwd.cmp", "fwd.ball_cmp", "fwd.slc", "fwd.gate",
          "bwd.gate", "bwd.dq_ball", "bwd.dq_cmp", "bwd.dq_slc", "bwd.kv_ball", "bwd.kv_cmp", "bwd.kv", "bwd.mlp",
          "bwd.slc_csr", "bwd.slc_kv")
PHASE_STEPS = 5   # steps of each phase-breakdown pass (run before the timed region)
FLUSH_BYTES = 512 << 20   # written before each cold step: twice the MALL
MFMA_PHASES = ("fwd.ball", "fwd.cmp", "fwd.ball_cmp", "fwd.slc", "bwd.dq_ball", "bwd.dq_cmp", "bwd.dq_slc", "bwd.kv_ball",
               "bwd.kv_cmp", "bwd.kv")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_{phase}_{workload}.txt")


def _sources_sha(files):
    import hashlib
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()


def measured_traffic(phase, workload):
    """HBM bytes per launch of `phase` from the committed counter summary, or None when
    there is none or the kernel's sources changed since the counters were taken."""
    path = TRAFFIC_FILE.format(phase=phase.replace(".", "_"), workload=workload)
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith((" ", "#")):
            key, val = line.split(":", 1)
            kv[key.strip()] = val.strip()
    try:
        if _sources_sha(kv["sources"].split()) != kv["sources_sha256"]:
            return None
        return float(kv["traffic_bytes_per_launch"])
    except (KeyError, OSError, ValueError):
        return None


COPY_BYTES = 1 << 30


def copy_calibration():
    """A plain device copy of known size (1 GiB read, 1 GiB written per launch), the
    yardstick for the FETCH_SIZE / WRITE_SIZE counters."""
    import torch
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(4):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": COPY_BYTES, "copy_bytes_written": COPY_BYTES, "launches": 4}))


def _pmc_per_dispatch(csv_path, counter, match):
    import csv
    tot, disp = 0.0, set()
    for r in csv.DictReader(open(csv_path)):
        if r["Counter_Name"] == counter and match(r["Kernel_Name"]):
            tot += float(r["Counter_Value"])
            disp.add(r["Dispatch_Id"])
    if not disp:
        raise SystemExit(f"{csv_path}: no dispatch of the kernel with counter {counter}")
    return tot / len(disp), len(disp)


def summarize_traffic(args):
    """Write the traffic summary of one phase's kernel from four rocprofv3 --pmc runs
    (FETCH_SIZE and WRITE_SIZE over the bench, then over --copy-calibration)."""
    fetch_csv, write_csv, cfetch_csv, cwrite_csv = args.summarize_traffic
    kernel, phase = args.kernel, args.phase
    from workloads import CONFIGS
    cfg = CONFIGS[args.config]
    short = lambda n: n.replace("(anonymous namespace)::", "").replace("void ", "").split("(")[0].split("::")[-1]
    is_kernel = lambda n: short(n) == kernel
    is_copy = lambda n: "copy" in n.lower()
    f_kib, nf = _pmc_per_dispatch(fetch_csv, "FETCH_SIZE", is_kernel)
    w_kib, nw = _pmc_per_dispatch(write_csv, "WRITE_SIZE", is_kernel)
    cf_kib, _ = _pmc_per_dispatch(cfetch_csv, "FETCH_SIZE", is_copy)
    cw_kib, _ = _pmc_per_dispatch(cwrite_csv, "WRITE_SIZE", is_copy)
    ff = COPY_BYTES / (cf_kib * 1024)
    fw = COPY_BYTES / (cw_kib * 1024)
    traffic = f_kib * 1024 * ff + w_kib * 1024 * fw
    srcs = args.sources.split()
    out = TRAFFIC_FILE.format(phase=phase.replace(".", "_"), workload=cfg.name)
    with open(out, "w") as fh:
        fh.write(f"# HBM traffic per launch of the {phase} kernel, workload {cfg.name}\n")
        fh.write("# Commands (repository root on the MI355X box, after cd /tmp && export TMPDIR=/tmp):\n")
        for c in args.commands:
            fh.write(f"#   {c}\n")
        fh.write("# FETCH_SIZE / WRITE_SIZE are KiB per dispatch; each is scaled by the ratio of the known\n"
                 "# bytes of a plain 1 GiB device copy to what the same counter reads for that copy.\n")
        fh.write(f"phase: {phase}\nworkload: {cfg.name}\nkernel: {kernel}\n")
        fh.write(f"dispatches: fetch {nf}, write {nw}\n")
        fh.write(f"fetch_kib_per_dispatch: {f_kib:.1f}\nwrite_kib_per_dispatch: {w_kib:.1f}\n")
        fh.write(f"copy_fetch_kib_per_dispatch: {cf_kib:.1f}\ncopy_write_kib_per_dispatch: {cw_kib:.1f}\n")
        fh.write(f"fetch_scale: {ff:.4f}\nwrite_scale: {fw:.4f}\n")
        fh.write(f"traffic_bytes_per_launch: {traffic:.0f}\n")
        fh.write(f"sources: {' '.join(srcs)}\nsources_sha256: {_sources_sha(srcs)}\n")
    print(open(out).read())


SQ_COUNTERS = ("SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_VALU_MFMA_BUSY_CYCLES", "SQ_BUSY_CU_CYCLES", "SQ_INSTS_VALU",
               "SQ_INSTS_MFMA", "SQ_INSTS_LDS", "SQ_WAIT_INST_ANY", "SQ_ACTIVE_INST_VALU", "GRBM_GUI_ACTIVE")
# second pass: instruction mix for the issue bound, and cycles where MFMA and VALU overlap
SQ_ISSUE_COUNTERS = ("SQ_INSTS_VALU_TRANS_F32", "SQ_VALU_MFMA_COEXEC_CYCLES", "SQ_VALU_MFMA_BUSY_CYCLES",
                     "SQ_INSTS_VALU", "SQ_INSTS_MFMA", "GRBM_GUI_ACTIVE")
N_CU = 256
N_XCD = 8


def _short_kernel(name):
    """Kernel name without namespaces, return type and argument list (template arguments kept)."""
    n = name.replace("(anonymous namespace)::", "").replace("bsa::", "")
    if n.startswith("void "):
        n = n[5:]
    depth = 0
    for i, ch in enumerate(n):
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0:
            return n[:i]
    return n


def _per_kernel(csv_path, counters):
    """{kernel: {counter: mean value per dispatch, "_n": dispatches}} from a rocprofv3 counter CSV."""
    import csv
    acc = {}
    for r in csv.DictReader(open(csv_path)):
        if r["Counter_Name"] not in counters:
            continue
        k = _short_kernel(r["Kernel_Name"])
        d = acc.setdefault(k, {})
        d.setdefault(r["Counter_Name"], {})[r["Dispatch_Id"]] = d.get(r["Counter_Name"], {}).get(
            r["Dispatch_Id"], 0.0) + float(r["Counter_Value"])
    out = {}
    for k, d in acc.items():
        out[k] = {c: sum(v.values()) / len(v) for c, v in d.items()}
        out[k]["_n"] = max(len(v) for v in d.values())
    return out


def summarize_counters(args):
    """Per-kernel table from one rocprofv3 kernel trace (durations) and counter runs:
    FETCH_SIZE, WRITE_SIZE (HBM bytes, scaled by a plain 1 GiB copy) and the SQ/GRBM
    instruction and MFMA counters."""
    import csv
    trace, fetch, write, sq, sq2, cfetch, cwrite = args.summarize_counters
    dur = {}
    for r in csv.DictReader(open(trace)):
        k = _short_kernel(r["Kernel_Name"])
        dur.setdefault(k, []).append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9)
    f = _per_kernel(fetch, ("FETCH_SIZE",))
    w = _per_kernel(write, ("WRITE_SIZE",))
    q = _per_kernel(sq, SQ_COUNTERS)
    q2 = _per_kernel(sq2, SQ_ISSUE_COUNTERS)
    is_copy = lambda n: "copy" in n.lower()
    cf = [v["FETCH_SIZE"] for k, v in _per_kernel(cfetch, ("FETCH_SIZE",)).items() if is_copy(k)]
    cw = [v["WRITE_SIZE"] for k, v in _per_kernel(cwrite, ("WRITE_SIZE",)).items() if is_copy(k)]
    ff, fw = COPY_BYTES / (cf[0] * 1024), COPY_BYTES / (cw[0] * 1024)
    total = sum(sum(v) for v in dur.values())
    rows = []
    for k, ds in sorted(dur.items(), key=lambda kv: -sum(kv[1])):
        t = sum(ds) / len(ds)
        if sum(ds) < 0.002 * total:
            continue
        fb = f.get(k, {}).get("FETCH_SIZE", float("nan")) * 1024 * ff
        wb = w.get(k, {}).get("WRITE_SIZE", float("nan")) * 1024 * fw
        c = q.get(k, {})
        c2 = q2.get(k, {})
        mops = c.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0)
        gui = c.get("GRBM_GUI_ACTIVE", float("nan"))
        clk = gui / N_XCD / t if gui == gui else float("nan")   # Hz
        # issue-serialized time: every MFMA (16x16x32 bf16: 16 cycles at the published 2.5
        # PFLOP/s), transcendental (a quarter of the fp32 rate: 8 cycles) and other VALU
        # instruction (wave64 at the fp32 rate of the published 157.3 TFLOP/s, 32 lanes per
        # SIMD: 2 cycles; a lower bound, some forms take longer) of the launch issued one
        # after another on the 1024 SIMDs, at the measured clock
        nm, ntr, nv = (c2.get(x, float("nan")) for x in ("SQ_INSTS_MFMA", "SQ_INSTS_VALU_TRANS_F32", "SQ_INSTS_VALU"))
        issue_s = (16 * nm + 8 * ntr + 2 * (nv - nm - ntr)) / (N_CU * 4) / clk
        busy2 = c2.get("SQ_VALU_MFMA_BUSY_CYCLES", float("nan"))
        rows.append({
            "kernel": k, "calls": len(ds), "avg_us": t * 1e6, "gpu_time_pct": 100 * sum(ds) / total,
            "fetch_mb": fb / 1e6, "write_mb": wb / 1e6, "hbm_gbps": (fb + wb) / t / 1e9,
            "mfma_tflops_executed": 512 * mops / t / 1e12,
            # GRBM_GUI_ACTIVE counts GPU-busy cycles summed over the 8 XCDs
            "mfma_busy_pct": 100 * c.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) / (gui / N_XCD * N_CU * 4) if gui == gui
            else float("nan"),
            "clock_ghz": gui / N_XCD / t / 1e9 if gui == gui else float("nan"),
            "valu_insts": c.get("SQ_INSTS_VALU", float("nan")), "mfma_insts": c.get("SQ_INSTS_MFMA", float("nan")),
            "trans_insts": ntr, "lds_insts": c.get("SQ_INSTS_LDS", float("nan")),
            "issue_bound_pct": 100 * issue_s / t,
            "coexec_pct": 100 * c2.get("SQ_VALU_MFMA_COEXEC_CYCLES", float("nan")) / busy2 if busy2 else float("nan"),
        })
    out = args.counters_out
    with open(out, "w") as fh:
        fh.write(f"# Per-kernel counters: {args.counters_title}\n\n")
        fh.write("Commands (repository root on the MI355X box, after `cd /tmp && export TMPDIR=/tmp`):\n\n")
        for cmd in args.commands:
            fh.write(f"    {cmd}\n")
        fh.write("\nDurations from the kernel trace (every kernel alone: the library on one stream). HBM bytes =\n"
                 "FETCH_SIZE and WRITE_SIZE (KiB per dispatch) scaled by what they read for a plain 1 GiB device\n"
                 f"copy (fetch x{ff:.3f}, write x{fw:.3f}). MFMA TFLOP/s executed = 512 x SQ_INSTS_VALU_MFMA_MOPS_BF16 /\n"
                 "duration (every MFMA FLOP issued, recomputation included). MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES /\n"
                 "(GRBM_GUI_ACTIVE / 8 XCDs x 256 CUs x 4 SIMDs); clock = GRBM_GUI_ACTIVE / 8 / duration. Instruction\n"
                 "counts are per dispatch (all waves). Kernels under 0.2% of GPU time are left out. GRBM_GUI_ACTIVE\n"
                 "spans the dispatch's whole busy window, which for a short kernel includes launch and drain time\n"
                 "outside its traced duration: clock and MFMA busy are meaningful for kernels of 100 us and more.\n"
                 "Issue bound = the time the launch's MFMA (16 cycles each, from the bf16 peak), transcendental\n"
                 "(8, a quarter of the fp32 rate) and other VALU instructions (2, the fp32 rate of the published\n"
                 "157.3 TFLOP/s; a lower bound; SQ_INSTS_VALU counts MFMA and transcendental instructions too)\n"
                 "take issued one after another on the 1024 SIMDs at the measured clock, over the duration: near\n"
                 "100 the kernel is bound by issue with MFMA and VALU work serialised, well below 100 it waits on\n"
                 "latency (LDS, memory, dependencies). Co-exec = SQ_VALU_MFMA_COEXEC_CYCLES /\n"
                 "SQ_VALU_MFMA_BUSY_CYCLES, the share of MFMA-busy cycles in which VALU work also ran (second\n"
                 "counter pass, with the transcendental count).\n\n")
        cols = ("kernel", "calls", "avg_us", "gpu_time_pct", "fetch_mb", "write_mb", "hbm_gbps",
                "mfma_tflops_executed", "mfma_busy_pct", "clock_ghz", "valu_insts", "mfma_insts", "trans_insts",
                "lds_insts", "issue_bound_pct", "coexec_pct")
        fh.write("| " + " | ".join(cols) + " |\n|" + "---|" * len(cols) + "\n")
        for r in rows:
            cells = []
            for c in cols:
                v = r[c]
                if isinstance(v, str):
                    cells.append(f"`{v}`")
                elif c in ("calls",):
                    cells.append(str(v))
                elif c.endswith("insts"):
                    cells.append(f"{v:.3g}")
                elif c == "clock_ghz":
                    cells.append(f"{v:.2f}")
                else:
                    cells.append(f"{v:.1f}")
            fh.write("| " + " | ".join(cells) + " |\n")
    print(open(out).read())


LDS_COUNTERS = ("SQ_INSTS_LDS", "SQ_LDS_IDX_ACTIVE", "SQ_LDS_BANK_CONFLICT", "SQ_LDS_ADDR_CONFLICT",
                "SQ_LDS_UNALIGNED_STALL", "SQ_WAIT_INST_LDS", "GRBM_GUI_ACTIVE")


def summarize_lds(args):
    """Per-kernel LDS bank-conflict table from one rocprofv3 --pmc run of LDS_COUNTERS."""
    (csv_path,) = args.summarize_lds
    q = _per_kernel(csv_path, LDS_COUNTERS)
    rows = sorted(((k, c) for k, c in q.items() if c.get("SQ_INSTS_LDS", 0) > 0),
                  key=lambda kc: -kc[1].get("SQ_LDS_IDX_ACTIVE", 0))
    with open(args.counters_out, "w") as fh:
        fh.write(f"# LDS bank conflicts per kernel: {args.counters_title}\n\n")
        fh.write("Commands (repository root on the MI355X box, after `cd /tmp && export TMPDIR=/tmp`):\n\n")
        for cmd in args.commands:
            fh.write(f"    {cmd}\n")
        fh.write("\nPer dispatch, summed over the chip: LDS instructions, LDS busy cycles (SQ_LDS_IDX_ACTIVE) and\n"
                 "the cycles of those lost to bank and address conflicts and unaligned accesses; conflict % =\n"
                 "SQ_LDS_BANK_CONFLICT / SQ_LDS_IDX_ACTIVE. Kernels without LDS instructions are left out.\n\n")
        fh.write("| kernel | dispatches | lds_insts | lds_active_cycles | bank_conflict_cycles | conflict_pct | "
                 "addr_conflict_cycles | unaligned_stall_cycles |\n|---|---|---|---|---|---|---|---|\n")
        for k, c in rows:
            act = c.get("SQ_LDS_IDX_ACTIVE", 0.0)
            bank = c.get("SQ_LDS_BANK_CONFLICT", 0.0)
            fh.write(f"| `{k}` | {c['_n']} | {c.get('SQ_INSTS_LDS', 0):.3g} | {act:.3g} | {bank:.3g} | "
                     f"{100 * bank / act if act else 0.0:.2f} | {c.get('SQ_LDS_ADDR_CONFLICT', 0):.3g} | "
                     f"{c.get('SQ_LDS_UNALIGNED_STALL', 0):.3g} |\n")
    print(open(args.counters_out).read())


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=3)
    ap.add_argument("--variant", choices=sorted(VARIANTS), default="bsa")
    ap.add_argument("--sweep", action="store_true",
                    help="sequence-length sweep: BSA layer vs full attention (one JSON line per length)")
    ap.add_argument("--model", action="store_true",
                    help="sequence-length sweep of the 18-block model (RMSNorm + BSA + SwiGLU), forward + backward, "
                         "BSA vs full attention (one JSON line per length)")
    ap.add_argument("--lengths", default="1024,2048,4096,8192,16384,32768,65536")
    ap.add_argument("--cpu-baseline", type=int, default=1, help="time the float64 oracle on a sample (0 = skip)")
    ap.add_argument("--rep-steps", type=int, default=100,
                    help="steps of the warm and of the cold median after the timed region (0 = skip)")
    ap.add_argument("--copy-calibration", action="store_true", help="run only the 1 GiB plain copy")
    ap.add_argument("--summarize-traffic", nargs=4, metavar="CSV",
                    help="counter CSVs: FETCH_SIZE bench, WRITE_SIZE bench, FETCH_SIZE copy, WRITE_SIZE copy")
    ap.add_argument("--phase", default="bwd.kv")
    ap.add_argument("--kernel", default="dense_bwd_kv_pair_kernel<64, false>")
    ap.add_argument("--sources", default="paper_2506_12541_amd/csrc/attn_bwd.hip paper_2506_12541_amd/csrc/attn_common.hpp "
                                         "paper_2506_12541_amd/csrc/common.hpp paper_2506_12541_amd/csrc/kernels.hpp "
                                         "paper_2506_12541_amd/build.py")
    ap.add_argument("--commands", nargs="*", default=[])
    ap.add_argument("--summarize-counters", nargs=7, metavar="CSV",
                    help="kernel trace, FETCH_SIZE, WRITE_SIZE, SQ and SQ issue counter CSVs of the bench, "
                         "FETCH_SIZE and WRITE_SIZE CSVs of --copy-calibration")
    ap.add_argument("--summarize-lds", nargs=1, metavar="CSV", help="LDS counter CSV of the bench (LDS_COUNTERS)")
    ap.add_argument("--counters-out", default=os.path.join(ROOT, "profiles", "counters.md"))
    ap.add_argument("--counters-title", default="")
    ap.add_argument("--streams", type=int, default=2,
                    help="library streams (1 = every kernel alone; 0 = also no shared launches)")
    ap.add_argument("--oracle-baselines", action="store_true",
                    help="time the float64 oracle in full on configs 1, 2, 3 and 5 (CPU only)")
    ap.add_argument("--forward-only", action="store_true",
                    help="time tree + permute + forward (e.g. --config 4, the 2^20-point workload)")
    return ap.parse_args()


def cpu_baseline(cfg, pts_np, inp_np, variant="bsa"):
    """The float64 oracle on a bounded sample of the same workload: the full ball tree
    plus one of the heads' forward and backward; the head time is scaled by the head
    count to give points/s for the whole step."""
    import numpy as np

    from oracle import bsa as ob
    from oracle.tree import build_ball_tree

    cores = len(os.sched_getaffinity(0))
    okw = {"q_coarsen": "mlp", "group_compression": True} if variant == "group_cmp" else {}
    P = ob.Params(ball=cfg.ball, cmp_block=cfg.cmp_block, slc_block=cfg.slc_block, topk=cfg.topk, group=cfg.group,
                  **okw)
    t0 = time.perf_counter()
    perm = build_ball_tree(pts_np[0], cfg.n_pad)
    t_tree = time.perf_counter() - t0
    h = 0
    sl = lambda a: np.ascontiguousarray(a[:, h:h + 1])
    valid = (perm >= 0)[None]
    q, k, v, do = (sl(inp_np[n]) for n in ("q", "k", "v", "do"))
    t0 = time.perf_counter()
    fwd = ob.forward(q, k, v, valid, inp_np["gate"], inp_np["phi_k"], inp_np["phi_v"], P, phi_q=inp_np["phi_q"])
    ob.backward(q, k, v, valid, inp_np["gate"], inp_np["phi_k"], inp_np["phi_v"], P, fwd, do, phi_q=inp_np["phi_q"])
    t_head = time.perf_counter() - t0
    total = t_tree + cfg.heads * t_head
    return {"value": cfg.batch * cfg.n_real / total, "unit": "points/s", "cores": cores, "kind": "oracle",
            "sample": f"ball tree of the full {cfg.n_real}-point cloud ({t_tree:.2f} s) + forward and backward of "
                      f"1 of {cfg.heads} heads ({t_head:.2f} s), scaled x{cfg.heads}; float64 numpy"}


def cpu_baseline_large(cfg, pts_np, hi, groups=32):
    """The float64 oracle's forward on a bounded sample of the 2^20-point workload: the full
    ball tree, then for one head the compression of every block (the part that does not
    shrink with the sample) and the three branches and the gate for `groups` sampled query
    groups; extrapolated linearly to every group and head (labelled as such)."""
    import numpy as np

    from oracle import bsa as ob
    from oracle.tree import build_ball_tree

    cores = len(os.sched_getaffinity(0))
    P = ob.Params(ball=cfg.ball, cmp_block=cfg.cmp_block, slc_block=cfg.slc_block, topk=cfg.topk, group=cfg.group)
    t0 = time.perf_counter()
    perm = build_ball_tree(pts_np[0], cfg.n_pad)
    t_tree = time.perf_counter() - t0
    valid = perm >= 0
    x = {n: a.astype(np.float64) for n, a in hi.head(0).items()}
    phk = {w: a.astype(np.float64) for w, a in hi.phi_k.items()}
    phv = {w: a.astype(np.float64) for w, a in hi.phi_v.items()}
    t0 = time.perf_counter()
    kc, _ = ob.compress(x["k"], valid, phk, P)
    vc, _ = ob.compress(x["v"], valid, phv, P)
    t_fixed = time.perf_counter() - t0
    ngroups = cfg.n_pad // cfg.group
    gs = np.random.default_rng(0).choice(ngroups, groups, replace=False)
    t0 = time.perf_counter()
    sel = ob.topk_blocks(ob.group_block_scores(x["q"], kc, valid, P, groups=gs), P.topk)
    full_sel = np.full((ngroups, P.topk), -1, np.int64)
    full_sel[gs] = sel
    rows = (gs[:, None] * cfg.group + np.arange(cfg.group)[None, :]).reshape(-1)
    for s0 in np.unique((rows // cfg.ball) * cfg.ball):
        sl = slice(s0, s0 + cfg.ball)
        ob.ball_branch(x["q"][sl], x["k"][sl], x["v"][sl], valid[sl], P)
    ob.compression_branch(x["q"], kc, vc, ob.block_valid(valid, cfg.cmp_block), valid, P, rows=rows)
    ob.selection_branch(x["q"], x["k"], x["v"], valid, full_sel, P, groups=gs)
    t_groups = time.perf_counter() - t0
    total = t_tree + cfg.heads * (t_fixed + t_groups * ngroups / groups)
    return {"value": cfg.batch * cfg.n_real / total, "unit": "points/s", "cores": cores, "kind": "oracle",
            "sample": f"ball tree of the full {cfg.n_real}-point cloud ({t_tree:.1f} s) + one head's compression of "
                      f"every block ({t_fixed:.1f} s) and forward of {groups} of {ngroups} query groups "
                      f"({t_groups:.1f} s); extrapolated x{ngroups // groups} groups, x{cfg.heads} heads; "
                      "forward only, float64 numpy"}


def oracle_baselines(args):
    """The float64 oracle timed in full on configs 1, 2, 3 and 5 (forward for 1 and 2,
    forward + backward for 3 and 5), tree included, on this host's cores; one JSON line each."""
    import numpy as np

    from oracle import bsa as ob
    from oracle.tree import build_ball_tree
    from workloads import CONFIGS, make_inputs, make_points

    cores = len(os.sched_getaffinity(0))
    for cid in (1, 2, 5, 3):
        cfg = CONFIGS[cid]
        pts = make_points(cfg)
        inp = make_inputs(cfg, layout="ball", with_grad=cfg.passes == "fwdbwd")
        P = ob.Params(ball=cfg.ball, cmp_block=cfg.cmp_block, slc_block=cfg.slc_block, topk=cfg.topk,
                      group=cfg.group)
        t0 = time.perf_counter()
        valid = np.stack([build_ball_tree(pts[b], cfg.n_pad) >= 0 for b in range(cfg.batch)])
        t_tree = time.perf_counter() - t0
        args_ = (inp["q"], inp["k"], inp["v"], valid, inp["gate"], inp["phi_k"], inp["phi_v"], P)
        t0 = time.perf_counter()
        fwd = ob.forward(*args_)
        t_fwd = time.perf_counter() - t0
        t_bwd = 0.0
        if cfg.passes == "fwdbwd":
            t0 = time.perf_counter()
            ob.backward(*args_, fwd, inp["do"])
            t_bwd = time.perf_counter() - t0
        total = t_tree + t_fwd + t_bwd
        print(json.dumps({"config": cid, "workload": cfg.name, "passes": cfg.passes, "cores": cores,
                          "tree_s": round(t_tree, 2), "forward_s": round(t_fwd, 2), "backward_s": round(t_bwd, 2),
                          "points_per_s": round(cfg.batch * cfg.n_real / total, 1), "kind": "oracle, float64 numpy"}),
              flush=True)


def sweep(args):
    """Layer runtime against sequence length, BSA vs full attention (the shape of the
    paper's Fig. 2, here for one layer rather than the 18-block model).

    Each length N runs the 65536-point workload's layer settings on one N-point Gaussian
    mixture cloud (H=8, d=64, bf16). BSA: forward + backward of the layer on rows already
    in ball order, timed with host clocks over the steps (both streams). Full attention:
    the same ball-attention kernels with one ball of N tokens (Eq. 3 with m = N is softmax
    attention over every key), forward + backward, taken from their phase events with the
    library on one stream so nothing overlaps them."""
    import numpy as np
    import torch

    from paper_2506_12541_amd import _lib
    from paper_2506_12541_amd import bsa as gb
    from workloads import Config, make_inputs

    lib = _lib.load()
    dev = torch.device("cuda:0")
    for n in (1024, 2048, 4096, 8192, 16384, 32768, 65536):
        cfg = Config(f"sweep_{n}", 1, n, n, 8, 64, "bf16", 256, 16, 16, 32, 16, 16, "gmm", "fwdbwd")
        inp = make_inputs(cfg, seed=3, layout="ball", with_grad=True)
        t = lambda a, d=torch.float32: torch.from_numpy(np.ascontiguousarray(a)).to(dev).to(d)
        q, k, v, do = (t(inp[x], torch.bfloat16) for x in ("q", "k", "v", "do"))
        gate = t(inp["gate"])
        phk = {w: t(a) for w, a in inp["phi_k"].items()}
        phv = {w: t(a) for w, a in inp["phi_v"].items()}

        def run(p, saved, steps):
            for _ in range(steps):
                o, sv = gb.forward(p, q, k, v, None, gate, phk, phv, saved=saved)
                gb.backward(p, q, k, v, None, gate, phk, phv, sv, do)

        p = gb.Params.from_config(cfg)
        saved = gb.Saved(p, dev)
        run(p, saved, 3)
        torch.cuda.synchronize()
        steps = max(5, min(50, (1 << 21) // n))
        t0 = time.perf_counter()
        run(p, saved, steps)
        torch.cuda.synchronize()
        bsa_ms = (time.perf_counter() - t0) / steps * 1e3

        pf = gb.Params.from_config(dataclasses.replace(cfg, ball=n))
        saved_f = gb.Saved(pf, dev)
        _lib.check(lib.bsa_set_streams(0), "streams")   # one stream, the ball kernels in launches of their own
        run(pf, saved_f, 2)
        torch.cuda.synchronize()
        fsteps = max(3, min(20, (1 << 19) // n))
        phases = ("fwd.ball", "bwd.dq_ball", "bwd.kv_ball")
        lib.bsa_timing_select(",".join(phases).encode())
        lib.bsa_timing_enable(1)
        run(pf, saved_f, fsteps)
        torch.cuda.synchronize()
        full_ms = 0.0
        for name in phases:
            tot, cnt = _lib.C.c_double(), _lib.C.c_int32()
            _lib.check(lib.bsa_timing_query(name.encode(), _lib.C.byref(tot), _lib.C.byref(cnt)), "timing")
            full_ms += tot.value / fsteps
        lib.bsa_timing_enable(0)
        lib.bsa_timing_select(None)
        _lib.check(lib.bsa_set_streams(2), "streams")
        fwd_f, bwd_f = algorithmic_flops(cfg)
        full_flop = 3.5 * 4.0 * n * n * cfg.head_dim * cfg.heads   # forward 4 N^2 d + backward 2.5x
        print(json.dumps({"n": n, "bsa_layer_ms": round(bsa_ms, 4), "full_attention_ms": round(full_ms, 4),
                          "full_over_bsa": round(full_ms / bsa_ms, 3),
                          "bsa_tflops": round((sum(fwd_f.values()) + sum(bwd_f.values())) / bsa_ms / 1e9, 1),
                          "full_tflops": round(full_flop / full_ms / 1e9, 1),
                          "workload": "1 cloud, H=8, d=64, bf16, ball 256, cmp 16, slc 32, top-16, group 16; "
                                      "forward + backward of the layer"}), flush=True)
        del saved, saved_f
        torch.cuda.empty_cache()


BLOCK_PHASES = ("blk.norm", "blk.gemm", "blk.wgrad", "blk.elem")
N_BLOCKS = 18   # the paper's model depth (Section 3.1)


def block_flops(n, C, F):
    """Channel-product FLOPs of one block per token count n: forward 2 n C (3C + C + 2F + F),
    backward twice that (activation and weight gradients)."""
    fwd = 2.0 * n * C * (3 * C + C + 2 * F + F)
    return fwd, 2.0 * fwd


def model_sweep(args):
    """Runtime of the 18-block model against sequence length, BSA vs full attention (the
    shape of the paper's Fig. 2).

    Each length N runs one N-point Gaussian-mixture cloud in ball order through 18 blocks
    (RMSNorm + BSA layer + SwiGLU, C = 512 = 8 heads x 64, F = 2048, bf16 products, the
    65536-point workload's layer settings), forward then backward, with per-block seeded
    weights; timed with host clocks over whole steps. The full-attention model is the same
    step with each block's BSA layer time replaced by that of softmax attention over every
    key (the ball kernels with one ball of N tokens, forward + backward, from their phase
    events on one stream): model_full = model_bsa - 18 layer_bsa + 18 layer_full, where
    layer_bsa is the measured forward + backward of one BSA layer on the same inputs."""
    import numpy as np
    import torch

    from paper_2506_12541_amd import _lib
    from paper_2506_12541_amd import bsa as gb
    from workloads import Config, make_block_inputs

    lib = _lib.load()
    dev = torch.device("cuda:0")
    for n in (int(v) for v in args.lengths.split(",")):
        cfg = Config(f"model_{n}", 1, n, n, 8, 64, "bf16", 256, 16, 16, 32, 16, 16, "gmm", "fwdbwd")
        C = cfg.heads * cfg.head_dim
        valid = np.ones((1, n), bool)
        p = gb.Params.from_config(cfg)
        blocks = []
        for i in range(N_BLOCKS):
            inp = make_block_inputs(cfg, valid, seed=1000 + i) if i == 0 or n <= 8192 else dict(blocks[0]["np"])
            t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
            blocks.append({"np": inp, "W": {k: t(a) for k, a in inp["W"].items()},
                           "phk": {w: t(a) for w, a in inp["phi_k"].items()},
                           "phv": {w: t(a) for w, a in inp["phi_v"].items()},
                           "saved": gb.BlockSaved(p, inp["ffn"], dev)})
        F = blocks[0]["np"]["ffn"]
        x0 = torch.from_numpy(blocks[0]["np"]["x"]).to(dev)
        dy0 = torch.from_numpy(blocks[0]["np"]["dy"]).to(dev)

        def step():
            xs = [x0]
            for b in blocks:
                y, _ = gb.block_forward(p, F, b["W"], b["phk"], b["phv"], xs[-1], saved=b["saved"])
                xs.append(y)
            g = dy0
            for i in reversed(range(N_BLOCKS)):
                b = blocks[i]
                g = gb.block_backward(p, F, b["W"], b["phk"], b["phv"], xs[i], b["saved"], g)["dx"]
            return g

        step()
        torch.cuda.synchronize()
        steps = max(2, min(10, (1 << 17) // n))
        t0 = time.perf_counter()
        for _ in range(steps):
            step()
        torch.cuda.synchronize()
        model_ms = (time.perf_counter() - t0) / steps * 1e3

        # one BSA layer forward + backward on the first block's Q/K/V (both streams)
        sv = blocks[0]["saved"]
        q, k, v, gate = sv.q.clone(), sv.k.clone(), sv.v.clone(), sv.gate.clone()
        do = torch.randn_like(q.float()).to(q.dtype)
        phk, phv = blocks[0]["phk"], blocks[0]["phv"]
        lsaved = gb.Saved(p, dev)

        def layer(pp, saved, reps):
            for _ in range(reps):
                o, s2 = gb.forward(pp, q, k, v, None, gate, phk, phv, saved=saved)
                gb.backward(pp, q, k, v, None, gate, phk, phv, s2, do)

        layer(p, lsaved, 2)
        torch.cuda.synchronize()
        reps = max(3, min(30, (1 << 19) // n))
        t0 = time.perf_counter()
        layer(p, lsaved, reps)
        torch.cuda.synchronize()
        bsa_layer_ms = (time.perf_counter() - t0) / reps * 1e3

        # full attention: the ball kernels with one ball of n tokens, one stream, in
        # launches of their own
        pf = gb.Params.from_config(dataclasses.replace(cfg, ball=n))
        fsaved = gb.Saved(pf, dev)
        _lib.check(lib.bsa_set_streams(0), "streams")
        layer(pf, fsaved, 1)
        torch.cuda.synchronize()
        fsteps = max(2, min(20, (1 << 19) // n))
        phases = ("fwd.ball", "bwd.dq_ball", "bwd.kv_ball")
        lib.bsa_timing_select(",".join(phases).encode())
        lib.bsa_timing_enable(1)
        layer(pf, fsaved, fsteps)
        torch.cuda.synchronize()
        full_layer_ms = 0.0
        for name in phases:
            tot, cnt = _lib.C.c_double(), _lib.C.c_int32()
            _lib.check(lib.bsa_timing_query(name.encode(), _lib.C.byref(tot), _lib.C.byref(cnt)), "timing")
            full_layer_ms += tot.value / fsteps
        # the block's own kernels, by phase (one stream, one model step)
        lib.bsa_timing_select(",".join(BLOCK_PHASES).encode())
        lib.bsa_timing_enable(1)
        step()
        torch.cuda.synchronize()
        blk = {}
        for name in BLOCK_PHASES:
            tot, cnt = _lib.C.c_double(), _lib.C.c_int32()
            _lib.check(lib.bsa_timing_query(name.encode(), _lib.C.byref(tot), _lib.C.byref(cnt)), "timing")
            blk[name] = round(tot.value / N_BLOCKS, 4)
        lib.bsa_timing_enable(0)
        lib.bsa_timing_select(None)
        _lib.check(lib.bsa_set_streams(2), "streams")
        full_model_ms = model_ms - N_BLOCKS * bsa_layer_ms + N_BLOCKS * full_layer_ms
        fwd_f, bwd_f = block_flops(n, C, F)
        gemm_ms = blk["blk.gemm"] + blk["blk.wgrad"]
        print(json.dumps({
            "n": n, "model_bsa_ms": round(model_ms, 3), "model_full_attention_ms": round(full_model_ms, 3),
            "full_over_bsa": round(full_model_ms / model_ms, 3), "bsa_layer_ms": round(bsa_layer_ms, 4),
            "full_attention_layer_ms": round(full_layer_ms, 4), "block_phases_ms": blk,
            "block_products_tflops": round((fwd_f + bwd_f) / (gemm_ms * 1e-3) / 1e12, 1) if gemm_ms > 0 else None,
            "workload": f"1 cloud of {n} points, 18 blocks (RMSNorm + BSA + SwiGLU), C=512 (8 heads x 64), F=2048, "
                        "bf16 products; layer: ball 256, cmp 16, slc 32, top-16, group 16; forward + backward"}),
              flush=True)
        del blocks, lsaved, fsaved
        torch.cuda.empty_cache()


def main():
    args = parse()
    if args.model:
        model_sweep(args)
        return
    if args.sweep:
        sweep(args)
        return
    if args.summarize_traffic:
        summarize_traffic(args)
        return
    if args.summarize_counters:
        summarize_counters(args)
        return
    if args.summarize_lds:
        summarize_lds(args)
        return
    if args.oracle_baselines:
        oracle_baselines(args)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}); the multi-GPU sharding is a design "
              "in DESIGN.md, not a measured path", file=sys.stderr)
        sys.exit(2)

    if args.copy_calibration:
        copy_calibration()
        return

    import numpy as np
    import torch

    from paper_2506_12541_amd import _lib
    from paper_2506_12541_amd import bsa as gb
    from workloads import CONFIGS, make_inputs, make_points

    cfg = CONFIGS[args.config]
    if args.variant == "g1":
        cfg = dataclasses.replace(cfg, group=1)
    dev = torch.device("cuda:0")
    pts_np = make_points(cfg)
    p = gb.Params.from_config(cfg, **VARIANTS[args.variant])
    dt = p.torch_dtype
    t = lambda a, d=None: torch.from_numpy(np.ascontiguousarray(a)).to(dev).to(d or torch.float32)
    H, d = cfg.heads, cfg.head_dim
    pts = t(pts_np)
    large = cfg.batch == 1 and cfg.n_real == cfg.n_pad and cfg.n_pad >= (1 << 20)
    if large:
        # 2^20 points x 16 heads: inputs drawn head by head into the per-point layout (every
        # slot is a real point, so a head's [n, d] draw serves as its per-point columns)
        from workloads import HeadInputs
        hi = HeadInputs(cfg)
        xq, xk, xv = (torch.empty((1, cfg.n_real, H * d), dtype=dt, device=dev) for _ in range(3))
        dout = None if args.forward_only else torch.empty((1, H, cfg.n_pad, d), dtype=dt, device=dev)
        names = ("q", "k", "v") if args.forward_only else ("q", "k", "v", "do")

        def put(h, x):
            for name, dst in (("q", xq), ("k", xk), ("v", xv)):
                dst[0, :, h * d:(h + 1) * d].copy_(t(x[name], dt))
            if dout is not None:
                dout[0, h].copy_(t(x["do"], dt))

        hi.heads(put, names)
        gate_pts = t(hi.gate)
        inp_np = {"phi_k": hi.phi_k, "phi_v": hi.phi_v, "phi_q": hi.phi_q}
    else:
        inp_np = make_inputs(cfg, layout="points", with_grad=False)
        inp_np["do"] = make_inputs(cfg, layout="ball", with_grad=True)["do"]
        xq, xk, xv = (t(inp_np[n], dt) for n in ("q", "k", "v"))
        gate_pts = t(inp_np["gate"])
        dout = t(inp_np["do"], dt)
    phi_k = {w: t(a) for w, a in inp_np["phi_k"].items()}
    phi_v = {w: t(a) for w, a in inp_np["phi_v"].items()}
    phi_q = {w: t(a) for w, a in inp_np["phi_q"].items()}
    saved = gb.Saved(p, dev)

    def step():
        perm = gb.build_ball_tree(pts, cfg.n_pad)
        q, valid = gb.permute(xq, perm, H, d, with_valid=True)
        k = gb.permute(xk, perm, H, d)
        v = gb.permute(xv, perm, H, d)
        gate = gb.permute(gate_pts, perm, 1, 3).view(cfg.batch, cfg.n_pad, 3)
        # every slot holds a real point when n_real == n_pad: the layer may skip key masks
        vmask = None if cfg.n_real == cfg.n_pad else valid
        o, sv = gb.forward(p, q, k, v, vmask, gate, phi_k, phi_v, saved=saved, phi_q=phi_q)
        if args.forward_only:
            return o, None
        grads = gb.backward(p, q, k, v, vmask, gate, phi_k, phi_v, sv, dout, phi_q=phi_q)
        return o, grads

    lib = _lib.load()
    _lib.check(lib.bsa_set_streams(args.streams), "streams")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    def phase_ms(names, steps):
        out = {}
        for name in names:
            tot = _lib.C.c_double()
            cnt = _lib.C.c_int32()
            _lib.check(lib.bsa_timing_query(name.encode(), _lib.C.byref(tot), _lib.C.byref(cnt)), "timing")
            out[name] = tot.value / max(1, steps)
        return out

    # phase passes (not the timed region): every phase records a pair of events, which
    # itself adds a little time, so the breakdowns are taken on steps of their own: first
    # as the step runs (two streams; phases that overlap share the chip), then with every
    # kernel alone (one stream), which gives each phase's own roofline
    lib.bsa_timing_select(None)
    lib.bsa_timing_enable(1)
    for _ in range(PHASE_STEPS):
        step()
    torch.cuda.synchronize()
    phases = phase_ms(PHASES, PHASE_STEPS)
    lib.bsa_timing_enable(0)
    _lib.check(lib.bsa_set_streams(1), "streams")
    lib.bsa_timing_enable(1)
    for _ in range(PHASE_STEPS):
        step()
    torch.cuda.synchronize()
    alone = phase_ms(PHASES, PHASE_STEPS)
    lib.bsa_timing_enable(0)
    # and every branch in launches of its own (streams mode 0: the shared launches split),
    # for the per-branch rooflines
    _lib.check(lib.bsa_set_streams(0), "streams")
    lib.bsa_timing_enable(1)
    for _ in range(PHASE_STEPS):
        step()
    torch.cuda.synchronize()
    separate = phase_ms(PHASES, PHASE_STEPS)
    lib.bsa_timing_enable(0)
    _lib.check(lib.bsa_set_streams(args.streams), "streams")
    for _ in range(2):
        step()
    torch.cuda.synchronize()
    # dominant kernel: the bf16 contraction phase with the longest time of its own
    dom = max(MFMA_PHASES, key=lambda n: alone[n])

    # timed region: exactly `steps` steps; only the dominant kernel's phase records events
    # (its live duration), plus one event per step on the caller's stream (the step's own
    # work ends there: the library joins its second stream back into it)
    lib.bsa_timing_select(dom.encode())
    lib.bsa_timing_enable(1)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev[0].record()
    for i in range(args.steps):
        step()
        ev[i + 1].record()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    dom_ms = phase_ms([dom], args.steps)[dom]
    lib.bsa_timing_enable(0)
    lib.bsa_timing_select(None)
    step_ms = sorted(ev[i].elapsed_time(ev[i + 1]) for i in range(args.steps))
    median_ms = step_ms[len(step_ms) // 2] if len(step_ms) % 2 else 0.5 * (step_ms[len(step_ms) // 2 - 1] +
                                                                            step_ms[len(step_ms) // 2])

    # warm and cold medians (after the timed region; not part of `value`): warm = steps back
    # to back; cold = a 512 MiB write before each step evicts the 256 MB MALL and the L2s
    def median_of(flush, n):
        flush_buf = torch.empty(FLUSH_BYTES // 4, dtype=torch.float32, device=dev) if flush else None
        times = []
        a_ev = [torch.cuda.Event(enable_timing=True) for _ in range(n)]
        b_ev = [torch.cuda.Event(enable_timing=True) for _ in range(n)]
        for i in range(n):
            if flush:
                flush_buf.fill_(float(i))
            a_ev[i].record()
            step()
            b_ev[i].record()
        torch.cuda.synchronize()
        times = sorted(a_ev[i].elapsed_time(b_ev[i]) for i in range(n))
        return times[n // 2]

    warm_ms = median_of(False, args.rep_steps) if args.rep_steps else None
    cold_ms = median_of(True, args.rep_steps) if args.rep_steps else None

    ms = elapsed / args.steps * 1e3
    fwd_f, bwd_f = algorithmic_flops(cfg, args.variant)
    flops = sum(fwd_f.values()) + (0.0 if args.forward_only else sum(bwd_f.values()))
    # the layer runs independent branches concurrently on two streams, so its time is the
    # step's wall time less the serial tree and permutation phases, not the sum of phases
    layer_ms = ms - phases["tree"] - phases["permute"]
    tflops = flops / (layer_ms * 1e-3) / 1e12
    pf = phase_flops(cfg, args.variant)
    achieved = pf[dom] / (dom_ms * 1e-3) / 1e12
    wl = cfg.name if args.variant == "bsa" else f"{args.variant}_{cfg.name}"
    traffic = measured_traffic(dom, wl)
    # per phase and branch from the separate launches; the shared launches from the pass
    # that runs them (their own entries)
    roof_ms = dict(separate)
    for n in ("fwd.ball_cmp", "bwd.kv"):
        roof_ms[n] = alone.get(n, 0.0)
    phase_roof, branch_roof = rooflines(cfg, args.variant, roof_ms)
    result = {
        "metric": ("BSA layer forward points/sec and TFLOP/s (fraction of MFMA peak) at "
                   f"N={cfg.n_pad}, 1 GPU" if args.forward_only else
                   "BSA layer fwd+bwd points/sec and TFLOP/s (fraction of MFMA peak) at N=65536, 1 GPU"),
        "value": cfg.batch * cfg.n_real / (ms * 1e-3),
        "unit": "points/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {cfg.batch}x{cfg.n_real} points (32-component Gaussian mixture), "
                               f"H={cfg.heads} d={cfg.head_dim}, ball {cfg.ball}, cmp block {cfg.cmp_block}, "
                               f"slc block {cfg.slc_block}, top-{cfg.topk}, group {cfg.group}"
                               + {"bsa": "", "group_cmp": "; MLP query coarsening (Eq. 13-14) + group compression "
                                                          "(Eq. 15)",
                                  "g1": "; per-token selection (Eq. 6-8, no grouping)"}[args.variant]
                               + ("; tree + permute + forward" if args.forward_only else
                                  "; tree + permute + forward + backward"),
                   "variant": args.variant,
                   "points": cfg.batch * cfg.n_real, "heads": cfg.heads, "head_dim": cfg.head_dim},
        "ms_per_step_median": round(median_ms, 4),
        "timing": {"warm_median_ms": None if warm_ms is None else round(warm_ms, 4),
                   "cold_median_ms": None if cold_ms is None else round(cold_ms, 4),
                   "steps_each": args.rep_steps, "cold_flush_bytes": FLUSH_BYTES,
                   "note": "medians of per-step HIP events after the timed region; cold = a 512 MiB device "
                           "write before each step"},
        "tflops": tflops,
        "mfma_frac": tflops * 1e12 / MFMA_BF16_PEAK,
        "algorithmic_gflop_per_step": flops / 1e9,
        "phase_ms": {n: round(v, 4) for n, v in phases.items()},
        "phase_ms_steps": PHASE_STEPS,
        # these phases run on the library's second stream beside others, so their
        # durations include time shared with the concurrent branch
        "concurrent_phases": concurrent_phases(phases),
        "phase_ms_alone": {n: round(v, 4) for n, v in alone.items()},
        # one stream and no shared launches: each branch's own phases (the rooflines below)
        "phase_ms_separate": {n: round(v, 4) for n, v in separate.items()},
        "phase_roofline": phase_roof,
        "branch_roofline": branch_roof,
        "roofline": {"bound": "mfma", "kernel": dom, "achieved": achieved, "peak": MFMA_BF16_PEAK / 1e12,
                     "unit": "TFLOP/s", "frac": achieved * 1e12 / MFMA_BF16_PEAK, "traffic": traffic,
                     "launch_ms": dom_ms, "launch_ms_alone": round(alone[dom], 4),
                     "algorithmic_gflop_per_launch": pf[dom] / 1e9},
    }
    if args.cpu_baseline and large:
        result["cpu_baseline"] = cpu_baseline_large(cfg, pts_np, hi)
    elif args.cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(cfg, pts_np, {**inp_np, **make_inputs(cfg, layout="ball",
                                                                                     with_grad=True)},
                                              args.variant)
    print(json.dumps(result))


if __name__ == "__main__":
    main()
