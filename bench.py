"""Benchmark of the replicated-encoder step on one MI355X.

One step = one pass of the whole hot path over one synthetic micro-batch of the
Qwen2-VL-ViT-shaped workload (24 images, sides log-uniform in [224, 1344]):
trained forward with tape -> merge scatter into the LLM input buffer -> merge
gather of the upstream gradient -> backward with fp32 weight-gradient
accumulation.  Inputs are resident in HBM before the timed region.

Prints one JSON line (rank 0).  See the design doc for the FLOP model, the roofline
figures and the CPU-baseline sample."""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6     # MI355X dense bf16 MFMA (256 CU x 4096 FLOP/clk x 2.4 GHz)
PEAK_F32_TFLOPS = 157.3
PEAK_HBM_GBPS = 8000.0
METRIC = "encoder patch-tokens/sec fwd+bwd on 1 MI355X; % bf16 MFMA peak"


def log(msg: str):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def model_flops(cfg, n_patches: int, sum_len2: int, trainable: int) -> float:
    """Algorithmic FLOPs of one step (recompute and padding excluded).

    forward F = 2 N Kpe h + L (8 N h^2 + 4 N h m + 4 h sum_i L_i^2) + 8 N h^2 + 2 N h H;
    trained (mode 1) = 3 F minus the patch-gradient GEMM (2 N Kpe h), which the trainable
    source does not compute (nothing is sent upstream); only the merger trainable
    (mode 2) = F plus the merger's input and weight gradients, 2 (8 N h^2 + 2 N h H);
    frozen = F."""
    N, h, m, H, L = n_patches, cfg.hidden, cfg.mlp, cfg.llm_hidden, cfg.layers
    kpe = cfg.k_pe
    merger = 8 * N * h * h + 2 * N * h * H
    F = (2 * N * kpe * h + L * (8 * N * h * h + 4 * N * h * m + 4 * h * sum_len2) + merger)
    if int(trainable) == 2:
        return float(F + 2 * merger)
    return float(3 * F - 2 * N * kpe * h) if trainable else float(F)


def hardware_flops(cfg, n_patches: int, sum_len2: int, trainable: bool) -> float:
    """MFMA work the kernels actually issue: the model FLOPs plus the attention backward's
    recompute (the dQ kernel recomputes S and dP, the dK/dV kernel S: 6 h d sum L^2 per
    layer), the head-dim padding of the products over d (d rounded up to 32 for S and
    dP: one in the forward, four in the backward) and the forward's row sums of P, taken
    by MFMAs with a ones operand (32 FLOP per query-key pair and head).  Ragged tile edges
    are not counted (the issued-FLOP counter in profiles/ measures them: about 1 % more)."""
    h, d, L = cfg.hidden, cfg.hidden // cfg.heads, cfg.layers
    dpad = (d + 31) // 32 * 32
    extra = 2.0 * h * sum_len2 * (dpad - d) / d      # one S-type product, padding only
    extra += 32.0 * (h // d) * sum_len2              # forward row sums of P
    per_layer = extra
    if int(trainable) == 1:
        per_layer += 6.0 * h * sum_len2 + 4 * (2.0 * h * sum_len2 * dpad / d)
        per_layer -= 4 * (2.0 * h * sum_len2)        # those four products' unpadded share
    return model_flops(cfg, n_patches, sum_len2, trainable) + L * per_layer


# ---- HBM traffic of the dominant kernel (rocprofv3 PMC counters) ---------------------
# FETCH_SIZE / WRITE_SIZE are read in two separate `rocprofv3 --pmc` runs of this script
# (one counter per run), each scaled by what the same counter reads for a plain copy of
# known size: the library's row gather with identity indices (--copy-calibration).
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic.json")
CAL_ROWS, CAL_COLS = 32768, 3584          # bf16 rows copied by the calibration gather
CAL_READ = CAL_ROWS * CAL_COLS * 2 + 8 * CAL_ROWS
CAL_WRITE = CAL_ROWS * CAL_COLS * 2
EPI_NAMES = ["store", "gelu", "resid", "gelubwd", "f32", "storerope"]
# What `traffic` counts: the TCC (L2) FETCH_SIZE + WRITE_SIZE counters, i.e. bytes moved
# between the L2 and the data fabric.  Reads served by the 256 MB Infinity Cache are
# included, so this bounds HBM traffic from above; it is per launch, like `achieved`.
TRAFFIC_NOTE = ("L2<->fabric bytes per launch (TCC FETCH_SIZE + WRITE_SIZE, scaled by a "
                "known-size copy; includes Infinity-Cache hits, so an upper bound on HBM bytes)")


def source_digest() -> str:
    """Digest of the kernel sources and the host code that launches them: stored traffic is
    reported only while it matches.  The host-only scheduling sources (owner map, schedule
    algebra) launch nothing and are left out."""
    import hashlib
    h = hashlib.sha256()
    src = os.path.join(ROOT, "paper_2607_03229_amd", "csrc")
    host_only = {"owner.cpp", "derive.cpp"}
    for f in sorted(os.listdir(src)):
        if f.endswith((".hip", ".cpp", ".h")) and f not in host_only:
            h.update(f.encode())
            with open(os.path.join(src, f), "rb") as fh:
                h.update(fh.read())
    return h.hexdigest()[:16]


def kernel_class(name: str):
    """Library profiling class of a dispatched kernel symbol (mangled or demangled)."""
    import re
    lay = {(0, 0): "NT", (0, 1): "NN", (1, 1): "TN"}
    m = re.search(r"gemm_big_kernel<(true|false), (true|false), (\d)>", name)
    if m:
        return f"gemm_{lay[(int(m.group(1) == 'true'), int(m.group(2) == 'true'))]}_{EPI_NAMES[int(m.group(3))]}"
    m = re.search(r"gemm_nn_kernel(?:<|ILi)(\d)", name)
    if m:
        return f"gemm_NN_{EPI_NAMES[int(m.group(1))]}"
    m = re.search(r"gemm_(?:big_)?kernelI(?:DF16b|f)?Lb([01])ELb([01])ELi(\d)E", name)
    if m:
        return f"gemm_{lay[(int(m.group(1)), int(m.group(2)))]}_{EPI_NAMES[int(m.group(3))]}"
    for key, cls in (("attn_fwd_kernel", "attn_fwd"), ("attn_bwd_dq_kernel", "attn_bwd_dq"),
                     ("attn_bwd_dkdv_kernel", "attn_bwd_dkdv"), ("rows_copy_kernel", "rows_copy")):
        if key in name:
            return cls
    return None


def _pmc_by_dispatch(db: str, counter: str):
    import sqlite3
    c = sqlite3.connect(db)
    out = {}
    for name, disp, cn, cv in c.execute(
            "select name, dispatch_id, counter_name, counter_value from pmc_events"):
        if cn != counter:
            continue
        key = (disp, name)
        out[key] = out.get(key, 0.0) + float(cv)
    return out


def summarize_pmc(fetch_cal: str, write_cal: str, fetch_db: str, write_db: str, cmds: str):
    """Scale the counters by the calibration copy and store bytes per dispatch per class."""
    def cal(db, counter, known):
        vals = [v for (d, n), v in _pmc_by_dispatch(db, counter).items() if kernel_class(n) == "rows_copy"]
        if not vals:
            raise SystemExit(f"no calibration copy dispatch in {db}")
        kib = sorted(vals)[len(vals) // 2]
        return known / (kib * 1024.0), kib
    ff, fk = cal(fetch_cal, "FETCH_SIZE", CAL_READ)
    fw, wk = cal(write_cal, "WRITE_SIZE", CAL_WRITE)
    per = {}
    for counter, db, fac in (("FETCH_SIZE", fetch_db, ff), ("WRITE_SIZE", write_db, fw)):
        for (d, n), kib in _pmc_by_dispatch(db, counter).items():
            cls = kernel_class(n)
            if cls is None or cls == "rows_copy":
                continue
            e = per.setdefault(cls, {"FETCH_SIZE": [0.0, 0], "WRITE_SIZE": [0.0, 0]})
            e[counter][0] += kib * 1024.0 * fac
            e[counter][1] += 1
    table = {}
    for cls, e in per.items():
        f, nf = e["FETCH_SIZE"]
        w, nw = e["WRITE_SIZE"]
        if nf and nw:
            table[cls] = {"fetch_bytes": round(f / nf), "write_bytes": round(w / nw),
                          "bytes": round(f / nf + w / nw), "dispatches": nf}
    rec = {"digest": source_digest(), "calibration": {
               "copy_read_bytes": CAL_READ, "copy_write_bytes": CAL_WRITE,
               "fetch_kib": fk, "write_kib": wk, "fetch_scale": ff, "write_scale": fw},
           "per_launch": table, "commands": cmds}
    with open(TRAFFIC_FILE, "w") as fh:
        json.dump(rec, fh, indent=1)
    print(json.dumps(rec, indent=1))


def summarize_mfma_flops(db: str, out: str, cmds: str, workload: str = "c4_qwen2vl_trained",
                         seed: int = 0):
    """One rocprofv3 --pmc pass of SQ_INSTS_VALU_MFMA_MOPS_BF16 over one bench step: the bf16
    MFMA FLOPs the kernels issued (the counter counts multiply-add operations / 512), per
    kernel class and in total, against the analytic model and hardware FLOPs."""
    import workload as W
    wl = W.make_workload(workload, seed)
    n, s2 = wl.n_patches, int(np.sum(np.diff(wl.cu_seqlens).astype(np.int64) ** 2))
    mf = model_flops(wl.cfg, n, s2, wl.trainable)
    hw = hardware_flops(wl.cfg, n, s2, wl.trainable)
    per = {}
    for (d, name), v in _pmc_by_dispatch(db, "SQ_INSTS_VALU_MFMA_MOPS_BF16").items():
        cls = kernel_class(name) or name.split("(")[0][-48:]
        e = per.setdefault(cls, [0, 0.0])
        e[0] += 1
        e[1] += v * 512.0
    total = sum(v for _, v in per.values())
    lines = [
        f"# bf16 MFMA FLOPs issued in one training step ({workload}, seed {seed})", "",
        "One `rocprofv3 --pmc` pass of one bench step; `SQ_INSTS_VALU_MFMA_MOPS_BF16` counts the "
        "MFMA multiply-add operations / 512 (the profiler's own `MfmaFlopsBF16` = counter x 512). "
        "Commands (on the MI355X box):", "", "```", cmds.strip(), "```", "",
        f"Measured: **{total / 1e12:.3f} TFLOP** per step.  Model FLOPs (bench.py `model_flops`): "
        f"{mf / 1e12:.3f} TFLOP; hardware model (`hardware_flops`: plus the attention backward's "
        f"recompute, the head-dim padding and the forward's row-sum MFMAs): {hw / 1e12:.3f} TFLOP "
        f"(measured / hardware model = {total / hw:.4f}).", "",
        "| kernel class | dispatches | TFLOP per step | share |", "|---|---:|---:|---:|"]
    for cls, (nd, v) in sorted(per.items(), key=lambda kv: -kv[1][1]):
        if v <= 0:
            continue
        lines.append(f"| `{cls}` | {nd} | {v / 1e12:.3f} | {100 * v / total:.1f} % |")
    with open(out, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print(f"wrote {out}: measured {total / 1e12:.3f} TFLOP, hardware model {hw / 1e12:.3f}")


def summarize_traffic_md(out: str, workload: str = "c4_qwen2vl_trained", seed: int = 0):
    """profiles/hbm_traffic.json (written by --summarize-pmc) -> its markdown table."""
    with open(TRAFFIC_FILE) as fh:
        rec = json.load(fh)
    c = rec["calibration"]
    rows = sorted(rec["per_launch"].items(), key=lambda kv: -kv[1]["bytes"])
    lines = [
        f"# L2<->fabric traffic per launch: encoder training step ({workload}, seed {seed})", "",
        "Two `rocprofv3 --pmc` runs of one bench step (FETCH_SIZE, then WRITE_SIZE), each scaled "
        "by what the same counter reads for a plain copy of known size: the library's row gather "
        "with identity indices, 32768 rows x 3584 bf16 (`bench.py --copy-calibration`).  The TCC "
        "counters count bytes between the L2 and the data fabric, including reads the 256 MB "
        "Infinity Cache serves, so they bound HBM traffic from above.", "",
        "Commands (on the MI355X box; this table: `python3 bench.py --summarize-traffic-md "
        f"{out}`):", "", "```", rec.get("commands", "").strip(), "```", "",
        f"Calibration: the copy reads {c['copy_read_bytes']:,} B and writes "
        f"{c['copy_write_bytes']:,} B; FETCH_SIZE read {c['fetch_kib']:,.0f} KiB (scale "
        f"{c['fetch_scale']:.3f}), WRITE_SIZE {c['write_kib']:,.0f} KiB (scale {c['write_scale']:.3f}).",
        "", f"Source digest of the kernels measured: `{rec['digest']}` (bench.py reports the traffic "
        "only while the tree's kernel sources hash to it).", "",
        "| kernel class | dispatches | fetch MB/launch | write MB/launch | total MB/launch |",
        "|---|---:|---:|---:|---:|"]
    for k, v in rows:
        lines.append(f"| `{k}` | {v['dispatches']} | {v['fetch_bytes'] / 1e6:,.1f} | "
                     f"{v['write_bytes'] / 1e6:,.1f} | {v['bytes'] / 1e6:,.1f} |")
    with open(out, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print(f"wrote {out}")


# ---- rocprofv3 summaries kept under profiles/ ---------------------------------------
SQ_PASS1 = ("SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_MFMA SQ_INSTS_VALU SQ_ACTIVE_INST_VALU "
            "SQ_LDS_BANK_CONFLICT SQ_ACTIVE_INST_LDS SQ_WAVE_CYCLES SQ_WAIT_ANY GRBM_GUI_ACTIVE")
SQ_PASS2 = ("SQ_VALU_MFMA_COEXEC_CYCLES SQ_INSTS_LDS SQ_WAIT_INST_LDS SQ_INSTS_VALU_TRANS_F32 "
            "SQ_INSTS_SALU GRBM_GUI_ACTIVE")
N_XCD, N_CU, N_SIMD = 8, 256, 1024


def summarize_trace(db: str, bench_json: str, cmds: str, out: str):
    """rocprofv3 --kernel-trace --stats database -> markdown table of the top kernels, with
    the library's class of each and the bench line of the same run."""
    import sqlite3
    c = sqlite3.connect(db)
    rows = list(c.execute("select name, total_calls, total_duration, average, percentage "
                          "from top_kernels order by total_duration desc"))
    r = json.loads(open(bench_json).read().strip().splitlines()[-1])
    L = [f"# Kernel trace: encoder training step, {r['config']['workload']} (seed {r['config']['seed']})",
         "", "Command (on the MI355X box):", "", "```", cmds, "```", "",
         "| kernel [library class] | calls | total ms | avg us | % of kernel time |",
         "|---|---:|---:|---:|---:|"]
    for name, n, tot, avg, pct in rows[:28]:
        cls = kernel_class(name)
        short = name if len(name) < 90 else name[:87] + "..."
        L.append(f"| `{short}`{' [' + cls + ']' if cls else ''} | {n} | {tot / 1e3:.1f} | "
                 f"{avg:.1f} | {pct:.1f} |")
    L += ["", f"Bench line of the same run: {r['ms_per_step']} ms/step, {r['value']:,} patch-tokens/s, "
              f"{r['model_tflop_per_step']} model TFLOP/step = {r['achieved_tflops']} TFLOP/s = "
              f"{r['mfma_pct_of_peak']} % of the {PEAK_BF16_TFLOPS} TFLOP/s bf16 dense peak "
              f"(hardware FLOPs: {r['hw_mfma_pct_of_peak']} %)."]
    for key in ("roofline", "roofline_largest_class"):
        roof = r.get(key)
        if not roof:
            continue
        tr = [x for x in rows if kernel_class(x[0]) == roof["kernel"]]
        if tr:
            n = sum(x[1] for x in tr)
            tot = sum(x[2] for x in tr)
            L.append(f"`{key}` class `{roof['kernel']}` ({roof['stream']} stream): the library's "
                     f"HIP events give avg {roof['avg_ms'] * 1e3:.1f} us over {roof['launches']} "
                     f"launches; the trace gives avg {tot / n:.1f} us over {n} dispatches "
                     f"(the trace also covers the warmup step and the per-kernel pass).")
    open(out, "w").write("\n".join(L) + "\n")
    print("\n".join(L))


def summarize_sq(db1: str, db2: str, cmds: str, out: str):
    """Two rocprofv3 --pmc passes of SQ counters over one step -> per kernel class averages
    and the derived per-SIMD / per-CU fractions (formulas in the table header)."""
    per = {}
    for db, names in ((db1, SQ_PASS1.split()), (db2, SQ_PASS2.split())):
        for counter in names:
            vals = _pmc_by_dispatch(db, counter)
            for (d, n), v in vals.items():
                cls = kernel_class(n) or ("layernorm_bwd" if "ln_bwd_kernel" in n else
                                          "layernorm" if "ln_fwd_kernel" in n else None)
                if cls is None:
                    continue
                e = per.setdefault(cls, {}).setdefault(counter, {})
                e[(db, d)] = v
    L = [f"# SQ counters per kernel class: encoder training step (c4_qwen2vl_trained, seed 0)", "",
         "Two `rocprofv3 --pmc` passes of one bench step (kernels are serialized while counters",
         "are taken, so these are each kernel's own figures, without the side-stream overlap).",
         "Commands (on the MI355X box):", "", "```", cmds, "```", "",
         f"Per dispatch: `cyc` = GRBM_GUI_ACTIVE / {N_XCD} (GPU-active cycles of one XCD); "
         f"MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (cyc x {N_SIMD} SIMDs); MFMA+VALU co-issue = "
         f"SQ_VALU_MFMA_COEXEC_CYCLES / (cyc x {N_SIMD}); VALU active = 4 SQ_ACTIVE_INST_VALU / "
         f"(cyc x {N_SIMD}); LDS bank-conflict = SQ_LDS_BANK_CONFLICT / (cyc x {N_CU} CUs); "
         "waiting = SQ_WAIT_ANY / SQ_WAVE_CYCLES; waves/SIMD = 4 SQ_WAVE_CYCLES / "
         f"(cyc x {N_SIMD}).  Instruction counts are per SIMD per dispatch.", "",
         "| class | dispatches | MFMA busy | co-issue | VALU active | LDS bank-conflict | waiting "
         "| waves/SIMD | MFMA inst | VALU inst | trans inst | LDS inst |",
         "|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|"]

    def avg(e, c):
        v = list(e.get(c, {}).values())
        return sum(v) / len(v) if v else float("nan")

    rows = []
    for cls, e in per.items():
        cyc = avg(e, "GRBM_GUI_ACTIVE") / N_XCD
        if not cyc or cyc != cyc:
            continue
        nd = len(e.get("SQ_INSTS_MFMA", {}))
        rows.append((avg(e, "SQ_VALU_MFMA_BUSY_CYCLES") * nd, cls, [
            nd, avg(e, "SQ_VALU_MFMA_BUSY_CYCLES") / (cyc * N_SIMD),
            avg(e, "SQ_VALU_MFMA_COEXEC_CYCLES") / (cyc * N_SIMD),
            4 * avg(e, "SQ_ACTIVE_INST_VALU") / (cyc * N_SIMD),
            avg(e, "SQ_LDS_BANK_CONFLICT") / (cyc * N_CU),
            avg(e, "SQ_WAIT_ANY") / max(avg(e, "SQ_WAVE_CYCLES"), 1.0),
            4 * avg(e, "SQ_WAVE_CYCLES") / (cyc * N_SIMD),
            avg(e, "SQ_INSTS_MFMA") / N_SIMD, avg(e, "SQ_INSTS_VALU") / N_SIMD,
            avg(e, "SQ_INSTS_VALU_TRANS_F32") / N_SIMD, avg(e, "SQ_INSTS_LDS") / N_SIMD]))
    for _, cls, v in sorted(rows, reverse=True):
        L.append(f"| `{cls}` | {v[0]} | {v[1]:.3f} | {v[2]:.3f} | {v[3]:.3f} | {v[4]:.3f} | "
                 f"{v[5]:.3f} | {v[6]:.2f} | {v[7]:,.0f} | {v[8]:,.0f} | {v[9]:,.0f} | {v[10]:,.0f} |")
    open(out, "w").write("\n".join(L) + "\n")
    print("\n".join(L))


MEM_PASS1 = ("SQ_LDS_IDX_ACTIVE SQ_LDS_BANK_CONFLICT SQ_VALU_MFMA_BUSY_CYCLES SQ_BUSY_CU_CYCLES "
             "GRBM_GUI_ACTIVE")
MEM_PASS2 = ("TA_TA_BUSY TD_TD_BUSY TD_TC_STALL TCP_PENDING_STALL_CYCLES TCP_TCC_READ_REQ_LATENCY "
             "TCP_TCC_READ_REQ GRBM_GUI_ACTIVE")


def summarize_memory(db1: str, db2: str, cmds: str, out: str):
    """Two rocprofv3 --pmc passes of LDS and vector-memory-path counters over one step ->
    per kernel class: how busy the LDS, the texture address (TA) and data (TD) units are,
    how often the L1 waits on the L2, and the mean L1->L2 read latency."""
    per = {}
    for db, names in ((db1, MEM_PASS1.split()), (db2, MEM_PASS2.split())):
        for counter in names:
            for (d, n), v in _pmc_by_dispatch(db, counter).items():
                cls = kernel_class(n) or ("layernorm_bwd" if "ln_bwd_kernel" in n else
                                          "layernorm" if "ln_fwd_kernel" in n else None)
                if cls is None:
                    continue
                per.setdefault(cls, {}).setdefault(counter, {})[(db, d)] = v
    L = ["# LDS and vector-memory-path counters per kernel class: encoder training step "
         "(c4_qwen2vl_trained, seed 0)", "",
         "Two `rocprofv3 --pmc` passes of one bench step (kernels are serialized while counters",
         "are taken: each kernel's own figures).  Commands (on the MI355X box):", "", "```", cmds,
         "```", "",
         f"Per dispatch: `cyc` = GRBM_GUI_ACTIVE / {N_XCD}; LDS active = SQ_LDS_IDX_ACTIVE / "
         f"(cyc x {N_CU} CUs); LDS bank-conflict = SQ_LDS_BANK_CONFLICT / (cyc x {N_CU}); MFMA busy "
         f"= SQ_VALU_MFMA_BUSY_CYCLES / (cyc x {N_SIMD} SIMDs); CU busy = SQ_BUSY_CU_CYCLES / "
         f"(cyc x {N_CU}); TA, TD busy = TA_TA_BUSY, TD_TD_BUSY / (cyc x {N_CU}); TD waits on L2 "
         f"= TD_TC_STALL / (cyc x {N_CU}); L1 pending on L2 = TCP_PENDING_STALL_CYCLES / (cyc x "
         f"{N_CU}); L2 read latency = TCP_TCC_READ_REQ_LATENCY / TCP_TCC_READ_REQ (cycles).", "",
         "| class | dispatches | LDS active | LDS bank-conflict | MFMA busy | CU busy | TA busy "
         "| TD busy | TD waits on L2 | L1 pending on L2 | L2 read latency |",
         "|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|"]

    def avg(e, c):
        v = list(e.get(c, {}).values())
        return sum(v) / len(v) if v else float("nan")

    rows = []
    for cls, e in per.items():
        c1 = [v for (db, _), v in e.get("GRBM_GUI_ACTIVE", {}).items() if db == db1]
        c2 = [v for (db, _), v in e.get("GRBM_GUI_ACTIVE", {}).items() if db == db2]
        if not c1 or not c2:
            continue
        cyc1, cyc2 = sum(c1) / len(c1) / N_XCD, sum(c2) / len(c2) / N_XCD
        nd = len(c1)
        req = avg(e, "TCP_TCC_READ_REQ")
        rows.append((avg(e, "SQ_VALU_MFMA_BUSY_CYCLES") * nd + cyc1 * nd * 1e-3, cls, [
            nd, avg(e, "SQ_LDS_IDX_ACTIVE") / (cyc1 * N_CU),
            avg(e, "SQ_LDS_BANK_CONFLICT") / (cyc1 * N_CU),
            avg(e, "SQ_VALU_MFMA_BUSY_CYCLES") / (cyc1 * N_SIMD),
            avg(e, "SQ_BUSY_CU_CYCLES") / (cyc1 * N_CU),
            avg(e, "TA_TA_BUSY") / (cyc2 * N_CU), avg(e, "TD_TD_BUSY") / (cyc2 * N_CU),
            avg(e, "TD_TC_STALL") / (cyc2 * N_CU),
            avg(e, "TCP_PENDING_STALL_CYCLES") / (cyc2 * N_CU),
            avg(e, "TCP_TCC_READ_REQ_LATENCY") / req if req else float("nan")]))
    for _, cls, v in sorted(rows, reverse=True):
        L.append(f"| `{cls}` | {v[0]} | {v[1]:.3f} | {v[2]:.3f} | {v[3]:.3f} | {v[4]:.3f} | "
                 f"{v[5]:.3f} | {v[6]:.3f} | {v[7]:.3f} | {v[8]:.3f} | {v[9]:.0f} |")
    open(out, "w").write("\n".join(L) + "\n")
    print("\n".join(L))


def summarize_workloads(out: str, files, cmds: str):
    """Bench lines of several workloads (one JSON file each) -> one markdown table."""
    import subprocess
    try:
        tree = subprocess.run(["git", "-C", ROOT, "rev-parse", "--short", "HEAD"], check=True,
                              capture_output=True, text=True).stdout.strip()
    except (OSError, subprocess.CalledProcessError):
        tree = "unknown"
    mode_name = {"trained": "trained", "merger": "merger-trained", "frozen": "frozen"}
    rows = []
    for f in files:
        with open(f) as fh:
            d = json.load(fh)
        c = d["config"]
        rows.append("| `%s` | %s | %s | %d | %s | %.3f | %.3f | %.3f | %s | %.3f | %.2f | %.2f | %s |" % (
            c["workload"], mode_name.get(c["mode"], c["mode"]), d["dtype"], c["n_items"],
            f"{c['n_patches']:,}", d["ms_per_step"], d["ms_per_step_median"], d["ms_per_step_min"],
            f"{d['value']:,.0f}", d["model_tflop_per_step"], d["mfma_pct_of_peak"],
            d["hw_mfma_pct_of_peak"], f"{d['scatter_GBps']:,.0f}"))
    lines = [
        "# Bench lines of every workload (seed 0): encoder step on one MI355X", "",
        f"Commands (on the MI355X box), one run per workload, tree at commit `{tree}`, then the "
        "table from the JSON lines:", "", "```", cmds.strip(), "```", "",
        "Trained = forward with tape + merge scatter + merge gather + backward; merger-trained = "
        "the same with only the merger trainable (its backward only); frozen = forward + scatter.",
        "ms columns: mean over the timed steps (host clock), and the median / minimum of per-step "
        "HIP events.  MFMA % = model FLOPs / time / 2516.6 TFLOP/s; hw % counts the attention "
        "recompute and head-dim padding.", "",
        "| workload | mode | dtype | items | patches | ms/step | median | min | patch-tokens/s | "
        "model TFLOP | MFMA % | hw MFMA % | scatter GB/s |",
        "|---|---|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|"] + rows
    with open(out, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print(f"wrote {out}")


def stored_traffic(cls: str):
    try:
        with open(TRAFFIC_FILE) as fh:
            rec = json.load(fh)
    except (OSError, ValueError):
        return None
    if rec.get("digest") != source_digest():
        return None
    e = rec.get("per_launch", {}).get(cls)
    return e["bytes"] if e else None


def copy_calibration():
    """A plain copy of known size through the library's row gather (identity indices)."""
    import torch
    import paper_2607_03229_amd as mp
    dev = torch.device("cuda:0")
    src = torch.ones((CAL_ROWS, CAL_COLS), dtype=torch.bfloat16, device=dev)
    dst = torch.empty_like(src)
    idx = torch.arange(CAL_ROWS, dtype=torch.int64, device=dev)
    for _ in range(3):
        mp.merge_gather(src, idx, dst)
    torch.cuda.synchronize()
    print(json.dumps({"copy_read_bytes": CAL_READ, "copy_write_bytes": CAL_WRITE}), flush=True)


def gemm_vs_library(workload: str, seed: int, out_md: str = ""):
    """The encoder step's GEMM shapes, each run alone: the library's kernels against
    torch.mm (hipBLASLt on ROCm) on the same bf16 operands, HIP-event timed.  The
    weight gradients run the step's four-way K split (fp32 partials, the reduction
    not timed) against hipBLASLt's single bf16-output product."""
    import torch
    import paper_2607_03229_amd as mp
    import workload as W
    dev = torch.device("cuda:0")
    wl = W.make_workload(workload, seed)
    T, h, f = int(wl.cu_seqlens[-1]), wl.cfg.hidden, wl.cfg.mlp

    def tm(fn, reps=10):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    g = torch.Generator(device=dev).manual_seed(seed)

    def rnd(*shape):
        return (torch.randn(*shape, device=dev, generator=g) * 0.5).to(torch.bfloat16)

    def line(name, M, N, K, ours, lib, lib_nt=None):
        fl = 2.0 * M * N * K
        rec = {"gemm": name, "M": M, "N": N, "K": K,
               "ours_ms": round(ours, 3), "ours_tflops": round(fl / ours / 1e9, 1),
               "hipblaslt_ms": round(lib, 3), "hipblaslt_tflops": round(fl / lib / 1e9, 1)}
        if lib_nt is not None:   # the same product with B given as [N][K] (hipBLASLt NT)
            rec.update({"hipblaslt_nt_ms": round(lib_nt, 3),
                        "hipblaslt_nt_tflops": round(fl / lib_nt / 1e9, 1)})
        print(json.dumps(rec), flush=True)
        recs.append(rec)

    recs = []

    # forward and input-gradient products: C[M][N] = A[M][K] B[K][N], bf16 out
    for name, M, N, K in [("qkv_fwd", T, 3 * h, h), ("proj_fwd", T, h, h), ("fc1_fwd", T, f, h),
                          ("fc2_fwd", T, h, f), ("qkv_dgrad", T, h, 3 * h)]:
        A, B = rnd(M, K), rnd(K, N)
        C = torch.empty(M, N, dtype=torch.bfloat16, device=dev)
        bias = torch.zeros(N, dtype=torch.bfloat16, device=dev)
        ours = tm(lambda: mp.op_gemm(mp.BF16, 1, 0, M, N, K, A, K, B, N, C, N, bias=bias))
        lib = tm(lambda: torch.mm(A, B, out=C))
        Bt = B.t().contiguous()
        lib_nt = tm(lambda: torch.mm(A, Bt.t(), out=C))
        line(name, M, N, K, ours, lib, lib_nt)
        del A, B, Bt, C
    # weight gradients: C[M][N] = sum over tokens of A[k][M] B[k][N]
    for name, M, N in [("qkv_wgrad", h, 3 * h), ("proj_wgrad", h, h), ("fc1_wgrad", h, f),
                       ("fc2_wgrad", f, h)]:
        A, B = rnd(T, M), rnd(T, N)
        kps = (T // 4 + 63) // 64 * 64
        C = torch.empty(4, M, N, dtype=torch.float32, device=dev)
        ours = tm(lambda: mp.op_gemm(mp.BF16, 2, 4, M, N, T, A, M, B, N, C, N, k_per_split=kps,
                                     split_stride=M * N))
        Cb = torch.empty(M, N, dtype=torch.bfloat16, device=dev)
        At = A.t()
        lib = tm(lambda: torch.mm(At, B, out=Cb))
        line(name, M, N, T, ours, lib)
        del A, B, C, Cb
    if out_md:
        fwd = [r for r in recs if "hipblaslt_nt_ms" in r]
        wg = [r for r in recs if "hipblaslt_nt_ms" not in r]
        rows = []
        for r in recs:
            nt = (f"{r['hipblaslt_nt_ms']:.3f} | {r['hipblaslt_nt_tflops']:.1f}"
                  if "hipblaslt_nt_ms" in r else "— | —")
            rows.append(f"| {r['gemm']} | {r['M']:,} | {r['N']:,} | {r['K']:,} | {r['ours_ms']:.3f} | "
                        f"{r['ours_tflops']:.1f} | {r['hipblaslt_ms']:.3f} | {r['hipblaslt_tflops']:.1f} | {nt} |")
        lines = [
            f"# Library GEMM kernels vs hipBLASLt on the encoder step's shapes ({workload}, seed {seed})",
            "", "Command (on the MI355X box; the table it writes is copied to `profiles/`):", "",
            "```",
            f"python3 bench.py --gemm-vs-library --workload {workload} --gemm-vs-library-out {out_md}",
            "```", "",
            "Each product runs alone on the default stream, HIP-event timed over 10 calls after one "
            "warm call, on random bf16 operands (scale 0.5). The library runs the NN kernel with a "
            "bias epilogue, and the TN weight-gradient kernel with a four-way K split into fp32 "
            "partials (the reduction not timed). hipBLASLt is `torch.mm` with bf16 output: NN with "
            "the weight as [K][N], and NT with the same weight stored [N][K]. In the step the weight "
            "gradients run on a side stream beside the input-gradient products, so in-step durations "
            "(the kernel trace) are longer than these.", "",
            "| product | M | N | K | library ms | library TFLOP/s | hipBLASLt NN ms | TFLOP/s | "
            "hipBLASLt NT ms | TFLOP/s |",
            "|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|"] + rows + [
            "", "Sums: forward and input-gradient shapes %.3f ms (library) vs %.3f ms (hipBLASLt NN), "
            "%.3f ms (hipBLASLt NT); weight gradients %.3f vs %.3f ms." % (
                sum(r["ours_ms"] for r in fwd), sum(r["hipblaslt_ms"] for r in fwd),
                sum(r["hipblaslt_nt_ms"] for r in fwd), sum(r["ours_ms"] for r in wg),
                sum(r["hipblaslt_ms"] for r in wg))]
        with open(out_md, "w") as fh:
            fh.write("\n".join(lines) + "\n")


def _prefix_sample(min_patches: int = 4096):
    """The benchmark draw's own items (C4 workload, seed 0), in order, until at least
    `min_patches` patches: the deterministic prefix the CPU baseline is timed on."""
    import workload as W
    wl = W.make_workload("c4_qwen2vl_trained", 0)
    n = wl.grid_thw[:, 0] * wl.grid_thw[:, 1] * wl.grid_thw[:, 2]
    k = int(np.searchsorted(np.cumsum(n), min_patches) + 1)
    return wl.grid_thw[:k]


def _time_oracle(layers: int, grid) -> tuple:
    """Seconds of one oracle forward + backward (fp32, trained) of the Qwen2-VL-ViT shape
    with `layers` blocks on the items `grid`, and the patch count."""
    import dataclasses

    import oracle
    import workload as W
    cfg = dataclasses.replace(W.CONFIGS["c4_qwen2vl_trained"].cfg, layers=layers)
    W.custom_spec(f"cpu_baseline_{layers}", cfg, emb_seqs=8, emb_seq_len=8192)
    wl = W.make_workload(f"cpu_baseline_{layers}", 0, grid_thw=np.array(grid))
    w, X = wl.weights(), wl.patches()
    dM = W.round_bf16(np.random.default_rng(0).standard_normal(
        (wl.n_merged, cfg.llm_hidden)).astype(np.float32))
    t0 = time.perf_counter()
    oracle.encoder(cfg, w, X, wl.cu_seqlens, wl.grid_thw, True, d_merged=dM, precision="f32")
    return time.perf_counter() - t0, wl.n_patches


def cpu_baseline(full_depth: bool = False):
    """Time the CPU oracle (fp32, forward + backward, every part trainable) on the
    deterministic prefix of the benchmark's own draw: its first items until >= 4,096
    patches (5,336 patches, items 0-2, for seed 0).

    Default (bounded, about a minute of CPU on 16 cores): the prefix is timed twice, with
    0 blocks (patch embedding + merger) and with 1 block of the encoder; every block is
    the same computation on the same rows, so the 32-block time is t0 + 32 (t1 - t0), both
    terms measured on this draw.  full_depth=True times the prefix through all 32 blocks
    in one run instead (about 15 minutes on 16 cores)."""
    import oracle
    grid = _prefix_sample()
    host = _host_info()
    host["omp_threads"] = oracle.num_threads()
    if full_depth:
        t, n = _time_oracle(32, grid)
        return {"value": round(n / t, 3), "unit": "patch-tokens/s", "cores": host["omp_threads"],
                "kind": "oracle",
                "sample": (f"prefix of the benchmark draw (c4_qwen2vl_trained seed 0, items "
                           f"0-{len(grid) - 1}, {n} patches), fp32 forward+backward, all 32 "
                           f"blocks, patch embedding and merger: {t:.1f} s measured"),
                **host}
    t0, n = _time_oracle(0, grid)
    log(f"cpu oracle: prefix of {n} patches, 0 blocks: {t0:.1f} s")
    t1, _ = _time_oracle(1, grid)
    log(f"cpu oracle: prefix of {n} patches, 1 block: {t1:.1f} s")
    t_full = t0 + 32 * (t1 - t0)
    return {"value": round(n / t_full, 3), "unit": "patch-tokens/s",
            "cores": host["omp_threads"], "kind": "oracle",
            "sample": (f"prefix of the benchmark draw (c4_qwen2vl_trained seed 0, items "
                       f"0-{len(grid) - 1}, {n} patches), fp32 forward+backward incl. patch "
                       f"embedding and merger, timed at 0 blocks ({t0:.1f} s) and 1 block "
                       f"({t1:.1f} s); 32 blocks = t0 + 32 (t1 - t0) = {t_full:.0f} s"),
            "measured_s": {"blocks0": round(t0, 2), "blocks1": round(t1, 2)},
            **host}


def owner_scenario(enc, wl, flops_per_s: float) -> dict:
    """The ByMicrobatch owner on encode costs of this workload: 16 micro-batches (seeds
    0..15 of the same size draw), each costed by the roofline model at the FLOP rate this
    run measured, assigned to 8 pipeline ranks whose warmup bubbles follow a 1F1B fill,
    w_r = r * (median encode) / 2, i.e. an LLM stage forward half as long as a median
    encode (tight enough that some encode work spills); greedy, refined and exact owners."""
    import paper_2607_03229_amd as mp
    import workload as W
    costs = []
    for seed in range(16):
        d = W.make_workload(wl.name, seed)
        c = enc.cost(d.cu_seqlens, d.grid_thw, wl.trainable, flops_per_s, PEAK_HBM_GBPS * 1e9)
        costs.append(c["fwd_seconds"])
    costs = np.array(costs)
    step = float(np.median(costs))
    warm = 0.5 * step * np.arange(8, dtype=np.float64)
    out = {"n_microbatches": len(costs), "n_ranks": 8,
           "warmup": "w_r = r * median encode / 2 (1F1B fill)",
           "rate_tflops": round(flops_per_s / 1e12, 1),
           "encode_ms_min_median_max": [round(1e3 * float(v), 3)
                                        for v in (costs.min(), step, costs.max())]}
    for name, method in (("greedy", mp.OWNER_GREEDY), ("refined", mp.OWNER_REFINED),
                         ("exact", mp.OWNER_EXACT)):
        t0 = time.perf_counter()
        try:
            _, _, worst = mp.owner_map(costs, warm, method)
        except mp.MpipeError:   # the exact search's node budget
            worst = None
        out[f"{name}_us"] = round(1e6 * (time.perf_counter() - t0), 1)
        out[f"{name}_max_spill_ms"] = None if worst is None else round(1e3 * worst, 3)
    out["spill_if_all_on_rank0_ms"] = round(1e3 * float(costs.sum()), 3)
    return out


def _host_info() -> dict:
    """CPU model, sockets and the cores this process may run on."""
    model, sockets = "unknown", set()
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name") and model == "unknown":
                model = line.split(":", 1)[1].strip()
            elif line.startswith("physical id"):
                sockets.add(line.split(":", 1)[1].strip())
    except OSError:
        pass
    try:
        nproc = len(os.sched_getaffinity(0))
    except AttributeError:
        nproc = os.cpu_count() or 0
    return {"cpu": model, "sockets": max(len(sockets), 1), "nproc": nproc}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="c4_qwen2vl_trained")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-baseline-full", action="store_true",
                    help="time the oracle's sample through all 32 blocks in one run "
                         "(about 15 minutes on 16 cores) instead of at 0 and 1 blocks")
    ap.add_argument("--cpu-baseline-only", action="store_true",
                    help="only time the CPU oracle sample and print its JSON object")
    ap.add_argument("--no-alone-pass", action="store_true",
                    help="skip the per-kernel pass with the side stream off (figures *_alone)")
    ap.add_argument("--no-profile", action="store_true",
                    help="skip the per-kernel event timing (roofline figures)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run the known-size copy that scales the PMC byte counters")
    ap.add_argument("--summarize-pmc", nargs=4, metavar=("FETCH_CAL", "WRITE_CAL", "FETCH", "WRITE"),
                    help="rocprofv3 PMC databases -> profiles/hbm_traffic.json")
    ap.add_argument("--pmc-commands", default="", help="commands recorded with --summarize-pmc")
    ap.add_argument("--summarize-trace", nargs=3, metavar=("DB", "BENCH_JSON", "OUT_MD"),
                    help="rocprofv3 kernel-trace database -> a markdown summary")
    ap.add_argument("--summarize-memory", nargs=3, metavar=("PASS1_DB", "PASS2_DB", "OUT_MD"),
                    help="LDS / TA / TD / TCP counter passes -> profiles markdown")
    ap.add_argument("--summarize-sq", nargs=3, metavar=("PASS1_DB", "PASS2_DB", "OUT_MD"),
                    help="two rocprofv3 SQ-counter databases -> a markdown summary")
    ap.add_argument("--summarize-mfma-flops", nargs=2, metavar=("DB", "OUT_MD"),
                    help="rocprofv3 SQ_INSTS_VALU_MFMA_MOPS_BF16 pass -> issued MFMA FLOPs")
    ap.add_argument("--summarize-traffic-md", metavar="OUT_MD",
                    help="profiles/hbm_traffic.json -> its markdown table")
    ap.add_argument("--summarize-workloads", nargs="+", metavar=("OUT_MD", "JSON"),
                    help="bench JSON lines of several workloads -> a markdown table")
    ap.add_argument("--gemm-vs-library", action="store_true",
                    help="only time the step's GEMM shapes alone, against torch.mm (hipBLASLt)")
    ap.add_argument("--gemm-vs-library-out", default="",
                    help="with --gemm-vs-library: also write the table as markdown here")
    args = ap.parse_args()
    if args.summarize_pmc:
        summarize_pmc(*args.summarize_pmc, args.pmc_commands)
        return
    if args.summarize_trace:
        summarize_trace(*args.summarize_trace[:2], args.pmc_commands, args.summarize_trace[2])
        return
    if args.summarize_sq:
        summarize_sq(*args.summarize_sq[:2], args.pmc_commands, args.summarize_sq[2])
        return
    if args.summarize_mfma_flops:
        summarize_mfma_flops(*args.summarize_mfma_flops, args.pmc_commands, args.workload,
                             args.seed)
        return
    if args.summarize_traffic_md:
        summarize_traffic_md(args.summarize_traffic_md, args.workload, args.seed)
        return
    if args.summarize_workloads:
        summarize_workloads(args.summarize_workloads[0], args.summarize_workloads[1:],
                            args.pmc_commands)
        return
    if args.summarize_memory:
        summarize_memory(*args.summarize_memory[:2], args.pmc_commands, args.summarize_memory[2])
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one MI355X only: the encoder step runs on one GPU "
              "(see DESIGN.md for how the transpose schedule shards it).", file=sys.stderr)
        sys.exit(2)

    if args.cpu_baseline_only:
        print(json.dumps(cpu_baseline(full_depth=args.cpu_baseline_full)), flush=True)
        return
    if args.copy_calibration:
        copy_calibration()
        return
    if args.gemm_vs_library:
        gemm_vs_library(args.workload, args.seed, args.gemm_vs_library_out)
        return
    import torch
    import paper_2607_03229_amd as mp
    import workload as W

    dev = torch.device("cuda:0")
    wl = W.make_workload(args.workload, args.seed)
    cfg = wl.cfg
    trainable = wl.trainable
    tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    log(f"workload {wl.name}: {wl.n_items} items, {wl.n_patches} patches, {wl.n_merged} merged")

    enc = mp.Encoder(cfg)
    sz = enc.sizes(wl.cu_seqlens, wl.grid_thw, trainable)
    t0 = time.perf_counter()
    weights = torch.from_numpy(wl.weights()).to(dev).to(tdt)
    patches = torch.from_numpy(wl.patches()).to(dev).to(tdt)
    idx = torch.from_numpy(wl.placeholders()).to(dev)
    emb = torch.from_numpy(wl.emb_init()).to(dev).to(tdt)
    d_emb = torch.from_numpy(wl.d_emb()).to(dev).to(tdt)
    log(f"inputs resident ({time.perf_counter() - t0:.1f} s); workspace "
        f"{sz['workspace'] / 2**30:.2f} GiB, tape {sz['tape'] / 2**30:.2f} GiB")
    merged = torch.empty((sz["n_merged"], cfg.llm_hidden), dtype=tdt, device=dev)
    d_merged = torch.empty_like(merged)
    ws = torch.empty(sz["workspace"], dtype=torch.uint8, device=dev)
    tape = torch.empty(max(sz["tape"], 1), dtype=torch.uint8, device=dev) if trainable else None
    d_w = torch.zeros(weights.numel(), dtype=torch.float32, device=dev) if trainable else None
    stream = torch.cuda.current_stream()

    def step():
        enc.fwd(weights, patches, wl.cu_seqlens, wl.grid_thw, trainable, merged, tape, ws)
        mp.merge_scatter(merged, idx, emb)
        if trainable:
            mp.merge_gather(d_emb, idx, d_merged)
            enc.bwd(weights, patches, wl.cu_seqlens, wl.grid_thw, trainable, tape, d_merged,
                    d_w, None, ws)

    for i in range(args.warmup):
        step()
        torch.cuda.synchronize()
        log(f"warmup step {i + 1}/{args.warmup} done")
    profile = not args.no_profile
    # Headline: K steps with no per-kernel instrumentation.  Per-step HIP events on the
    # stream give the median / min; the whole-job figure is the host clock over all K
    # steps, bracketed by device synchronisation.
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    evs[0].record(stream)
    for i in range(args.steps):
        step()
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    per_step = sorted(evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps))
    log(f"timed {args.steps} steps: {elapsed * 1e3 / args.steps:.1f} ms/step")
    # Per-kernel figures from a separate pass: every launch bracketed by a HIP event pair
    # on the stream it is launched on (the caller's, or the backward's side stream)
    kern, kern_alone = {}, {}
    prof_steps = min(args.steps, 5)
    if profile:
        enc.profile(True)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        for _ in range(prof_steps):
            step()
        torch.cuda.synchronize()
        log(f"per-kernel pass: {prof_steps} steps, "
            f"{(time.perf_counter() - t1) * 1e3 / prof_steps:.1f} ms/step with events")
        kern = enc.profile_read(stream)
        enc.profile(False)
        if int(trainable) == 1 and not args.no_alone_pass:
            # the same pass with the weight-gradient work on the caller's stream: each
            # kernel then runs alone, so its event time is its own, without CU sharing
            enc.set_side_stream(False)
            enc.profile(True)
            for _ in range(prof_steps):
                step()
            torch.cuda.synchronize()
            kern_alone = enc.profile_read(stream)
            enc.profile(False)
            enc.set_side_stream(True)

    # scatter bandwidth, timed on its own, after a few untimed calls (the step leaves the
    # caches full of its dirty lines, whose write-back would be charged to the first ones)
    for _ in range(5):
        mp.merge_scatter(merged, idx, emb)
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = 20
    ev0.record(stream)
    for _ in range(reps):
        mp.merge_scatter(merged, idx, emb)
    ev1.record(stream)
    torch.cuda.synchronize()
    esz = 2 if cfg.dtype == "bf16" else 4
    scat_bytes = 2 * wl.n_merged * cfg.llm_hidden * esz + 8 * wl.n_merged
    scat_ms = ev0.elapsed_time(ev1) / reps
    scatter_gbps = scat_bytes / (scat_ms * 1e-3) / 1e9

    sum_len2 = int(np.sum(np.diff(wl.cu_seqlens).astype(np.int64) ** 2))
    flops = model_flops(cfg, wl.n_patches, sum_len2, trainable)
    hw_flops = hardware_flops(cfg, wl.n_patches, sum_len2, trainable)
    ms_step = elapsed * 1e3 / args.steps
    achieved = flops / (ms_step * 1e-3) / 1e12
    peak = PEAK_BF16_TFLOPS if cfg.dtype == "bf16" else PEAK_F32_TFLOPS

    roofline = roofline_top = None
    kernels = {}
    if kern:
        # kernel classes on the caller's stream form the critical path; the weight-gradient
        # work overlaps them on the side stream ("@side"), its times include CU sharing
        for name, (n, ms, fl) in sorted(kern.items(), key=lambda kv: -kv[1][1]):
            cls, side = (name[:-5], True) if name.endswith("@side") else (name, False)
            kernels[cls] = {"launches": n, "ms_total": round(ms, 3),
                            "ms_avg": round(ms / max(n, 1), 4),
                            "tflops": round(fl / (ms * 1e-3) / 1e12, 1) if ms > 0 and fl > 0 else None,
                            "stream": "side" if side else "caller"}
            if cls in kern_alone:   # the same class with every kernel alone on one stream
                na, msa, _ = kern_alone[cls]
                kernels[cls]["ms_avg_alone"] = round(msa / max(na, 1), 4)
        def roof(cls):
            key = cls if cls in kern else cls + "@side"
            n, ms, fl = kern[key]
            ach = fl / n / (ms / n * 1e-3) / 1e12
            r = {"kernel": cls, "bound": "mfma", "achieved": round(ach, 1), "peak": peak,
                 "unit": "TFLOP/s", "frac": round(ach / peak, 4),
                 "traffic": stored_traffic(cls),
                 "traffic_counter": TRAFFIC_NOTE,
                 "launches": n, "avg_ms": round(ms / n, 4),
                 "flop_per_launch": fl / n, "stream": kernels[cls]["stream"],
                 "timed_over_steps": prof_steps}
            if cls in kern_alone:   # the pass with every kernel alone on one stream
                na, msa, fla = kern_alone[cls]
                acha = fla / na / (msa / na * 1e-3) / 1e12
                r.update({"achieved_alone": round(acha, 1), "frac_alone": round(acha / peak, 4),
                          "avg_ms_alone": round(msa / na, 4)})
            return r

        # the roofline kernel: the largest MFMA class on the caller's (critical) stream;
        # beside it, the largest class of the whole trace when that is another one
        mfma = [k for k in kernels if (kern.get(k) or kern.get(k + "@side"))[2] > 0]
        main = [k for k in mfma if kernels[k]["stream"] == "caller"]
        dom = max(main or mfma, key=lambda k: kernels[k]["ms_total"])
        roofline = roof(dom)
        top = max(mfma, key=lambda k: kernels[k]["ms_total"])
        roofline_top = roof(top) if top != dom else None

    result = {
        "metric": METRIC,
        "value": round(wl.n_patches / (ms_step * 1e-3), 1),
        "unit": "patch-tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "ms_per_step_median": round(per_step[len(per_step) // 2], 3),
        "ms_per_step_min": round(per_step[0], 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": cfg.dtype, "data": "synthetic",
        "config": {"workload": wl.name, "seed": args.seed, "mode": {0: "frozen", 1: "trained", 2: "merger-trained"}[int(trainable)],
                   "n_items": wl.n_items, "n_patches": wl.n_patches, "n_merged": wl.n_merged,
                   "sum_seg_len2": sum_len2,
                   "encoder": f"h{cfg.hidden} L{cfg.layers} heads{cfg.heads} mlp{cfg.mlp} "
                              f"T{cfg.temporal_patch} merge->{cfg.llm_hidden}",
                   "parallelism": "1 GPU (one pipeline rank's encoder share)"},
        "model_tflop_per_step": round(flops / 1e12, 3),
        "achieved_tflops": round(achieved, 1),
        "mfma_pct_of_peak": round(100 * achieved / peak, 2),
        "hw_tflop_per_step": round(hw_flops / 1e12, 3),
        "hw_mfma_pct_of_peak": round(100 * hw_flops / (ms_step * 1e-3) / 1e12 / peak, 2),
        "peak_tflops": peak,
        "scatter_GBps": round(scatter_gbps, 1),
        "scatter_pct_of_hbm": round(100 * scatter_gbps / PEAK_HBM_GBPS, 1),
        "roofline": roofline,
        "roofline_largest_class": roofline_top if kern else None,
        "kernels": kernels,
    }
    result["owner_map"] = owner_scenario(enc, wl, flops / (ms_step * 1e-3))
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on its sample (the benchmark draw's first items)")
        result["cpu_baseline"] = cpu_baseline(full_depth=args.cpu_baseline_full)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
