"""Summaries of rocprofv3 output for the profiles/ folder.

    python profiling.py stats   --csv DIR/run_kernel_stats.csv --cmd "..." --out profiles/X.md
    python profiling.py traffic --fetch DIR1/run_counter_collection.csv \
        --write DIR2/run_counter_collection.csv --copy-bytes N --cmd "..." --out profiles/hbm_traffic.json \
        [--tag WORKLOAD --append]
    python profiling.py counters --mfma DIR3/run_counter_collection.csv --l2 DIR4/run_counter_collection.csv \
        --cmd "..." --out profiles/mfma_counters.json [--tag WORKLOAD --append]
    python profiling.py issue --csv DIR5/run_counter_collection.csv [--csv DIR6/...] \
        --cmd "..." --out profiles/simd_issue_breakdown.json

`traffic` turns FETCH_SIZE / WRITE_SIZE (KiB per dispatch) into bytes per
launch for every GCA kernel, scaled by what the same counters read for a plain
device copy of N bytes in the same run (the copy kernel is the dispatch whose
name contains "copy").  The result records a hash of the kernel sources, so a
reader (bench.py) can tell when the kernels have changed since the counters
were taken.  `--tag` suffixes the kernel names with "@WORKLOAD" (a kernel that
runs in two workloads, such as the cross attention at 64K training and at 16M
decode, is then kept apart) and `--append` adds the result to an existing file
taken from the same sources.
"""

import argparse
import csv
import hashlib
import json
import os
import statistics

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "paper_2410_01651_amd", "csrc")


def source_hash() -> str:
    """sha256 over the kernel sources (file names and contents, sorted)."""
    h = hashlib.sha256()
    for name in sorted(os.listdir(CSRC)):
        if name.endswith((".hip", ".hpp", ".cpp")):
            h.update(name.encode())
            with open(os.path.join(CSRC, name), "rb") as f:
                h.update(f.read())
    return h.hexdigest()


def short_name(kernel: str) -> str:
    for key in ("xattn_fwd_kernel", "bwd_dq_kernel", "bwd_dkdv_kernel", "chunk_scores_kernel", "topk_kernel",
                "fused_select_kernel", "select_part_kernel", "select_merge_kernel", "decode_scan_kernel", "xattn_decode_kernel", "weights_kernel",
                "fill_zero_kernel", "csr_count_kernel", "csr_scan_kernel", "csr_fill_kernel", "csr_sort_kernel",
                "dsel_kernel", "dlmk_q_kernel", "dlmk_k_kernel"):
        if key in kernel:
            return key
    if "copy" in kernel.lower():
        return "copy"
    return kernel[:60]


def stats_md(stats_csv: str, cmd: str) -> str:
    rows = list(csv.DictReader(open(stats_csv)))
    out = ["# rocprofv3 kernel statistics", "", "Command:", "", "```", cmd, "```", "",
           "| kernel | calls | total (us) | average (us) | min (us) | max (us) | % |",
           "|---|---|---|---|---|---|---|"]
    for r in rows:
        name = short_name(r["Name"])
        ns = lambda k: float(r[k]) / 1000.0
        out.append(f"| {name} | {r['Calls']} | {ns('TotalDurationNs'):.1f} | {ns('AverageNs'):.2f} | "
                   f"{ns('MinNs'):.2f} | {ns('MaxNs'):.2f} | {float(r['Percentage']):.2f} |")
    return "\n".join(out) + "\n"


def trace_md(trace_csv: str, cmd: str) -> str:
    """Per (kernel, grid size) duration statistics from a rocprofv3 kernel trace, so
    launches of one kernel on different workloads are reported apart."""
    groups = {}
    for r in csv.DictReader(open(trace_csv)):
        grid = r.get("Grid_Size") or r.get("Grid_Size_X") or "?"
        dur = (float(r["End_Timestamp"]) - float(r["Start_Timestamp"])) / 1000.0
        groups.setdefault((short_name(r["Kernel_Name"]), grid), []).append(dur)
    total = sum(sum(v) for v in groups.values())
    out = ["# rocprofv3 kernel trace, per kernel and grid size", "", "Command:", "", "```", cmd, "```", "",
           "| kernel | grid (work-items) | calls | average (us) | median (us) | min (us) | max (us) | % of GPU time |",
           "|---|---|---|---|---|---|---|---|"]
    for (name, grid), v in sorted(groups.items(), key=lambda kv: -sum(kv[1])):
        v = sorted(v)
        out.append(f"| {name} | {grid} | {len(v)} | {sum(v) / len(v):.2f} | {v[len(v) // 2]:.2f} | {v[0]:.2f} | "
                   f"{v[-1]:.2f} | {100 * sum(v) / total:.2f} |")
    return "\n".join(out) + "\n"


def _per_kernel(counter_csv: str, counter: str):
    vals = {}
    for r in csv.DictReader(open(counter_csv)):
        if r["Counter_Name"] != counter:
            continue
        vals.setdefault(short_name(r["Kernel_Name"]), []).append(float(r["Counter_Value"]))
    return vals


def traffic(fetch_csv: str, write_csv: str, copy_bytes: int, cmd: str, tag: str = "") -> dict:
    f = _per_kernel(fetch_csv, "FETCH_SIZE")
    w = _per_kernel(write_csv, "WRITE_SIZE")
    if "copy" not in f or "copy" not in w:
        raise SystemExit("no copy kernel in the counter output (run bench.py with --copy-calibration-mb)")
    # the calibration copy reads and writes copy_bytes each
    f_scale = copy_bytes / (max(f["copy"]) * 1024.0)
    w_scale = copy_bytes / (max(w["copy"]) * 1024.0)
    kernels = {}
    for k in sorted(set(f) & set(w)):
        if k == "copy":
            continue
        kernels[k + ("@" + tag if tag else "")] = {
            "fetch_bytes_per_launch": statistics.median(f[k]) * 1024.0 * f_scale,
            "write_bytes_per_launch": statistics.median(w[k]) * 1024.0 * w_scale,
            "dispatches": len(f[k]),
        }
    return {"source_sha256": source_hash(), "copy_bytes": copy_bytes,
            "fetch_scale": f_scale, "write_scale": w_scale, "command": [cmd], "kernels": kernels}


def _per_kernel_all(counter_csv: str):
    """{kernel: {counter: [value per dispatch]}} of one rocprofv3 counter run."""
    vals = {}
    for r in csv.DictReader(open(counter_csv)):
        k = vals.setdefault(short_name(r["Kernel_Name"]), {})
        k.setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
    return vals


def agent_counts(counter_csv: str):
    """(SIMDs, XCCs) of the GPU from the run_agent_info.csv beside a counter CSV."""
    path = os.path.join(os.path.dirname(counter_csv), os.path.basename(counter_csv).replace(
        "counter_collection", "agent_info"))
    for r in csv.DictReader(open(path)):
        if r.get("Name", "").startswith("gfx"):
            return int(r["Simd_Count"]), int(r["Num_Xcc"])
    raise SystemExit(f"no GPU agent in {path}")


def counters(mfma_csv: str, l2_csv: str, cmd: str, tag: str = "", ea_csv: str = "") -> dict:
    """Matrix-core busy fraction (SQ_VALU_MFMA_BUSY_CYCLES over the busy cycles of
    every SIMD, the MfmaUtil definition: GRBM_GUI_ACTIVE is reported summed over the
    XCCs, so one XCC's count is the sum divided by their number), bf16 matrix-core
    flops (SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512) and the L2 hit fraction (TCC_HIT /
    (TCC_HIT + TCC_MISS)) per launch, the median over each kernel's dispatches.
    With `ea_csv` (TCC_EA0_RDREQ_LEVEL_sum, TCC_EA0_RDREQ_sum) also the average
    latency of the reads that leave the L2 (requests in flight summed per cycle
    over requests): this stack exposes no last-level-cache (MALL) counter, and
    this latency is where its hits show (lower than reads served by HBM)."""
    simds, xccs = agent_counts(mfma_csv)
    m = _per_kernel_all(mfma_csv)
    l2 = _per_kernel_all(l2_csv) if l2_csv else {}
    ea = _per_kernel_all(ea_csv) if ea_csv else {}
    med = statistics.median
    kernels = {}
    for k, c in sorted(m.items()):
        if k == "copy":
            continue
        e = {"dispatches": len(c.get("GRBM_GUI_ACTIVE", []))}
        if "SQ_VALU_MFMA_BUSY_CYCLES" in c and "GRBM_GUI_ACTIVE" in c:
            busy = [b / (g / xccs * simds) for b, g in zip(c["SQ_VALU_MFMA_BUSY_CYCLES"], c["GRBM_GUI_ACTIVE"])
                    if g > 0]
            e["mfma_busy_frac"] = med(busy) if busy else None
            e["gui_active_cycles_per_xcc"] = med(c["GRBM_GUI_ACTIVE"]) / xccs
        if "SQ_INSTS_VALU_MFMA_MOPS_BF16" in c:
            e["mfma_bf16_flops_per_launch"] = med(c["SQ_INSTS_VALU_MFMA_MOPS_BF16"]) * 512.0
        if "SQ_BUSY_CU_CYCLES" in c:
            e["sq_busy_cu_cycles"] = med(c["SQ_BUSY_CU_CYCLES"])
        h = l2.get(k, {})
        if "TCC_HIT_sum" in h and "TCC_MISS_sum" in h:
            fr = [a / (a + b) for a, b in zip(h["TCC_HIT_sum"], h["TCC_MISS_sum"]) if a + b > 0]
            e["l2_hit_frac"] = med(fr) if fr else None
            e["l2_requests_per_launch"] = med([a + b for a, b in zip(h["TCC_HIT_sum"], h["TCC_MISS_sum"])])
        x = ea.get(k, {})
        if "TCC_EA0_RDREQ_LEVEL_sum" in x and "TCC_EA0_RDREQ_sum" in x:
            lat = [a / b for a, b in zip(x["TCC_EA0_RDREQ_LEVEL_sum"], x["TCC_EA0_RDREQ_sum"]) if b > 0]
            e["l2_miss_read_latency_cycles"] = med(lat) if lat else None
        kernels[k + ("@" + tag if tag else "")] = e
    return {"source_sha256": source_hash(), "simds": simds, "xccs": xccs, "command": [cmd], "kernels": kernels}


def issue(csvs, cmd: str) -> dict:
    """Where each SIMD's cycles go, per launch of the attention kernels, from SQ
    counter runs that each include GRBM_GUI_ACTIVE (medians over dispatches).

    SIMD fractions (of GRBM_GUI_ACTIVE per XCC times the SIMD count): VALU issue
    (SQ_ACTIVE_INST_VALU, quad-cycles, so x4; it counts every VALU-class
    instruction's issue, matrix-core ones included), matrix cores busy
    (SQ_VALU_MFMA_BUSY_CYCLES), both at once (SQ_VALU_MFMA_COEXEC_CYCLES) and
    neither (the rest).  Wave fractions (of SQ_WAVE_CYCLES, quad-cycles like the
    others): issuing any instruction, waiting at s_waitcnt or a barrier
    (SQ_WAIT_ANY), and ready but not issued (SQ_WAIT_INST_ANY: a dependency or
    another wave holding the unit).  Per wave: instruction counts by class."""
    simds, xccs = agent_counts(csvs[0])
    med = statistics.median
    per = {}
    for path in csvs:
        for k, c in _per_kernel_all(path).items():
            if k not in ("xattn_fwd_kernel", "bwd_dq_kernel", "bwd_dkdv_kernel"):
                continue
            gui = c.get("GRBM_GUI_ACTIVE")
            for name, vals in c.items():
                if name == "GRBM_GUI_ACTIVE":
                    continue
                # each run's own clock normalises its own counters
                per.setdefault(k, {})[name] = (med(vals), med(gui))
    kernels = {}
    for k, c in sorted(per.items()):
        def simd(name, quad=False):
            v, g = c[name]
            return v * (4.0 if quad else 1.0) / (g / xccs * simds)
        def wave(name):
            return c[name][0] / c["SQ_WAVE_CYCLES"][0]
        e = {}
        if "SQ_ACTIVE_INST_VALU" in c:
            e["simd_valu_issue_frac"] = simd("SQ_ACTIVE_INST_VALU", quad=True)
        if "SQ_VALU_MFMA_BUSY_CYCLES" in c:
            e["simd_mfma_busy_frac"] = simd("SQ_VALU_MFMA_BUSY_CYCLES")
        if "SQ_VALU_MFMA_COEXEC_CYCLES" in c:
            e["simd_valu_and_mfma_frac"] = simd("SQ_VALU_MFMA_COEXEC_CYCLES")
        if all(x in e for x in ("simd_valu_issue_frac", "simd_mfma_busy_frac", "simd_valu_and_mfma_frac")):
            e["simd_neither_frac"] = 1.0 - e["simd_valu_issue_frac"] - e["simd_mfma_busy_frac"] + \
                e["simd_valu_and_mfma_frac"]
        if "SQ_WAVE_CYCLES" in c:
            for name, key in (("SQ_ACTIVE_INST_ANY", "wave_issuing_frac"), ("SQ_WAIT_ANY", "wave_waitcnt_or_barrier_frac"),
                              ("SQ_WAIT_INST_ANY", "wave_ready_not_issued_frac"),
                              ("SQ_WAIT_INST_LDS", "wave_lds_wait_frac")):
                if name in c:
                    e[key] = wave(name)
        if "SQ_WAVES" in c:
            n = c["SQ_WAVES"][0]
            e["waves"] = n
            for name, key in (("SQ_INSTS_VALU", "valu"), ("SQ_INSTS_MFMA", "mfma"), ("SQ_INSTS_LDS", "lds"),
                              ("SQ_INSTS_SALU", "salu"), ("SQ_INSTS_VALU_TRANS_F32", "valu_trans_f32")):
                if name in c:
                    e.setdefault("instructions_per_wave", {})[key] = c[name][0] / n
        if "SQ_LDS_BANK_CONFLICT" in c:
            e["lds_bank_conflict_cycles_per_launch"] = c["SQ_LDS_BANK_CONFLICT"][0]
        kernels[k] = e
    return {"source_sha256": source_hash(), "simds": simds, "xccs": xccs, "command": [cmd], "kernels": kernels}


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="what", required=True)
    a = sub.add_parser("stats")
    a.add_argument("--csv", required=True, help="run_kernel_stats.csv; a run_kernel_trace.csv beside it adds a "
                                                "per-grid table")
    a.add_argument("--cmd", required=True)
    a.add_argument("--out", required=True)
    b = sub.add_parser("traffic")
    b.add_argument("--fetch", required=True)
    b.add_argument("--write", required=True)
    b.add_argument("--copy-bytes", type=int, required=True)
    b.add_argument("--cmd", required=True)
    b.add_argument("--out", required=True)
    b.add_argument("--tag", default="")
    b.add_argument("--append", action="store_true")
    c = sub.add_parser("counters")
    c.add_argument("--mfma", required=True, help="counter CSV with SQ_VALU_MFMA_BUSY_CYCLES, "
                                                 "SQ_INSTS_VALU_MFMA_MOPS_BF16, GRBM_GUI_ACTIVE")
    c.add_argument("--l2", default="", help="counter CSV with TCC_HIT_sum, TCC_MISS_sum")
    c.add_argument("--ea", default="", help="counter CSV with TCC_EA0_RDREQ_LEVEL_sum, TCC_EA0_RDREQ_sum")
    c.add_argument("--cmd", required=True)
    c.add_argument("--out", required=True)
    c.add_argument("--tag", default="")
    c.add_argument("--append", action="store_true")
    d = sub.add_parser("issue")
    d.add_argument("--csv", action="append", required=True, help="counter CSV of one SQ counter run")
    d.add_argument("--cmd", required=True)
    d.add_argument("--out", required=True)
    args = ap.parse_args()
    if args.what == "issue":
        json.dump(issue(args.csv, args.cmd), open(args.out, "w"), indent=1)
        print(args.out)
        return
    if args.what == "counters":
        data = counters(args.mfma, args.l2, args.cmd, args.tag, args.ea)
        if args.append and os.path.exists(args.out):
            old = json.load(open(args.out))
            if old.get("source_sha256") != data["source_sha256"]:
                raise SystemExit(f"{args.out} was taken from other kernel sources")
            old["command"] = list(old["command"]) + data["command"]
            old["kernels"].update(data["kernels"])
            data = old
        json.dump(data, open(args.out, "w"), indent=1)
        print(args.out)
        return
    if args.what == "stats":
        text = stats_md(args.csv, args.cmd)
        trace = os.path.join(os.path.dirname(args.csv), os.path.basename(args.csv).replace("kernel_stats",
                                                                                         "kernel_trace"))
        if os.path.exists(trace):
            text += "\n" + trace_md(trace, args.cmd)
        open(args.out, "w").write(text)
    else:
        data = traffic(args.fetch, args.write, args.copy_bytes, args.cmd, args.tag)
        if args.append:
            old = json.load(open(args.out))
            if old.get("source_sha256") != data["source_sha256"]:
                raise SystemExit(f"{args.out} was taken from other kernel sources")
            old["command"] = list(old["command"]) + data["command"]
            old["kernels"].update(data["kernels"])
            old.setdefault("scales", {})[args.tag or "-"] = [data["fetch_scale"], data["write_scale"]]
            data = old
        json.dump(data, open(args.out, "w"), indent=1)
    print(args.out)


if __name__ == "__main__":
    main()
