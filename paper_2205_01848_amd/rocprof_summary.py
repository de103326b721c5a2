"""Summarise rocprofv3 output of a bench.py run into profiles/.

    python -m paper_2205_01848_amd.rocprof_summary --workload c5 \\
        --stats <dir>/c5_kernel_stats.csv \\
        --fetch <dir>/fetch_counter_collection.csv --write <dir>/write_counter_collection.csv \\
        --copy-fetch <dir>/copyf_counter_collection.csv \\
        --copy-write <dir>/copyw_counter_collection.csv --copy-bytes 1073741824 \\
        --command "..." [--command "..."] --out profiles/<name>.md --json profiles/<name>.json

Byte counters are calibrated with a plain device copy of known size:
factor = copy bytes / (counter KiB * 1024) for FETCH_SIZE and WRITE_SIZE
separately, and every kernel's per-dispatch KiB is scaled by its factor.
The JSON keeps the calibrated bytes per dispatch and a hash of the HIP
sources, so bench.py reports them only while the kernels are unchanged.
"""
from __future__ import annotations

import argparse
import collections
import csv
import hashlib
import json
import os
import re

HERE = os.path.dirname(os.path.abspath(__file__))
PASS_NAMES = ["gemm_fwd_h", "gemm_fwd_y", "gemm_bwd_da", "gemm_bwd_dx", "gemm_bwd_dw2",
              "gemm_bwd_dw13", "gemm_bwd_dx"]


def source_hash() -> str:
    """sha256 over the library's HIP sources and headers (sorted by name)."""
    h = hashlib.sha256()
    csrc = os.path.join(HERE, "csrc")
    for fn in sorted(os.listdir(csrc)):
        if fn.endswith((".hip", ".hpp")):
            h.update(fn.encode())
            with open(os.path.join(csrc, fn), "rb") as f:
                h.update(f.read())
    with open(os.path.join(HERE, "..", "include", "moe.h"), "rb") as f:
        h.update(f.read())
    return h.hexdigest()[:16]


def short_name(name: str) -> str:
    # bf16 products: ffn_gemm16_kernel<MODE, PASS, Tile16<RB, CB, MINB>> (the
    # 128x128-tile instances, Tile16<4, 4, 2>, named with a _t128 suffix);
    # fp32: ffn_gemm_f32_kernel<MODE, PASS>
    m = re.search(r"ffn_gemm(16|_f32)_kernel<(\d+), (\d+)[,>]", name)
    if m:
        small = re.search(r"Tile16<4, 4, 2>", name) is not None
        return (PASS_NAMES[int(m.group(3))] + ("_f32" if m.group(1) == "_f32" else "")
                + ("_t128" if small else ""))
    # fp32 forward of small layers: ffn_gemm_f32_tiny_kernel<MODE> (modes 0, 1:
    # the first product, 2: the second)
    m = re.search(r"ffn_gemm_f32_tiny_kernel<(\d+)>", name)
    if m:
        return ("gemm_fwd_y" if m.group(1) == "2" else "gemm_fwd_h") + "_f32_tiny"
    m = re.search(r"moe::(?:\(anonymous namespace\)::)?(\w+)(<[^(]*>)?", name)
    if m:
        targs = (m.group(2) or "").replace("unsigned short", "bf16").replace("float", "f32")
        return m.group(1) + targs.replace(" ", "")
    if "Cijk_" in name:
        m = re.search(r"MT\d+x\d+x\d+_MI\d+x\d+x\d+", name)
        return "hipblaslt " + (m.group(0) if m else name[:40])
    return re.sub(r"\(.*", "", name)[:60]


def per_dispatch(path, counter):
    """{short kernel name: mean counter value per dispatch}."""
    acc = collections.defaultdict(list)
    with open(path) as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] == counter:
                acc[short_name(r["Kernel_Name"])].append(float(r["Counter_Value"]))
    return {k: sum(v) / len(v) for k, v in acc.items()}


def copy_factor(path, counter, nbytes):
    vals = []
    with open(path) as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] == counter and "copyBuffer" in r["Kernel_Name"]:
                vals.append(float(r["Counter_Value"]))
    kib = max(vals)
    return nbytes / (kib * 1024.0), kib


def counter_table(paths):
    """{short kernel name: {counter: mean value per dispatch, "_ns": mean
    duration}} over one or more counter-collection CSVs."""
    vals = collections.defaultdict(lambda: collections.defaultdict(list))
    durs = collections.defaultdict(dict)
    for path in paths:
        with open(path) as f:
            for r in csv.DictReader(f):
                n = short_name(r["Kernel_Name"])
                vals[n][r["Counter_Name"]].append(float(r["Counter_Value"]))
                key = (path, r["Dispatch_Id"])
                durs[n][key] = float(r["End_Timestamp"]) - float(r["Start_Timestamp"])
    out = {}
    for n, cs in vals.items():
        row = {c: sum(v) / len(v) for c, v in cs.items()}
        row["_ns"] = sum(durs[n].values()) / len(durs[n])
        row["_dispatches"] = len(durs[n])
        out[n] = row
    return out


def derived(row, n_xcd=8, n_simd=1024, n_cu=256):
    """Per-dispatch figures from the raw counters (values are sums over all
    instances of a counter; GRBM counters count once per XCD)."""
    d = {}
    gui = row.get("GRBM_GUI_ACTIVE")
    if gui:
        cyc = gui / n_xcd
        d["clock_GHz"] = cyc / row["_ns"]
        if "SQ_VALU_MFMA_BUSY_CYCLES" in row:
            d["mfma_busy"] = row["SQ_VALU_MFMA_BUSY_CYCLES"] / (cyc * n_simd)
        if "SQ_LDS_BANK_CONFLICT" in row:
            d["lds_conflict_of_cycles"] = row["SQ_LDS_BANK_CONFLICT"] / (cyc * n_cu)
    if row.get("SQ_WAVE_CYCLES") and "SQ_WAIT_INST_ANY" in row:
        d["wait_any_of_wave_cycles"] = row["SQ_WAIT_INST_ANY"] / row["SQ_WAVE_CYCLES"]
    if row.get("SQ_LDS_IDX_ACTIVE") and "SQ_LDS_BANK_CONFLICT" in row:
        d["lds_conflict_per_access"] = row["SQ_LDS_BANK_CONFLICT"] / max(
            row["SQ_LDS_IDX_ACTIVE"] - row["SQ_LDS_BANK_CONFLICT"], 1.0)
    hit, miss = row.get("TCC_HIT_sum"), row.get("TCC_MISS_sum")
    if hit is not None and miss is not None and hit + miss > 0:
        d["l2_hit_rate"] = hit / (hit + miss)
    if "TCC_EA0_RDREQ_sum" in row:
        d["ea_read_req"] = row["TCC_EA0_RDREQ_sum"]
    if row.get("TCP_TCC_READ_REQ_sum"):
        d["l2_read_latency_cycles"] = row["TCP_TCC_READ_REQ_LATENCY_sum"] / row["TCP_TCC_READ_REQ_sum"]
    return d


COUNTER_COLS = [("ms", "ms"), ("clock_GHz", "clock GHz"), ("mfma_busy", "MFMA busy"),
                ("wait_any_of_wave_cycles", "s_waitcnt share of wave cycles"),
                ("lds_conflict_of_cycles", "LDS bank-conflict cycles / CU cycles"),
                ("lds_conflict_per_access", "LDS conflicts per access"),
                ("l2_hit_rate", "L2 hit rate"), ("ea_read_req", "EA read requests (M)"),
                ("l2_read_latency_cycles", "L2 read latency (cycles)")]


def counters_main(a):
    tab = counter_table(a.pmc)
    lines = [f"# rocprofv3 counters: {a.workload}", "",
             "Commands (run from /tmp with TMPDIR=/tmp; R = repository root):", ""]
    lines += [f"    {c}" for c in a.command]
    lines += ["", "Each --pmc group ran in a process of its own; values are means per "
              "dispatch, sums over every instance of a counter (GRBM counters once per XCD, "
              "so cycles per XCD = GRBM_GUI_ACTIVE / 8).  clock = GRBM_GUI_ACTIVE / 8 / "
              "duration; MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (cycles x 1024 SIMDs); "
              "s_waitcnt share = SQ_WAIT_INST_ANY / SQ_WAVE_CYCLES; L2 hit rate = "
              "TCC_HIT / (TCC_HIT + TCC_MISS); L2 read latency = TCP_TCC_READ_REQ_LATENCY "
              "/ TCP_TCC_READ_REQ.", "",
              "| kernel | " + " | ".join(h for _, h in COUNTER_COLS) + " |",
              "|---" * (len(COUNTER_COLS) + 1) + "|"]
    keep = [n for n in tab if a.match is None or re.search(a.match, n)]
    keep.sort(key=lambda n: -tab[n]["_ns"])
    out = {"workload": a.workload, "source_hash": source_hash(), "kernels": {}}
    for n in keep[:a.top]:
        row = tab[n]
        d = derived(row)
        d["ms"] = row["_ns"] / 1e6
        out["kernels"][n] = {"raw": {k: v for k, v in row.items() if not k.startswith("_")},
                             "derived": d, "dispatches": row["_dispatches"]}
        cells = []
        for key, _ in COUNTER_COLS:
            v = d.get(key)
            if v is None:
                cells.append("")
            elif key == "ea_read_req":
                cells.append(f"{v / 1e6:.1f}")
            elif key in ("ms",):
                cells.append(f"{v:.3f}")
            elif key == "l2_read_latency_cycles":
                cells.append(f"{v:.0f}")
            else:
                cells.append(f"{v:.3f}")
        lines.append(f"| {n[:60]} | " + " | ".join(cells) + " |")
    mix = [n for n in keep[:a.top] if tab[n].get("SQ_INSTS_MFMA")]
    if mix:
        cols = [("SQ_INSTS_VALU", "VALU (MFMA included)"), ("SQ_INSTS_SALU", "SALU"),
                ("SQ_INSTS_VMEM_RD", "VMEM reads"), ("SQ_INSTS_LDS_LOAD", "LDS loads"),
                ("SQ_INSTS_LDS_STORE", "LDS stores"), ("SQ_INSTS", "all")]
        lines += ["", "Instructions per MFMA instruction (SQ_INSTS_* / SQ_INSTS_MFMA):", "",
                  "| kernel | MFMA (M) | " + " | ".join(h for _, h in cols) + " |",
                  "|---" * (len(cols) + 2) + "|"]
        for n in mix:
            row = tab[n]
            mf = row["SQ_INSTS_MFMA"]
            cells = [f"{row[c] / mf:.3f}" if c in row else "" for c, _ in cols]
            lines.append(f"| {n[:60]} | {mf / 1e6:.1f} | " + " | ".join(cells) + " |")
    lines += ["", f"Kernel sources hash: {out['source_hash']}", ""]
    with open(a.out, "w") as f:
        f.write("\n".join(lines))
    if a.json:
        with open(a.json, "w") as f:
            json.dump(out, f, indent=1)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--pmc", action="append", default=None,
                    help="counters mode: counter-collection CSVs (one per --pmc group)")
    ap.add_argument("--match", default=None, help="counters mode: kernel-name regex")
    ap.add_argument("--top", type=int, default=16)
    ap.add_argument("--workload", required=True)
    ap.add_argument("--stats")
    ap.add_argument("--fetch")
    ap.add_argument("--write")
    ap.add_argument("--copy-fetch")
    ap.add_argument("--copy-write")
    ap.add_argument("--copy-bytes", type=float, default=float(1 << 30))
    ap.add_argument("--command", action="append", default=[])
    ap.add_argument("--out", required=True)
    ap.add_argument("--json")
    a = ap.parse_args()
    if a.pmc:
        counters_main(a)
        return
    if not a.stats:
        ap.error("--stats is required without --pmc")

    rows = []
    with open(a.stats) as f:
        for r in csv.DictReader(f):
            rows.append((short_name(r["Name"]), int(r["Calls"]), float(r["AverageNs"]),
                         float(r["TotalDurationNs"]), float(r["Percentage"])))
    rows.sort(key=lambda r: -r[3])
    lines = [f"# rocprofv3 summary: workload {a.workload}", "",
             "Commands (run from /tmp with TMPDIR=/tmp; R = repository root):", ""]
    lines += [f"    {c}" for c in a.command]
    lines += ["", "## Kernel trace (--kernel-trace --stats)", "",
              "| kernel | calls | avg ms | total ms | % |", "|---|---|---|---|---|"]
    for n, c, avg, tot, pct in rows[:24]:
        lines.append(f"| {n} | {c} | {avg / 1e6:.4f} | {tot / 1e6:.2f} | {pct:.2f} |")
    out = {"workload": a.workload, "source_hash": source_hash(), "kernels": {}}
    if a.fetch and a.write and a.copy_fetch and a.copy_write:
        ff, fk = copy_factor(a.copy_fetch, "FETCH_SIZE", a.copy_bytes)
        wf, wk = copy_factor(a.copy_write, "WRITE_SIZE", a.copy_bytes)
        fetch = per_dispatch(a.fetch, "FETCH_SIZE")
        write = per_dispatch(a.write, "WRITE_SIZE")
        lines += ["", "## HBM traffic (--pmc FETCH_SIZE, then --pmc WRITE_SIZE; KiB per dispatch)",
                  "",
                  f"Calibration: a plain {a.copy_bytes / 2**30:.2f} GiB device copy reads "
                  f"FETCH_SIZE = {fk:.0f} KiB and WRITE_SIZE = {wk:.0f} KiB, so FETCH_SIZE is "
                  f"scaled by {ff:.3f} and WRITE_SIZE by {wf:.3f}.", "",
                  "| kernel | FETCH_SIZE KiB | WRITE_SIZE KiB | calibrated read GB | "
                  "calibrated write GB |", "|---|---|---|---|---|"]
        for n in sorted(set(fetch) & set(write), key=lambda n: -(fetch[n] + write[n])):
            rb = fetch[n] * 1024 * ff
            wb = write[n] * 1024 * wf
            out["kernels"][n] = {"read_bytes": rb, "write_bytes": wb}
            if rb + wb > 1e6:
                lines.append(f"| {n} | {fetch[n]:.0f} | {write[n]:.0f} | {rb / 1e9:.3f} | "
                             f"{wb / 1e9:.3f} |")
        out["calibration"] = {"fetch_factor": ff, "write_factor": wf}
    lines += ["", f"Kernel sources hash: {out['source_hash']}", ""]
    with open(a.out, "w") as f:
        f.write("\n".join(lines))
    if a.json:
        with open(a.json, "w") as f:
            json.dump(out, f, indent=1)


if __name__ == "__main__":
    main()
