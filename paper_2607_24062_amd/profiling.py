"""rocprofv3 summaries for the score kernels (observability, not the compute path).

Turns rocprofv3 CSV output (``--output-format csv``) into the short markdown
summaries kept under ``profiles/`` and derives the HBM traffic of a kernel
from two counter passes:

    rocprofv3 --pmc FETCH_SIZE --output-format csv -d DIR -o fetch -- python bench.py --counters
    rocprofv3 --pmc WRITE_SIZE --output-format csv -d DIR -o write -- python bench.py --counters

``bench.py --counters`` first runs a plain elementwise copy of a known size
(reads and writes ``COPY_BYTES``), so the counters, which report KiB per
dispatch, are scaled by what they read for that copy.

Command line:
    python -m paper_2607_24062_amd.profiling stats CSV TITLE COMMAND > profiles/x.md
    python -m paper_2607_24062_amd.profiling traffic FETCH_CSV WRITE_CSV TITLE COMMAND > profiles/y.md
    python -m paper_2607_24062_amd.profiling trace TRACE_CSV TITLE COMMAND [PREFIX] > profiles/z.md
    python -m paper_2607_24062_amd.profiling counters COUNTER_CSV TITLE COMMAND > profiles/w.md
"""
from __future__ import annotations

import csv
import hashlib
import json
import os
import re
import sys

COPY_BYTES = 1 << 30          # the calibration copy: 1 GiB read, 1 GiB written
COPY_KERNEL = "neg"           # it is torch.neg(out=...) on a bf16 tensor
KERNEL_SOURCES = ("csrc/score.hip", "csrc/acrl_internal.h")

_HERE = os.path.dirname(os.path.abspath(__file__))


def source_digest() -> str:
    """sha256 over the score kernel's sources: counters are stale once it changes."""
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(_HERE, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def short_name(name: str) -> str:
    n = name.replace("acrl::(anonymous namespace)::", "").replace("void ", "")
    return n.split("(")[0]


def kernel_stats(path: str):
    rows = []
    with open(path) as f:
        for r in csv.DictReader(f):
            rows.append({"name": short_name(r["Name"]), "calls": int(r["Calls"]),
                         "avg_ms": float(r["AverageNs"]) / 1e6, "min_ms": float(r["MinNs"]) / 1e6,
                         "max_ms": float(r["MaxNs"]) / 1e6, "pct": float(r["Percentage"])})
    return rows


def stats_markdown(path: str, title: str, command: str) -> str:
    out = ["# %s" % title, "", "Command (from the repository root on one MI355X):", "", "```",
           command, "```", "", "| kernel | calls | average ms | min ms | max ms | share |",
           "|---|---|---|---|---|---|"]
    for r in kernel_stats(path):
        out.append("| %s | %d | %.4f | %.4f | %.4f | %.2f%% |" % (
            r["name"], r["calls"], r["avg_ms"], r["min_ms"], r["max_ms"], r["pct"]))
    return "\n".join(out) + "\n"


def counter_means(path: str, counter: str):
    """Mean value of `counter` per dispatch, by kernel short name."""
    acc = {}
    with open(path) as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] != counter:
                continue
            acc.setdefault(short_name(r["Kernel_Name"]), []).append(float(r["Counter_Value"]))
    return {k: sum(v) / len(v) for k, v in acc.items()}


def traffic(fetch_csv: str, write_csv: str):
    """Per-dispatch HBM bytes of each acrl kernel, scaled by the copy calibration."""
    fetch = counter_means(fetch_csv, "FETCH_SIZE")
    write = counter_means(write_csv, "WRITE_SIZE")
    copy_f = [v for k, v in fetch.items() if COPY_KERNEL in k.lower()]
    copy_w = [v for k, v in write.items() if COPY_KERNEL in k.lower()]
    if not copy_f or not copy_w:
        raise RuntimeError("calibration copy kernel not found in the counter files")
    f_scale = COPY_BYTES / (copy_f[0] * 1024.0)
    w_scale = COPY_BYTES / (copy_w[0] * 1024.0)
    res = {"copy_fetch_kib": copy_f[0], "copy_write_kib": copy_w[0],
           "fetch_scale": f_scale, "write_scale": w_scale, "kernels": {}}
    for k in sorted(set(fetch) | set(write)):
        if COPY_KERNEL in k.lower():
            continue
        fb = fetch.get(k, 0.0) * 1024.0 * f_scale
        wb = write.get(k, 0.0) * 1024.0 * w_scale
        res["kernels"][k] = {"fetch_bytes": fb, "write_bytes": wb, "traffic_bytes": fb + wb}
    return res


def traffic_markdown(fetch_csv: str, write_csv: str, title: str, command: str) -> str:
    t = traffic(fetch_csv, write_csv)
    t["source_sha256"] = source_digest()
    out = ["# %s" % title, "", "Commands (from the repository root on one MI355X), one counter per pass:",
           "", "```", command, "```", "",
           "FETCH_SIZE / WRITE_SIZE are KiB per dispatch; each is scaled by its reading for a plain",
           "elementwise copy of %d bytes (fetch x%.4f, write x%.4f)." % (COPY_BYTES, t["fetch_scale"],
                                                                        t["write_scale"]),
           "", "| kernel | fetch GB | write GB | traffic GB |", "|---|---|---|---|"]
    for k, v in t["kernels"].items():
        out.append("| %s | %.3f | %.3f | %.3f |" % (k, v["fetch_bytes"] / 1e9, v["write_bytes"] / 1e9,
                                                 v["traffic_bytes"] / 1e9))
    out += ["", "Machine-readable (bench.py reads it while source_sha256 matches the kernel sources):",
            "", "```json", json.dumps(t, indent=1, sort_keys=True), "```"]
    return "\n".join(out) + "\n"


def load_traffic(md_path: str):
    """The JSON block of a traffic summary, or None if absent or stale."""
    if not os.path.exists(md_path):
        return None
    with open(md_path) as f:
        text = f.read()
    m = re.search(r"```json\n(.*?)\n```", text, re.S)
    if not m:
        return None
    t = json.loads(m.group(1))
    if t.get("source_sha256") != source_digest():
        return None
    return t


def mfma_markdown(counter_csv: str, trace_csv: str, title: str, commands: str) -> str:
    """Shader clock and matrix-core busy share per kernel, from one
    `--pmc SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE` pass and a kernel trace
    of the same command.  GRBM_GUI_ACTIVE reads the sum over the 8 XCDs, so
    clock = GUI_ACTIVE / 8 / duration; busy = MFMA_BUSY / (GUI_ACTIVE / 8 x
    1024 SIMDs); busy x clock / 2.4 GHz is the share of the MFMA peak."""
    cnt = {}
    with open(counter_csv) as f:
        for r in csv.DictReader(f):
            d = cnt.setdefault(short_name(r["Kernel_Name"]), {})
            d.setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
    dur = {}
    # durations from the kernel trace, or (trace_csv "-") from the counter
    # pass's own per-dispatch timestamps
    src = counter_csv if trace_csv == "-" else trace_csv
    seen = set()
    with open(src) as f:
        for r in csv.DictReader(f):
            key = (r.get("Dispatch_Id"), r["Kernel_Name"])
            if trace_csv == "-" and key in seen:
                continue
            seen.add(key)
            dur.setdefault(short_name(r["Kernel_Name"]), []).append(
                (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9)
    lines = ["# " + title, "", "Commands (from the repository root on one MI355X):", "", "```", commands, "```", "",
             "| kernel | dispatches | mean ms | clock GHz | MFMA busy | busy x clock / 2.4 GHz |",
             "|---|---|---|---|---|---|"]
    rows = []
    for k, d in cnt.items():
        if "GRBM_GUI_ACTIVE" not in d or "SQ_VALU_MFMA_BUSY_CYCLES" not in d or k not in dur:
            continue
        g = sum(d["GRBM_GUI_ACTIVE"]) / len(d["GRBM_GUI_ACTIVE"]) / 8.0
        m = sum(d["SQ_VALU_MFMA_BUSY_CYCLES"]) / len(d["SQ_VALU_MFMA_BUSY_CYCLES"])
        t = sum(dur[k]) / len(dur[k])
        if m <= 0 or t < 1e-3:
            continue
        clk = g / t / 1e9
        busy = m / (g * 1024.0)
        rows.append((t, "| %s | %d | %.2f | %.3f | %.1f%% | %.1f%% |" % (
            k, len(d["GRBM_GUI_ACTIVE"]), t * 1e3, clk, 100 * busy, 100 * busy * clk / 2.4)))
    lines += [r for _, r in sorted(rows, reverse=True)]
    return "\n".join(lines) + "\n"


def per_cu_markdown(counter_csv: str, title: str, command: str) -> str:
    """Per-kernel means of every counter of one `--pmc` pass, as events per
    CU-cycle: value / (GRBM_GUI_ACTIVE / 8 x 256 CUs); the pass must hold
    GRBM_GUI_ACTIVE."""
    cnt = {}
    with open(counter_csv) as f:
        for r in csv.DictReader(f):
            d = cnt.setdefault(short_name(r["Kernel_Name"]), {})
            d.setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
    names = sorted({c for d in cnt.values() for c in d if c != "GRBM_GUI_ACTIVE"})
    lines = ["# " + title, "", "Command (from the repository root on one MI355X):", "", "```", command, "```", "",
             "Values per CU-cycle (counter / (GRBM_GUI_ACTIVE / 8 x 256)).", "",
             "| kernel | GUI_ACTIVE / 8 | " + " | ".join(names) + " |",
             "|---|---|" + "---|" * len(names)]
    rows = []
    for k, d in cnt.items():
        if "GRBM_GUI_ACTIVE" not in d:
            continue
        g = sum(d["GRBM_GUI_ACTIVE"]) / len(d["GRBM_GUI_ACTIVE"]) / 8.0
        if g < 1e6:
            continue
        cells = ["%.4f" % (sum(d[c]) / len(d[c]) / (g * 256.0)) if c in d else "" for c in names]
        rows.append((g, "| %s | %.3e | %s |" % (k, g, " | ".join(cells))))
    lines += [r for _, r in sorted(rows, reverse=True)]
    return "\n".join(lines) + "\n"


def counters_markdown(counter_csv: str, title: str, command: str) -> str:
    """Per-dispatch mean of every counter of one --pmc pass, by kernel."""
    names, table = [], {}
    with open(counter_csv) as f:
        for r in csv.DictReader(f):
            c = r["Counter_Name"]
            if c not in names:
                names.append(c)
            d = table.setdefault(short_name(r["Kernel_Name"]), {})
            d.setdefault(c, []).append(float(r["Counter_Value"]))
    out = ["# %s" % title, "", "Command (from the repository root on one MI355X):", "", "```", command, "```", "",
           "Per-dispatch means.", "", "| kernel | dispatches | " + " | ".join(names) + " |",
           "|---|---|" + "---|" * len(names)]
    for k in sorted(table, key=lambda k: -max(sum(v) / len(v) for v in table[k].values())):
        n = max(len(v) for v in table[k].values())
        cells = ["%.4g" % (sum(table[k][c]) / len(table[k][c])) if c in table[k] else "" for c in names]
        out.append("| %s | %d | %s |" % (k, n, " | ".join(cells)))
    return "\n".join(out) + "\n"


def trace_rows(trace_csv: str, prefix: str = ""):
    """Per (kernel, launch size) from a --kernel-trace CSV: calls, mean,
    min and max duration (ms), for the kernels whose short name starts with
    `prefix`.  One launch size per workload and call shape, so the rows keep
    the workloads of one run apart."""
    acc = {}
    with open(trace_csv) as f:
        for r in csv.DictReader(f):
            k = short_name(r["Kernel_Name"])
            if not k.startswith(prefix):
                continue
            wg = int(r["Grid_Size_X"]) // max(int(r["Workgroup_Size_X"]), 1)
            acc.setdefault((k, wg), []).append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-6)
    return [(k, wg, len(v), sum(v) / len(v), min(v), max(v)) for (k, wg), v in acc.items()]


def trace_markdown(trace_csv: str, title: str, command: str, prefix: str = "") -> str:
    out = ["# %s" % title, "", "Command (from the repository root on one MI355X):", "", "```", command, "```", "",
           "| kernel | workgroups | calls | average ms | min ms | max ms |", "|---|---|---|---|---|---|"]
    for k, wg, n, a, lo, hi in sorted(trace_rows(trace_csv, prefix), key=lambda r: -r[2] * r[3]):
        out.append("| %s | %d | %d | %.4f | %.4f | %.4f |" % (k, wg, n, a, lo, hi))
    return "\n".join(out) + "\n"


def main(argv):
    if len(argv) >= 4 and argv[0] == "trace":
        sys.stdout.write(trace_markdown(argv[1], argv[2], argv[3], argv[4] if len(argv) > 4 else ""))
        return 0
    if len(argv) >= 4 and argv[0] == "counters":
        sys.stdout.write(counters_markdown(argv[1], argv[2], argv[3]))
        return 0
    if len(argv) >= 4 and argv[0] == "percu":
        sys.stdout.write(per_cu_markdown(argv[1], argv[2], argv[3]))
        return 0
    if len(argv) >= 5 and argv[0] == "mfma":
        sys.stdout.write(mfma_markdown(argv[1], argv[2], argv[3], argv[4]))
        return 0
    if len(argv) >= 4 and argv[0] == "stats":
        sys.stdout.write(stats_markdown(argv[1], argv[2], argv[3]))
    elif len(argv) >= 5 and argv[0] == "traffic":
        sys.stdout.write(traffic_markdown(argv[1], argv[2], argv[3], argv[4]))
    else:
        sys.stderr.write(__doc__)
        return 2
    return 0


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
