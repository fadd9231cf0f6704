"""Summaries of rocprofv3 runs of bench.py for profiles/.

    python -m paper_2010_14298_amd.profiling trace  <trace_dir> <out.md> "<command>"
    python -m paper_2010_14298_amd.profiling traffic <fetch_dir> <write_dir> <out.txt> "<commands>"
    python -m paper_2010_14298_amd.profiling counters <out.json> "<commands>" <pmc_dir> [<pmc_dir> ...]

`trace` reads the kernel-trace CSV of `rocprofv3 --kernel-trace --stats
--output-format csv` and writes per-kernel call counts and average / total
durations.  `counters` averages every counter of the given `rocprofv3 --pmc` passes per
kernel (and the derived VALUBusy / MfmaUtil when a pass collected them),
with the hash of the kernel sources.  `traffic` reads two `rocprofv3 --pmc FETCH_SIZE` / `--pmc
WRITE_SIZE` runs (KiB per dispatch), calibrates each counter on the plain
elementwise pass that `bench.py --copy-probe` launches (known bytes read and
written), and writes the scaled HBM bytes per dispatch of every kernel, with
the hash of the kernel sources they were taken on.
"""
import csv
import glob
import hashlib
import json
import os
import sys
from collections import defaultdict

HERE = os.path.dirname(os.path.abspath(__file__))
COPY_BYTES = 256 * 1024 * 1024   # bench.py --copy-probe: 256 MiB read + 256 MiB written per pass


def source_hash():
    """sha256 over the HIP sources, to tell whether counters match the current kernels."""
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(HERE, "csrc", "*"))):
        with open(f, "rb") as fh:
            h.update(os.path.basename(f).encode())
            h.update(fh.read())
    return h.hexdigest()[:16]


def _short(name):
    name = name.replace("void ", "").replace("(anonymous namespace)::", "")
    return name.split("(")[0][:90]


def _find(dirpath, suffix):
    hits = glob.glob(os.path.join(dirpath, "**", "*" + suffix), recursive=True)
    if not hits:
        raise FileNotFoundError(f"no *{suffix} under {dirpath}")
    return hits[0]


def trace(trace_dir, out, command):
    rows = list(csv.DictReader(open(_find(trace_dir, "kernel_trace.csv"))))
    agg = defaultdict(list)
    for r in rows:
        agg[_short(r["Kernel_Name"])].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    lines = [f"# Kernel trace: {os.path.basename(out)}", "", f"Command: `{command}`", "",
             f"Kernel sources: {source_hash()}", "",
             "| kernel | calls | avg us | total us |", "|---|---:|---:|---:|"]
    for k, v in sorted(agg.items(), key=lambda kv: -sum(kv[1])):
        lines.append(f"| `{k}` | {len(v)} | {sum(v) / len(v):.2f} | {sum(v):.1f} |")
    with open(out, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def _counter(dirpath, name):
    rows = list(csv.DictReader(open(_find(dirpath, "counter_collection.csv"))))
    agg = defaultdict(list)
    for r in rows:
        if r["Counter_Name"] == name:
            agg[_short(r["Kernel_Name"])].append(float(r["Counter_Value"]))
    return {k: sum(v) / len(v) for k, v in agg.items()}


def traffic(fetch_dir, write_dir, out, command):
    fetch = _counter(fetch_dir, "FETCH_SIZE")
    write = _counter(write_dir, "WRITE_SIZE")
    # the elementwise pass of bench.py --copy-probe (torch's neg kernel: 256 MiB in, 256 MiB out);
    # host transfers (rocclr copy kernels) read over PCIe and are not a calibration
    copy = [k for k in fetch if k.startswith("at::native") and "neg" in k]
    if not copy:
        raise RuntimeError("no device copy kernel in the FETCH_SIZE run (bench.py --copy-probe)")
    ck = max(copy, key=lambda k: fetch[k])
    f_read = COPY_BYTES / (fetch[ck] * 1024.0)
    f_write = COPY_BYTES / (write[ck] * 1024.0)
    kernels = {}
    for k in fetch:
        if k == ck:
            continue
        rb = fetch[k] * 1024.0 * f_read
        wb = write.get(k, 0.0) * 1024.0 * f_write
        kernels[k] = {"read_bytes": round(rb), "write_bytes": round(wb), "bytes": round(rb + wb)}
    res = {"command": command, "kernel_sources": source_hash(), "copy_kernel": ck,
           "copy_bytes_each_way": COPY_BYTES, "fetch_scale": round(f_read, 4), "write_scale": round(f_write, 4),
           "kernels": kernels}
    with open(out, "w") as f:
        json.dump(res, f, indent=1)
    print(json.dumps(res, indent=1))


def counters(out, command, dirs):
    kernels = defaultdict(dict)
    for d in dirs:
        rows = list(csv.DictReader(open(_find(d, "counter_collection.csv"))))
        agg = defaultdict(lambda: defaultdict(list))
        for r in rows:
            agg[_short(r["Kernel_Name"])][r["Counter_Name"]].append(float(r["Counter_Value"]))
        for k, cs in agg.items():
            for c, v in cs.items():
                kernels[k][c] = round(sum(v) / len(v), 4)
    res = {"command": command, "kernel_sources": source_hash(), "passes": len(dirs), "kernels": kernels}
    with open(out, "w") as f:
        json.dump(res, f, indent=1)
    print(json.dumps(res, indent=1))


if __name__ == "__main__":
    if sys.argv[1] == "counters":
        counters(sys.argv[2], sys.argv[3], sys.argv[4:])
    elif sys.argv[1] == "trace":
        trace(sys.argv[2], sys.argv[3], sys.argv[4])
    elif sys.argv[1] == "traffic":
        traffic(sys.argv[2], sys.argv[3], sys.argv[4], sys.argv[5])
    else:
        raise SystemExit(__doc__)
