"""Reduces rocprofv3 output to the short text summaries kept with the measurements.

    python -m paper_2606_24957_amd.rocprof_summary stats DIR --command CMD
        per-kernel launch counts and durations from a `--kernel-trace --stats` run
    python -m paper_2606_24957_amd.rocprof_summary traffic --fetch DIR --write DIR \\
            --kernel NAME --copy-bytes N --command CMD [--json-out FILE]
        HBM bytes per launch of the kernels whose name contains NAME, from one
        `--pmc FETCH_SIZE` and one `--pmc WRITE_SIZE` run over the same program.  Each
        counter is scaled by what it reads for the largest copy-kernel dispatch of the run
        (a plain device copy of N bytes: N read and N written).

Both print Markdown; `traffic` ends with an HTML comment holding the JSON record that
bench.py reads.
"""
import argparse
import collections
import csv
import glob
import hashlib
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
KERNEL_SOURCES = ("attn.hip", "common.hpp", "kernels.hpp")


def kernel_sources_sha() -> str:
    """First 16 hex digits of the sha256 over the sparse-attention kernel sources."""
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2606_24957_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def _short(name: str, width: int = 72) -> str:
    name = name.replace("(anonymous namespace)::", "")
    return name if len(name) <= width else name[: width - 3] + "..."


def _files(d, suffix):
    out = sorted(glob.glob(os.path.join(d, "**", "*" + suffix), recursive=True))
    if not out:
        raise SystemExit(f"no *{suffix} under {d}")
    return out


def stats(d, command, top=20):
    rows = []
    for path in _files(d, "kernel_stats.csv"):
        rows += list(csv.DictReader(open(path)))
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    total = sum(float(r["TotalDurationNs"]) for r in rows)
    print(f"Command: `{command}`\n")
    print("| kernel | calls | avg us | min us | max us | share |")
    print("|---|---:|---:|---:|---:|---:|")
    for r in rows[:top]:
        print(f"| `{_short(r['Name'])}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
              f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | "
              f"{100 * float(r['TotalDurationNs']) / total:.1f}% |")


def _per_dispatch(d, counter):
    """{dispatch id: (kernel name, value)} for one counter (summed over its instances)."""
    vals, names = collections.defaultdict(float), {}
    for path in _files(d, "counter_collection.csv"):
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            key = (path, r["Dispatch_Id"])
            vals[key] += float(r["Counter_Value"])
            names[key] = r["Kernel_Name"]
    return {k: (names[k], v) for k, v in vals.items()}


def traffic(fetch_dir, write_dir, kernel, copy_bytes, command, json_out=None):
    fetch = _per_dispatch(fetch_dir, "FETCH_SIZE")
    write = _per_dispatch(write_dir, "WRITE_SIZE")

    def copy_factor(per, counter):
        copies = [v for n, v in per.values() if "copyBuffer" in n or "copy_kernel" in n]
        if not copies or max(copies) <= 0:
            raise SystemExit(f"no copy dispatch with {counter} in the run")
        return copy_bytes / (max(copies) * 1024.0), max(copies)

    fr, fcopy = copy_factor(fetch, "FETCH_SIZE")
    fw, wcopy = copy_factor(write, "WRITE_SIZE")
    by_kernel = collections.defaultdict(lambda: ([], []))
    for n, v in fetch.values():
        if kernel in n:
            by_kernel[n][0].append(v)
    for n, v in write.values():
        if kernel in n:
            by_kernel[n][1].append(v)
    if not by_kernel:
        raise SystemExit(f"no dispatch of a kernel named like {kernel!r}")
    print(f"Commands: `{command}`\n")
    print(f"Copy calibration ({copy_bytes} B device copy): FETCH_SIZE reads {fcopy:.0f} KiB "
          f"-> factor {fr:.3f}; WRITE_SIZE reads {wcopy:.0f} KiB -> factor {fw:.3f}.\n")
    print("| kernel | launches | FETCH_SIZE KiB | WRITE_SIZE KiB | read MB | written MB | total MB |")
    print("|---|---:|---:|---:|---:|---:|---:|")
    best = None
    for n, (fv, wv) in sorted(by_kernel.items()):
        f = sum(fv) / max(1, len(fv))
        w = sum(wv) / max(1, len(wv))
        rd, wr = f * 1024 * fr, w * 1024 * fw
        print(f"| `{_short(n)}` | {len(fv)} | {f:.0f} | {w:.0f} | {rd / 1e6:.2f} | {wr / 1e6:.2f} | "
              f"{(rd + wr) / 1e6:.2f} |")
        if best is None or len(fv) > best[0]:
            best = (len(fv), n, rd + wr, rd, wr)
    rec = {"kernel": _short(best[1], 200), "bytes_per_launch": round(best[2]),
           "read_bytes": round(best[3]), "write_bytes": round(best[4]),
           "fetch_factor": round(fr, 4), "write_factor": round(fw, 4),
           "source_sha256": kernel_sources_sha()}
    print(f"\n<!-- traffic: {json.dumps(rec)} -->")
    if json_out:
        with open(json_out, "w") as fh:
            json.dump(rec, fh)


def main(argv=None):
    p = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    sub = p.add_subparsers(dest="what", required=True)
    s = sub.add_parser("stats")
    s.add_argument("dir")
    s.add_argument("--command", required=True)
    s.add_argument("--top", type=int, default=20)
    t = sub.add_parser("traffic")
    t.add_argument("--fetch", required=True)
    t.add_argument("--write", required=True)
    t.add_argument("--kernel", required=True)
    t.add_argument("--copy-bytes", type=int, required=True)
    t.add_argument("--command", required=True)
    t.add_argument("--json-out")
    a = p.parse_args(argv)
    if a.what == "stats":
        stats(a.dir, a.command, a.top)
    else:
        traffic(a.fetch, a.write, a.kernel, a.copy_bytes, a.command, a.json_out)


if __name__ == "__main__":
    sys.exit(main())
