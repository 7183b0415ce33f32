"""Summaries of rocprofv3 output for the profiles folder.

* ``stats``: the kernel-trace statistics of a run (``--kernel-trace --stats``)
  as a markdown table, with the command that produced them.
* ``traffic``: HBM bytes per dispatch of one kernel from a ``--pmc FETCH_SIZE``
  run and a ``--pmc WRITE_SIZE`` run of ``bench.py --profile-attn N``.  Both
  counters are calibrated against the device-to-device copy of known size
  that the profile mode ends with (each counter is scaled so that the copy
  reads, and writes, exactly its size), then averaged over the kernel's
  dispatches.  The result is written as JSON next to the source hash the
  bench compares against, so that a changed kernel does not report stale
  traffic.
"""
import argparse
import collections
import csv
import glob
import json
import os


def _rows(path_or_dir, suffix):
    if os.path.isdir(path_or_dir):
        files = sorted(glob.glob(os.path.join(path_or_dir, "**", f"*{suffix}"), recursive=True))
        if not files:
            raise FileNotFoundError(f"no *{suffix} under {path_or_dir}")
        path_or_dir = files[0]
    with open(path_or_dir, newline="") as f:
        return list(csv.DictReader(f))


def kernel_stats_md(stats, title, command, limit=12):
    rows = _rows(stats, "kernel_stats.csv")
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    out = [f"# {title}", "", "Command:", "", "```", command, "```", "",
           "| kernel | calls | avg us | min us | max us | % time |", "|---|---|---|---|---|---|"]
    for r in rows[:limit]:
        name = r["Name"]
        if len(name) > 70:
            name = name[:67] + "..."
        out.append(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                   f"{float(r['MinNs']) / 1e3:.1f} | {float(r['MaxNs']) / 1e3:.1f} | "
                   f"{float(r['Percentage']):.2f} |")
    return "\n".join(out) + "\n"


def per_dispatch(counter_dir, counter):
    """{dispatch id: (kernel name, value summed over the counter's instances)}"""
    acc = collections.OrderedDict()
    for r in _rows(counter_dir, "counter_collection.csv"):
        if r["Counter_Name"] != counter:
            continue
        d = int(r["Dispatch_Id"])
        name, v = acc.get(d, (r["Kernel_Name"], 0.0))
        acc[d] = (name, v + float(r["Counter_Value"]))
    return acc


def traffic(fetch_dir, write_dir, kernel, copy_bytes):
    out = {}
    for counter, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        disp = per_dispatch(d, counter)
        copies = [v for n, v in disp.values() if "copyBuffer" in n]
        vals = [v for n, v in disp.values() if kernel in n]
        if not copies or not vals:
            raise ValueError(f"{counter}: need the copy and at least one {kernel} dispatch")
        copy_kib = max(copies)              # the large calibration copy
        scale = copy_bytes / (copy_kib * 1024.0)
        out[counter] = {"kib_per_dispatch": vals, "copy_kib": copy_kib, "scale": scale,
                        "bytes_per_dispatch": sum(vals) / len(vals) * 1024.0 * scale}
    return out


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("stats", help="run_kernel_stats.csv or its directory")
    s.add_argument("--title", required=True)
    s.add_argument("--command", required=True)
    s.add_argument("--out", required=True)
    t = sub.add_parser("traffic")
    t.add_argument("--fetch", required=True, help="output directory of the FETCH_SIZE run")
    t.add_argument("--write", required=True, help="output directory of the WRITE_SIZE run")
    t.add_argument("--meta", required=True, help="the JSON line bench.py --profile-attn printed")
    t.add_argument("--kernel", default="attn_bf16")
    t.add_argument("--command", required=True)
    t.add_argument("--out", required=True)
    a = ap.parse_args()
    if a.cmd == "stats":
        with open(a.out, "w") as f:
            f.write(kernel_stats_md(a.stats, a.title, a.command))
        return
    meta = None
    for line in open(a.meta):
        line = line.strip()
        if line.startswith("{") and "profile_attn" in line:
            meta = json.loads(line)
    if meta is None:
        raise SystemExit("no profile_attn line in " + a.meta)
    tr = traffic(a.fetch, a.write, a.kernel, meta["copy_bytes"])
    total = tr["FETCH_SIZE"]["bytes_per_dispatch"] + tr["WRITE_SIZE"]["bytes_per_dispatch"]
    res = {"kernel": a.kernel, "src_hash": meta["src_hash"], "command": a.command,
           "algorithmic_bytes": meta["attn_algorithmic_bytes"],
           "fetch_bytes_per_launch": tr["FETCH_SIZE"]["bytes_per_dispatch"],
           "write_bytes_per_launch": tr["WRITE_SIZE"]["bytes_per_dispatch"],
           "bytes_per_launch": total,
           "traffic_over_algorithmic": total / meta["attn_algorithmic_bytes"],
           "fetch_scale": tr["FETCH_SIZE"]["scale"], "write_scale": tr["WRITE_SIZE"]["scale"],
           "launches": len(tr["FETCH_SIZE"]["kib_per_dispatch"])}
    with open(a.out, "w") as f:
        json.dump(res, f, indent=1)
        f.write("\n")
    print(json.dumps(res))


if __name__ == "__main__":
    main()
