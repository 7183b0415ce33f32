"""Summaries of rocprofv3 output for the profiles folder.

* ``stats``: the kernel-trace statistics of a run (``--kernel-trace --stats``)
  as a markdown table, with the command that produced them.  Given
  ``--kernel``, ``--groups`` and ``--bench``, it also splits that kernel's
  launches, in start order, into the bench's phases (settling, warmup, the
  event-free timed loop, the instrumented loop) and sets the trace's
  averages of the timed and instrumented loops beside the ``avg_ms`` and
  ``instrumented_avg_ms`` the bench line printed in the same process.
* ``traffic``: HBM bytes per dispatch of one kernel from a ``--pmc FETCH_SIZE``
  run and a ``--pmc WRITE_SIZE`` run of ``bench.py --profile-attn N``.  Both
  counters are calibrated against the device-to-device copy of known size
  that the profile mode ends with (each counter is scaled so that the copy
  reads, and writes, exactly its size), then averaged over the kernel's
  dispatches.  The result is written as JSON next to the source hash the
  bench compares against, so that a changed kernel does not report stale
  traffic.
* ``steps``: HBM bytes per step of the decoder stack, per kernel, from a
  ``--pmc FETCH_SIZE`` run and a ``--pmc WRITE_SIZE`` run of ``bench.py
  --workload decoder-stack --profile-stack MODE``: the dispatches of the last
  ``steps`` steps (each starts with the marker kernel; the steps end at the
  run's final 1 GiB copy), calibrated against that copy as in ``traffic``; written as JSON (with the
  kernel-source hash the bench compares against) and as a markdown table.
* ``step-times``: per-kernel durations over the same step window, from a
  ``--kernel-trace`` run of ``bench.py --workload decoder-stack
  --profile-stack MODE``: calls and average microseconds per step, and the
  step's span and busy time.
* ``matrix``: matrix-core and vector-ALU use of one kernel from a ``--pmc``
  run with GRBM_GUI_ACTIVE, SQ_VALU_MFMA_BUSY_CYCLES, SQ_VALU_MFMA_COEXEC_CYCLES,
  SQ_ACTIVE_INST_VALU and SQ_INSTS_VALU_MFMA_MOPS_BF16: the clock (GPU busy
  cycles over the dispatch's duration), the share of SIMD cycles the matrix
  core was busy, the vector ALU's share, both at once, and the matrix flops
  executed against the algorithmic count.
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


def launch_groups_md(trace, kernel, groups, bench_line=None):
    """Average duration of one kernel's launches, split in start order into
    consecutive groups of the given sizes ((name, count) pairs; a count of
    -1 takes the rest)."""
    rows = [r for r in _rows(trace, "kernel_trace.csv") if kernel in r["Kernel_Name"]]
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    us = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in rows]
    out = ["", f"Launches of `{kernel}` in start order, by phase of the run:", "",
           "| phase | launches | avg us | min us | max us |", "|---|---|---|---|---|"]
    i, avgs = 0, {}
    for name, n in groups:
        part = us[i:] if n < 0 else us[i:i + n]
        i += len(part)
        if not part:
            continue
        avgs[name] = sum(part) / len(part)
        out.append(f"| {name} | {len(part)} | {avgs[name]:.1f} | {min(part):.1f} | {max(part):.1f} |")
    if bench_line is not None:
        rl = bench_line["roofline"]
        out += ["", "The bench line printed by the same process: "
                f"`value` = {bench_line['value']:.0f} {bench_line['unit']}."]
        # avg_ms comes from the event-free timed loop (its step time less the
        # other stages); instrumented_avg_ms from events around each launch
        for key, phase, how in (("avg_ms", "timed", "timed loop, step time less the other stages"),
                                ("instrumented_avg_ms", "instrumented",
                                 "HIP events around each launch")):
            if key in rl and phase in avgs:
                ev = rl[key] * 1e3
                out.append(f"`{key}` = {ev:.1f} us ({how}); the trace's {phase} launches "
                           f"average {avgs[phase]:.1f} us ({avgs[phase] / ev:.3f} of it).")
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


def _meta(path, key="profile_attn"):
    meta = None
    for line in open(path):
        line = line.strip()
        if line.startswith("{") and key in line:
            meta = json.loads(line)
    if meta is None:
        raise SystemExit(f"no {key} line in " + path)
    return meta


def _bench_line(path):
    line = None
    for raw in open(path):
        raw = raw.strip()
        if raw.startswith("{") and '"roofline"' in raw:
            line = json.loads(raw)
    if line is None:
        raise SystemExit("no bench line in " + path)
    return line


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


def steps(fetch_dir, write_dir, marker, n_steps, copy_bytes):
    """Per-kernel calibrated bytes of the last n_steps steps (a step starts
    with the marker kernel): {counter: (scale, {kernel: [calls, bytes]})}."""
    out = {}
    for counter, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        disp = list(per_dispatch(d, counter).values())
        copies = [v for n, v in disp if "copyBuffer" in n]
        if not copies:
            raise ValueError(f"{counter}: no calibration copy")
        scale = copy_bytes / (max(copies) * 1024.0)
        # the steps end at the calibration copy (the largest one; the
        # runtime's small copies for host reads come after it)
        end = max((i for i, (n, _) in enumerate(disp) if "copyBuffer" in n), key=lambda i: disp[i][1])
        marks = [i for i, (n, _) in enumerate(disp[:end]) if marker in n]
        if len(marks) < n_steps:
            raise ValueError(f"{counter}: {len(marks)} steps found, {n_steps} asked")
        agg = collections.OrderedDict()
        for n, v in disp[marks[-n_steps]:end]:
            e = agg.setdefault(n, [0, 0.0])
            e[0] += 1
            e[1] += v * 1024.0 * scale
        out[counter] = (scale, agg)
    return out


def step_times(trace_dir, marker, n_steps):
    """Kernel-trace durations of the last n_steps steps before the calibration
    copy: (span_us, [(kernel, calls, total_us)] by total time)."""
    rows = sorted(_rows(trace_dir, "kernel_trace.csv"), key=lambda r: int(r["Start_Timestamp"]))
    # up to the calibration copy: the longest copy (the runtime's small copies
    # for host reads come after it)
    dur = lambda r: int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
    copies = [i for i, r in enumerate(rows) if "copyBuffer" in r["Kernel_Name"]]
    if copies:
        rows = rows[:max(copies, key=lambda i: dur(rows[i]))]
    marks = [i for i, r in enumerate(rows) if marker in r["Kernel_Name"]]
    if len(marks) < n_steps:
        raise ValueError(f"{len(marks)} steps found, {n_steps} asked")
    sel = rows[marks[-n_steps]:]
    agg = collections.OrderedDict()
    for r in sel:
        e = agg.setdefault(r["Kernel_Name"], [0, 0.0])
        e[0] += 1
        e[1] += (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
    span = (int(sel[-1]["End_Timestamp"]) - int(sel[0]["Start_Timestamp"])) / 1e3
    return span, sorted(((k, c, t) for k, (c, t) in agg.items()), key=lambda x: -x[2])


def per_dispatch_instances(counter_dir):
    """{dispatch id: {"name", "ns", counter: [instance values]}}"""
    acc = collections.OrderedDict()
    for r in _rows(counter_dir, "counter_collection.csv"):
        d = int(r["Dispatch_Id"])
        e = acc.setdefault(d, {"name": r["Kernel_Name"],
                               "ns": int(r["End_Timestamp"]) - int(r["Start_Timestamp"])})
        e.setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
    return acc


def _gpu_agent(counter_dir):
    for r in _rows(counter_dir, "agent_info.csv"):
        if r.get("Agent_Type") == "GPU":
            return r
    return {}


def matrix(counter_dir, kernel, flops):
    ag = _gpu_agent(counter_dir)
    xcc = int(ag.get("Num_Xcc", 8)) or 8
    simds = int(ag.get("Simd_Count", 1024)) or 1024
    cus = int(ag.get("Cu_Count", 256)) or 256
    out = []
    for d, e in per_dispatch_instances(counter_dir).items():
        if kernel not in e["name"]:
            continue
        # GRBM_GUI_ACTIVE comes summed over the XCDs: busy cycles of one XCD
        gui = sum(e["GRBM_GUI_ACTIVE"]) / xcc
        res = {"dispatch": d, "duration_us": e["ns"] / 1e3, "clock_ghz": gui / e["ns"],
               "mfma_busy_pct": 100.0 * sum(e["SQ_VALU_MFMA_BUSY_CYCLES"]) / (gui * simds),
               "mfma_and_valu_pct": 100.0 * sum(e["SQ_VALU_MFMA_COEXEC_CYCLES"]) / (gui * simds),
               "valu_busy_pct": 100.0 * sum(e["SQ_ACTIVE_INST_VALU"]) / (gui * cus)}
        if "SQ_INSTS_VALU_MFMA_MOPS_BF16" in e:
            ex = sum(e["SQ_INSTS_VALU_MFMA_MOPS_BF16"]) * 512.0
            res["mfma_flops"] = ex
            res["mfma_flops_over_algorithmic"] = ex / flops if flops else None
        out.append(res)
    if not out:
        raise ValueError(f"no {kernel} dispatch in {counter_dir}")
    return out


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("stats", help="run_kernel_stats.csv or its directory")
    s.add_argument("--title", required=True)
    s.add_argument("--command", required=True)
    s.add_argument("--out", required=True)
    s.add_argument("--kernel", help="substring of one kernel's name")
    s.add_argument("--groups", help="phase=count,... of that kernel's launches (-1: the rest)")
    s.add_argument("--bench", help="file whose last JSON line is the bench line of the same run")
    t = sub.add_parser("traffic")
    t.add_argument("--fetch", required=True, help="output directory of the FETCH_SIZE run")
    t.add_argument("--write", required=True, help="output directory of the WRITE_SIZE run")
    t.add_argument("--meta", required=True, help="the JSON line bench.py --profile-attn printed")
    t.add_argument("--kernel", default="attn_bf16")
    t.add_argument("--command", required=True)
    t.add_argument("--out", required=True)
    st = sub.add_parser("steps")
    st.add_argument("--fetch", required=True, help="output directory of the FETCH_SIZE run")
    st.add_argument("--write", required=True, help="output directory of the WRITE_SIZE run")
    st.add_argument("--meta", required=True, help="the JSON line bench.py --profile-stack printed")
    st.add_argument("--title", required=True)
    st.add_argument("--command", required=True)
    st.add_argument("--out-json", required=True)
    st.add_argument("--out-md", required=True)
    tt = sub.add_parser("step-times")
    tt.add_argument("--trace", required=True, help="output directory of the --kernel-trace run")
    tt.add_argument("--meta", required=True, help="the JSON line bench.py --profile-stack printed")
    tt.add_argument("--title", required=True)
    tt.add_argument("--command", required=True)
    tt.add_argument("--out", required=True)
    m = sub.add_parser("matrix")
    m.add_argument("--pmc", required=True, help="output directory of the --pmc run")
    m.add_argument("--meta", required=True, help="the JSON line bench.py --profile-attn printed")
    m.add_argument("--kernel", default="attn_bf16")
    m.add_argument("--command", required=True)
    m.add_argument("--out", required=True)
    a = ap.parse_args()
    if a.cmd == "step-times":
        meta = _meta(a.meta, "profile_stack")
        n = meta["steps"]
        span, ks = step_times(a.trace, meta["marker"], n)
        busy = sum(t for _, _, t in ks) / n
        md = [f"# {a.title}", "", "Command:", "", "```", a.command, "```", "",
              f"Kernel-trace durations over the last {n} steps (each starts with "
              f"`{meta['marker']}`; the run ends with a calibration copy, outside the steps). "
              f"Per step: {span / n:.1f} us from the first launch's start to the last one's end "
              f"under the tracer, {busy:.1f} us of kernel time, {sum(c for _, c, _ in ks) / n:.0f} "
              "launches.", "",
              "| kernel | calls/step | avg us | us/step |", "|---|---|---|---|"]
        for k, c, t in ks:
            name = k if len(k) <= 70 else k[:67] + "..."
            md.append(f"| `{name}` | {c / n:.1f} | {t / c:.2f} | {t / n:.1f} |")
        with open(a.out, "w") as f:
            f.write("\n".join(md) + "\n")
        print(f"span/step {span / n:.1f} us, busy/step {busy:.1f} us")
        return
    if a.cmd == "steps":
        meta = _meta(a.meta, "profile_stack")
        n = meta["steps"]
        tr = steps(a.fetch, a.write, meta["marker"], n, meta["copy_bytes"])
        fs, fa = tr["FETCH_SIZE"]
        ws, wa = tr["WRITE_SIZE"]
        kernels = []
        for name, (calls, fb) in fa.items():
            wb = wa.get(name, [calls, 0.0])[1]
            kernels.append({"kernel": name, "calls_per_step": calls / n,
                            "fetch_bytes_per_call": fb / calls, "write_bytes_per_call": wb / calls,
                            "bytes_per_step": (fb + wb) / n})
        kernels.sort(key=lambda k: -k["bytes_per_step"])
        total = sum(k["bytes_per_step"] for k in kernels)
        res = {"mode": meta["profile_stack"], "src_hash": meta["src_hash"], "command": a.command,
               "steps": n, "step_algorithmic_bytes": meta["step_algorithmic_bytes"],
               "bytes_per_step": total,
               "traffic_over_algorithmic": total / meta["step_algorithmic_bytes"],
               "fetch_scale": fs, "write_scale": ws, "kernels": kernels}
        with open(a.out_json, "w") as f:
            json.dump(res, f, indent=1)
            f.write("\n")
        md = [f"# {a.title}", "", "Command (each counter in a run of its own):", "", "```",
              a.command, "```", "",
              f"FETCH_SIZE and WRITE_SIZE per dispatch over the last {n} steps, each scaled so "
              f"that the run's final 1 GiB copy reads and writes 1 GiB (FETCH_SIZE x{fs:.3f}, "
              f"WRITE_SIZE x{ws:.3f}).", "",
              f"Per step: {total / 1e6:.1f} MB against {meta['step_algorithmic_bytes'] / 1e6:.1f} MB "
              f"algorithmic (all weights once plus each layer's KV cache): "
              f"{total / meta['step_algorithmic_bytes']:.3f}x.", "",
              "| kernel | calls/step | read MB/call | written MB/call | MB/step |",
              "|---|---|---|---|---|"]
        for k in kernels:
            name = k["kernel"] if len(k["kernel"]) <= 70 else k["kernel"][:67] + "..."
            md.append(f"| `{name}` | {k['calls_per_step']:.1f} | {k['fetch_bytes_per_call'] / 1e6:.3f} | "
                      f"{k['write_bytes_per_call'] / 1e6:.3f} | {k['bytes_per_step'] / 1e6:.1f} |")
        with open(a.out_md, "w") as f:
            f.write("\n".join(md) + "\n")
        print(json.dumps({k: v for k, v in res.items() if k != "kernels"}))
        return
    if a.cmd == "matrix":
        meta = _meta(a.meta)
        per = matrix(a.pmc, a.kernel, meta.get("attn_algorithmic_flops"))
        keys = [k for k in per[0] if k != "dispatch"]
        # the first launch of the process reads start-up cycles into its
        # busy count; the mean is over the later ones
        later = per[1:] if len(per) > 1 else per
        res = {"kernel": a.kernel, "src_hash": meta["src_hash"], "command": a.command,
               "algorithmic_flops": meta.get("attn_algorithmic_flops"), "launches": len(per),
               "mean_over": "launches 2..N" if len(per) > 1 else "launch 1",
               "mean": {k: sum(p[k] for p in later) / len(later) for k in keys},
               "per_launch": per}
        with open(a.out, "w") as f:
            json.dump(res, f, indent=1)
            f.write("\n")
        print(json.dumps(res["mean"]))
        return
    if a.cmd == "stats":
        text = kernel_stats_md(a.stats, a.title, a.command)
        if a.kernel and a.groups:
            groups = [(g.split("=")[0], int(g.split("=")[1])) for g in a.groups.split(",")]
            line = _bench_line(a.bench) if a.bench else None
            text += launch_groups_md(a.stats, a.kernel, groups, line)
        with open(a.out, "w") as f:
            f.write(text)
        return
    meta = _meta(a.meta)
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
