"""Summaries of rocprofv3 CSV output (``-f csv``) for the library's kernels.

  python -m paper_2510_26843_amd.profsum stats <prefix>_kernel_stats.csv [--top N]
      per-kernel calls / average / total, as a markdown table

  python -m paper_2510_26843_amd.profsum forward <prefix>_kernel_trace.csv [--launches N]
      the trace cut into forwards (each starts at an embedding launch):
      per-kernel time per forward for the forwards with N launches (default:
      the most launches), their wall time and the gaps between launches

  python -m paper_2510_26843_amd.profsum traffic --fetch F.csv --write W.csv
         --kernel REGEX --grid G --copy-bytes B [--out record.json]
      HBM bytes per dispatch of one kernel from two counter passes
      (FETCH_SIZE, then WRITE_SIZE, in KiB per dispatch), each scaled by what
      the same counter reads for the library's copy kernel (k_copy16) moving B
      bytes; the record carries the SHA-256 of the kernel source it was
      taken on.

  python -m paper_2510_26843_amd.profsum counters A.csv [B.csv ...]
         --kernel 'label=REGEX@GRID[:i/n]' [--kernel ...] [--copy-bytes B]
      mean value per dispatch of every counter in the given counter passes,
      for each listed kernel (GRID 0: any grid; :i/n keeps the matching
      dispatches whose index in dispatch order is i modulo n, e.g. the O and
      down projections, which share one kernel and grid, alternate).  With
      --copy-bytes, FETCH_SIZE and WRITE_SIZE are also given as HBM bytes,
      scaled by what they read for the copy kernel k_copy16 moving B bytes.
"""
import argparse
import collections
import csv
import hashlib
import json
import os
import re
import sys

KERNELS_SRC = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc", "kernels.hip")


def short_name(name: str) -> str:
    name = re.sub(r"\(.*$", "", name)
    return name.replace("void ", "").replace("cas::", "")


def stats_table(path: str, top: int) -> str:
    rows = list(csv.DictReader(open(path)))
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    out = ["| kernel | calls | avg us | min us | max us | total ms | % |", "|---|---:|---:|---:|---:|---:|---:|"]
    for r in rows[:top]:
        out.append(f"| `{short_name(r['Name'])}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                   f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | "
                   f"{float(r['TotalDurationNs']) / 1e6:.3f} | {float(r['Percentage']):.1f} |")
    return "\n".join(out)


def forward_table(path: str, launches: int) -> str:
    rows = list(csv.DictReader(open(path)))
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    fwds, cur = [], None
    for r in rows:
        n = short_name(r["Kernel_Name"])
        if n.startswith("k_embed"):
            cur = []
            fwds.append(cur)
        if cur is not None and not n.startswith(("k_tile", "__amd")):
            wg = int(r["Workgroup_Size_X"]) * int(r["Workgroup_Size_Y"]) * int(r["Workgroup_Size_Z"])
            grid = (int(r["Grid_Size_X"]) * int(r["Grid_Size_Y"]) * int(r["Grid_Size_Z"])) // max(wg, 1)
            cur.append((n, grid, int(r["Start_Timestamp"]), int(r["End_Timestamp"])))
    by_len = collections.defaultdict(list)
    for f in fwds:
        by_len[len(f)].append(f)
    if not by_len:
        return "no forwards in the trace"
    n = launches or max(by_len)
    sel = by_len.get(n, [])
    if not sel:
        return f"no forward with {n} launches; counts seen: {sorted(by_len)}"
    wall = sum(f[-1][3] - f[0][2] for f in sel) / len(sel) / 1e3
    busy = sum(sum(e - s for _, _, s, e in f) for f in sel) / len(sel) / 1e3
    agg = collections.OrderedDict()
    for f in sel:
        for name, grid, s, e in f:
            a = agg.setdefault((name, grid), [0, 0.0])
            a[0] += 1
            a[1] += (e - s) / 1e3
    out = [f"{len(sel)} forwards of {n} launches: wall {wall:.1f} us (first to last launch), kernels "
           f"{busy:.1f} us, gaps {wall - busy:.1f} us", "",
           "| kernel | workgroups | launches/forward | avg us | us/forward |", "|---|---:|---:|---:|---:|"]
    for (name, grid), (c, t) in sorted(agg.items(), key=lambda kv: -kv[1][1]):
        out.append(f"| `{name}` | {grid} | {c / len(sel):.0f} | {t / c:.2f} | {t / len(sel):.1f} |")
    return "\n".join(out)


def counter_means(path: str, counter: str):
    """(kernel name, grid size) -> list of counter values (KiB per dispatch)."""
    agg = collections.defaultdict(list)
    for r in csv.DictReader(open(path)):
        if r["Counter_Name"] == counter:
            agg[(r["Kernel_Name"], int(r["Grid_Size"]))].append(float(r["Counter_Value"]))
    return agg


def pick(agg, regex: str, grid: int):
    vals = [v for (k, g), vs in agg.items() if re.search(regex, k) and (grid == 0 or g == grid) for v in vs]
    if not vals:
        raise SystemExit(f"no dispatch of /{regex}/ with grid {grid}")
    return sum(vals) / len(vals), len(vals)


def traffic(args) -> dict:
    f = counter_means(args.fetch, "FETCH_SIZE")
    w = counter_means(args.write, "WRITE_SIZE")
    cf, ncf = pick(f, r"k_copy16", 0)
    cw, ncw = pick(w, r"k_copy16", 0)
    kf, nkf = pick(f, args.kernel, args.grid)
    kw, nkw = pick(w, args.kernel, args.grid)
    sf = args.copy_bytes / (cf * 1024.0)
    sw = args.copy_bytes / (cw * 1024.0)
    fetch_b = kf * 1024.0 * sf
    write_b = kw * 1024.0 * sw
    with open(KERNELS_SRC, "rb") as fh:
        sha = hashlib.sha256(fh.read()).hexdigest()
    return {"kernel": args.kernel, "grid_size": args.grid, "dispatches": [nkf, nkw],
            "fetch_kib_per_dispatch": round(kf, 3), "write_kib_per_dispatch": round(kw, 3),
            "copy_bytes": args.copy_bytes, "copy_fetch_kib": round(cf, 3), "copy_write_kib": round(cw, 3),
            "fetch_scale": round(sf, 5), "write_scale": round(sw, 5),
            "hbm_fetch_bytes_per_launch": round(fetch_b), "hbm_write_bytes_per_launch": round(write_b),
            "hbm_bytes_per_launch": round(fetch_b + write_b), "kernels_sha256": sha}


def _kernel_spec(spec: str):
    label, rest = spec.split("=", 1)
    regex, grid = rest.rsplit("@", 1)
    sel = None
    if ":" in grid:
        grid, sel = grid.split(":")
        i, n = sel.split("/")
        sel = (int(i), int(n))
    return label, regex, int(grid), sel


def counter_table(paths, specs, copy_bytes=0) -> str:
    """Mean value per dispatch of each counter, per listed kernel."""
    rows = []
    for p in paths:
        rows += list(csv.DictReader(open(p)))
    counters = sorted({r["Counter_Name"] for r in rows})
    # dispatch order per (counter, kernel, grid)
    per = collections.defaultdict(list)
    for r in rows:
        per[(r["Counter_Name"], r["Kernel_Name"], int(r["Grid_Size"]))].append(
            (int(r.get("Dispatch_Id", 0) or 0), float(r["Counter_Value"])))
    scale = {}
    if copy_bytes:
        for c in ("FETCH_SIZE", "WRITE_SIZE"):
            vals = [v for (cn, k, g), vs in per.items() if cn == c and "k_copy16" in k for _, v in vs]
            if vals:
                scale[c] = copy_bytes / (sum(vals) / len(vals) * 1024.0)
    head = ["kernel", "dispatches"] + counters + [f"{c} bytes" for c in ("FETCH_SIZE", "WRITE_SIZE") if c in scale]
    out = ["| " + " | ".join(head) + " |", "|" + "---|" * len(head)]
    for spec in specs:
        label, regex, grid, sel = _kernel_spec(spec)
        cells, nd = [], 0
        means = {}
        for c in counters:
            vals = []
            for (cn, k, g), vs in per.items():
                if cn == c and re.search(regex, k) and (grid == 0 or g == grid):
                    vals += vs
            vals.sort()
            if sel:
                vals = [v for j, v in enumerate(vals) if j % sel[1] == sel[0]]
            nd = max(nd, len(vals))
            means[c] = sum(v for _, v in vals) / len(vals) if vals else None
            cells.append("—" if means[c] is None else f"{means[c]:.4g}")
        extra = [f"{means[c] * 1024.0 * scale[c]:,.0f}" if means.get(c) is not None else "—"
                 for c in ("FETCH_SIZE", "WRITE_SIZE") if c in scale]
        out.append(f"| {label} | {nd} | " + " | ".join(cells + extra) + " |")
    if scale:
        out.append("")
        out.append("Calibration (copy kernel): " + ", ".join(f"{c} scale {v:.4f}" for c, v in scale.items()))
    return "\n".join(out)


def main(argv=None):
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("csv")
    s.add_argument("--top", type=int, default=25)
    fw = sub.add_parser("forward")
    fw.add_argument("csv")
    fw.add_argument("--launches", type=int, default=0)
    t = sub.add_parser("traffic")
    t.add_argument("--fetch", required=True)
    t.add_argument("--write", required=True)
    t.add_argument("--kernel", required=True)
    t.add_argument("--grid", type=int, default=0)
    t.add_argument("--copy-bytes", type=int, required=True)
    t.add_argument("--out")
    c = sub.add_parser("counters")
    c.add_argument("csv", nargs="+")
    c.add_argument("--kernel", action="append", required=True)
    c.add_argument("--copy-bytes", type=int, default=0)
    a = ap.parse_args(argv)
    if a.cmd == "stats":
        print(stats_table(a.csv, a.top))
    elif a.cmd == "forward":
        print(forward_table(a.csv, a.launches))
    elif a.cmd == "counters":
        print(counter_table(a.csv, a.kernel, a.copy_bytes))
    else:
        rec = traffic(a)
        txt = json.dumps(rec, indent=1)
        if a.out:
            with open(a.out, "w") as fh:
                fh.write(txt + "\n")
        print(txt)


if __name__ == "__main__":
    sys.exit(main())
