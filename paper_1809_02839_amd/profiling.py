"""Summaries of rocprofv3 output for the stage kernels.

Two summaries, written as short markdown files:

* kernel time: the per-kernel table of a `rocprofv3 --kernel-trace --stats
  --output-format csv` run (`*_kernel_stats.csv`);
* HBM traffic: per-dispatch `FETCH_SIZE` and `WRITE_SIZE` (KiB, from two
  `rocprofv3 --pmc` runs) scaled to bytes by what the same counters read for a
  reference copy dispatch of known size (the first dispatch whose kernel name
  contains the calibration marker). The file records a digest of the kernel
  sources the counters were taken with; a reader compares it with the current
  sources and treats the figures as stale when they differ.

* matrix-core activity: per-kernel means of one `--pmc` run over
  `SQ_VALU_MFMA_BUSY_CYCLES` (and any other counters), with the MFMA-busy
  fraction = MFMA busy cycles / (dispatch duration x 2.4 GHz x 1024 SIMDs),
  the duration taken from the dispatch's own start and end timestamps.

Command line:

    python -m paper_1809_02839_amd.profiling stats <kernel_stats.csv> <out.md> --title T --command C
    python -m paper_1809_02839_amd.profiling traffic <fetch_dir> <write_dir> <out.md>
        --calib-bytes B --calib-marker neg --title T --command C
    python -m paper_1809_02839_amd.profiling counters <pmc_dir> [<pmc_dir> ...] <out.md> --title T --command C
"""
import argparse
import csv
import glob
import hashlib
import os
import re

CSRC = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc")


def _code_only(text):
    """C++ source text without comments and with whitespace runs collapsed (a
    comment edit leaves the built kernels, and so the measurements, as they
    were). String and character literals are kept whole."""
    out, i, n = [], 0, len(text)
    while i < n:
        c = text[i]
        if c in "\"'":
            j = i + 1
            while j < n and text[j] != c:
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        elif text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def source_digest():
    """SHA-256 over the code of every kernel source and header (comments and
    whitespace ignored), in name order."""
    h = hashlib.sha256()
    for p in sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.hpp"))):
        h.update(os.path.basename(p).encode())
        with open(p, encoding="utf-8") as f:
            h.update(_code_only(f.read()).encode())
    return h.hexdigest()[:16]


def short_name(kernel):
    """`void ns::(anonymous namespace)::k<1, 0, true>(args)` -> `k<1, 0, true>`."""
    name = kernel.strip()
    if name.startswith("void "):
        name = name[5:]
    depth, cut = 0, len(name)
    for i, ch in enumerate(name):     # cut at the argument list (the first '(' outside <...>)
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0 and not name.startswith("(anonymous", i):
            cut = i
            break
    name = name[:cut].replace("(anonymous namespace)::", "")
    lt = name.find("<")
    head, tail = (name, "") if lt < 0 else (name[:lt], name[lt:])
    return re.sub(r"^.*::", "", head) + tail


def _counter_rows(run_dir):
    files = glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise FileNotFoundError(f"no counter_collection.csv under {run_dir}")
    rows = []
    for f in files:
        with open(f, newline="") as fh:
            rows.extend(csv.DictReader(fh))
    return rows


def counter_per_dispatch(run_dir, counter):
    """{dispatch id: (kernel name, summed counter value)} of one --pmc run."""
    out = {}
    for r in _counter_rows(run_dir):
        if r["Counter_Name"] != counter:
            continue
        d = int(r["Dispatch_Id"])
        name, v = out.get(d, (r["Kernel_Name"], 0.0))
        out[d] = (name, v + float(r["Counter_Value"]))
    return out


def traffic_table(fetch_dir, write_dir, calib_bytes, marker):
    """Per kernel: dispatches, mean FETCH/WRITE KiB, scale factors, mean bytes per dispatch."""
    fetch = counter_per_dispatch(fetch_dir, "FETCH_SIZE")
    write = counter_per_dispatch(write_dir, "WRITE_SIZE")

    def calib(table):
        for d in sorted(table):
            if marker in table[d][0]:
                return table[d][1]
        raise ValueError(f"no dispatch named like '{marker}'")
    f_read = calib_bytes / (calib(fetch) * 1024.0)
    f_write = calib_bytes / (calib(write) * 1024.0)

    def means(table):
        acc = {}
        for d, (name, v) in table.items():
            if marker in name:
                continue
            k = short_name(name)
            n, s = acc.get(k, (0, 0.0))
            acc[k] = (n + 1, s + v)
        return {k: (n, s / n) for k, (n, s) in acc.items()}
    mf, mw = means(fetch), means(write)
    rows = []
    for k in sorted(mf, key=lambda k: -mf[k][1]):
        if k not in mw:
            continue
        n, fk = mf[k]
        wk = mw[k][1]
        rows.append({"kernel": k, "dispatches": n, "fetch_kib": fk, "write_kib": wk,
                     "bytes": fk * 1024.0 * f_read + wk * 1024.0 * f_write})
    return rows, f_read, f_write


def write_traffic(out_md, rows, f_read, f_write, calib_bytes, title, command):
    with open(out_md, "w") as f:
        f.write(f"# {title}\n\n")
        f.write("Commands (from the repository root, one counter per run):\n\n```\n" + command.strip() + "\n```\n\n")
        f.write(f"Reference copy: {calib_bytes} bytes read and written; scale FETCH_SIZE x {f_read:.4f}, "
                f"WRITE_SIZE x {f_write:.4f} (bytes per KiB-count / 1024).\n\n")
        f.write(f"source digest: {source_digest()}\n\n")
        f.write("| kernel | dispatches | FETCH_SIZE KiB | WRITE_SIZE KiB | HBM bytes / dispatch |\n")
        f.write("|:--|--:|--:|--:|--:|\n")
        for r in rows:
            f.write(f"| {r['kernel']} | {r['dispatches']} | {r['fetch_kib']:.1f} | {r['write_kib']:.1f} | "
                    f"{r['bytes']:.0f} |\n")


def read_traffic(md_path, with_dispatches=False):
    """(digest, {kernel: bytes per dispatch}) from a traffic summary, or (None, {});
    with_dispatches: the values are (dispatches, bytes per dispatch)."""
    if not os.path.exists(md_path):
        return None, {}
    digest, table = None, {}
    with open(md_path) as f:
        for line in f:
            if line.startswith("source digest:"):
                digest = line.split(":", 1)[1].strip()
            elif line.startswith("| ") and not line.startswith("| kernel"):
                cells = [c.strip() for c in line.strip().strip("|").split("|")]
                if len(cells) == 5:
                    table[cells[0]] = (int(cells[1]), float(cells[4])) if with_dispatches else float(cells[4])
    return digest, table


SIMDS = 256 * 4          # MI355X: 256 compute units of four SIMDs
NOMINAL_CLOCK_HZ = 2.4e9  # the clock of the published peaks
DURATION = "duration ns"


def counter_means(run_dir):
    """{kernel short name: (dispatches, {counter: mean per dispatch})} of one
    --pmc run; the pseudo-counter DURATION is the mean dispatch duration."""
    per = {}
    names = {}
    for r in _counter_rows(run_dir):
        d = int(r["Dispatch_Id"])
        key = (d, r["Counter_Name"])
        per[key] = per.get(key, 0.0) + float(r["Counter_Value"])
        names[d] = short_name(r["Kernel_Name"])
        if "Start_Timestamp" in r and "End_Timestamp" in r:
            per[(d, DURATION)] = float(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
    acc = {}
    for (d, c), v in per.items():
        k = names[d]
        ds, sums = acc.setdefault(k, (set(), {}))
        ds.add(d)
        sums[c] = sums.get(c, 0.0) + v
    return {k: (len(ds), {c: v / len(ds) for c, v in sums.items()}) for k, (ds, sums) in acc.items()}


def write_counters(run_dirs, out_md, title, command, notes=""):
    """One table over one or more --pmc runs (each run's counters merged per kernel)."""
    table = {}
    for run_dir in ([run_dirs] if isinstance(run_dirs, str) else run_dirs):
        for k, (n, cs) in counter_means(run_dir).items():
            n0, cs0 = table.get(k, (n, {}))
            table[k] = (max(n0, n), {**cs0, **cs})
    counters = sorted({c for _, cs in table.values() for c in cs})
    mfma = "SQ_VALU_MFMA_BUSY_CYCLES" in counters and DURATION in counters
    with open(out_md, "w") as f:
        f.write(f"# {title}\n\n")
        f.write("Command (from the repository root):\n\n```\n" + command.strip() + "\n```\n\n")
        if notes:
            f.write(notes.strip() + "\n\n")
        f.write(f"source digest: {source_digest()}\n\n")
        head = ["kernel", "dispatches"] + [f"{c} / dispatch" for c in counters] + (["MFMA busy %"] if mfma else [])
        f.write("| " + " | ".join(head) + " |\n")
        f.write("|:--|" + "--:|" * (len(head) - 1) + "\n")
        order = sorted(table, key=lambda k: -table[k][1].get(DURATION, 0.0) * table[k][0])
        for k in order:
            n, cs = table[k]
            cells = [k, str(n)] + [f"{cs.get(c, 0.0):.4g}" for c in counters]
            if mfma:
                cyc = cs.get(DURATION, 0.0) * 1e-9 * NOMINAL_CLOCK_HZ * SIMDS
                cells.append(f"{100.0 * cs.get('SQ_VALU_MFMA_BUSY_CYCLES', 0.0) / cyc:.1f}" if cyc else "")
            f.write("| " + " | ".join(cells) + " |\n")


def write_stats(stats_csv, out_md, title, command, notes=""):
    with open(stats_csv, newline="") as fh:
        rows = list(csv.DictReader(fh))
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    with open(out_md, "w") as f:
        f.write(f"# {title}\n\n")
        f.write("Command (from the repository root):\n\n```\n" + command.strip() + "\n```\n\n")
        if notes:
            f.write(notes.strip() + "\n\n")
        f.write(f"source digest: {source_digest()}\n\n")
        f.write("| kernel | calls | total ns | average ns | percent | min ns | max ns |\n")
        f.write("|:--|--:|--:|--:|--:|--:|--:|\n")
        for r in rows:
            f.write(f"| {short_name(r['Name'])} | {r['Calls']} | {r['TotalDurationNs']} | "
                    f"{float(r['AverageNs']):.0f} | {float(r['Percentage']):.2f} | {r['MinNs']} | {r['MaxNs']} |\n")


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    sub = ap.add_subparsers(dest="cmd", required=True)
    a = sub.add_parser("stats")
    a.add_argument("stats_csv")
    a.add_argument("out_md")
    a.add_argument("--title", required=True)
    a.add_argument("--command", required=True)
    a.add_argument("--notes", default="")
    b = sub.add_parser("traffic")
    b.add_argument("fetch_dir")
    b.add_argument("write_dir")
    b.add_argument("out_md")
    b.add_argument("--calib-bytes", type=int, required=True)
    b.add_argument("--calib-marker", default="neg")
    b.add_argument("--title", required=True)
    b.add_argument("--command", required=True)
    c = sub.add_parser("counters")
    c.add_argument("pmc_dir", nargs="+")
    c.add_argument("out_md")
    c.add_argument("--title", required=True)
    c.add_argument("--command", required=True)
    c.add_argument("--notes", default="")
    args = ap.parse_args()
    if args.cmd == "stats":
        write_stats(args.stats_csv, args.out_md, args.title, args.command, args.notes)
    elif args.cmd == "counters":
        write_counters(args.pmc_dir, args.out_md, args.title, args.command, args.notes)
    else:
        rows, fr, fw = traffic_table(args.fetch_dir, args.write_dir, args.calib_bytes, args.calib_marker)
        write_traffic(args.out_md, rows, fr, fw, args.calib_bytes, args.title, args.command)
    print(f"wrote {args.out_md}")


if __name__ == "__main__":
    main()
