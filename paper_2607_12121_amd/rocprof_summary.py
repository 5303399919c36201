"""Short text summaries of rocprofv3 output, for the figures kept beside the code.

    python -m paper_2607_12121_amd.rocprof_summary stats  <kernel_stats.csv> --title T --cmd C
    python -m paper_2607_12121_amd.rocprof_summary traffic --fetch <fetch counter_collection.csv>
        --write <write counter_collection.csv> --kernel REGEX --copy-kernel REGEX
        --copy-bytes S --source FILE [FILE ...] --title T --cmd C [--cmd C ...]
    python -m paper_2607_12121_amd.rocprof_summary grids <kernel_trace.csv> --title T --cmd C
        [--include REGEX] [--bytes REGEX@GRID=BYTES ...] [--peak-gbs P]

`stats` turns a `--kernel-trace --stats` kernel table into a markdown table.

`grids` groups a `--kernel-trace` table by kernel and grid size (one line per
launch shape) with the median, minimum and mean duration; a `--bytes` entry gives
the algorithmic bytes of the launches of one kernel and grid, from which GB/s
and the fraction of the peak follow.

`mfma` turns one `--pmc` pass (SQ_INSTS_MFMA, SQ_VALU_MFMA_BUSY_CYCLES,
GRBM_GUI_ACTIVE) into MFMA figures per kernel and launch shape (launches of one
kernel grouped by their MFMA instruction count): the flops the MFMA instructions
performed, the ratio of the algorithmic flops to them (the rest is tile padding),
the clock under load (GRBM active cycles of one XCD over the duration), the MFMA
pipes' busy share of the SIMD cycles at that clock, and the achieved fraction of
the nominal bf16 peak.

`traffic` turns two `--pmc` passes (FETCH_SIZE, then WRITE_SIZE; both in KiB per
dispatch) into HBM bytes per launch of one kernel (with further `--kernel`
regexes: plus the kernels that follow it in the same launch, such as a merge
pass; with --grid, only launches of that size).  Each counter is scaled by
what it reads for a plain copy kernel of S bytes launched in the same run (the
copy reads S and writes S bytes), so the figure is in the copy's units.  The
summary records the sha256 of the kernel's sources (code only: comments and
layout excluded); a reader that finds other code treats the figure as stale.
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import os
import re
import sys
from collections import defaultdict


def _code_only(text: str) -> str:
    """Source text without comments and with whitespace runs collapsed: edits to
    comments or layout leave the digest (and the counters it vouches for) valid."""
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def source_digest(paths) -> str:
    h = hashlib.sha256()
    for p in sorted(paths):
        h.update(os.path.basename(p).encode())
        with open(p, encoding="utf-8") as f:
            h.update(_code_only(f.read()).encode())
    return h.hexdigest()


def _short(name: str) -> str:
    s = name.replace("void ", "").replace("(anonymous namespace)::", "")
    if s.startswith("at::"):
        return "torch " + s.split("<")[0].split("(")[0]
    return re.sub(r"\(.*$", "", s)


def stats(path: str, title: str, cmds) -> str:
    rows = list(csv.DictReader(open(path)))
    out = [f"# {title}", "", "command (run from the repo root on an MI355X):", ""]
    out += [f"    {c}" for c in cmds]
    out += ["", "rocprofv3 kernel statistics, durations in microseconds", "",
            "| kernel | calls | total us | avg us | min us | max us | % |", "|---|---|---|---|---|---|---|"]
    for r in rows:
        out.append(f"| {_short(r['Name'])[:72]} | {r['Calls']} | {float(r['TotalDurationNs']) / 1e3:.1f} | "
                   f"{float(r['AverageNs']) / 1e3:.3f} | {float(r['MinNs']) / 1e3:.3f} | "
                   f"{float(r['MaxNs']) / 1e3:.3f} | {float(r['Percentage']):.2f} |")
    return "\n".join(out) + "\n"


def _per_dispatch(path: str, counter: str, regex: str, grid=None):
    """{dispatch id: (counter value summed over its dimensions, duration ns)} of matching
    kernels (with `grid`: only launches of that many work-items)."""
    pat = re.compile(regex)
    val = defaultdict(float)
    dur = {}
    for r in csv.DictReader(open(path)):
        if r["Counter_Name"] != counter or not pat.search(r["Kernel_Name"]):
            continue
        if grid is not None and int(r["Grid_Size"]) != grid:
            continue
        val[r["Dispatch_Id"]] += float(r["Counter_Value"])
        dur[r["Dispatch_Id"]] = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
    return {k: (val[k], dur[k]) for k in val}


def _mean_us(fetch, write) -> float:
    d = [v for _, v in fetch.values()] + [v for _, v in write.values()]
    return sum(d) / len(d) / 1e3


def traffic(a) -> str:
    # a launch is one dispatch of the first kernel regex and at most one of each
    # further one (a kernel that follows it in the same launch; none is allowed)
    kernels = a.kernel
    fetch = _per_dispatch(a.fetch, "FETCH_SIZE", kernels[0], a.grid)
    write = _per_dispatch(a.write, "WRITE_SIZE", kernels[0], a.grid)
    cf = _per_dispatch(a.fetch, "FETCH_SIZE", a.copy_kernel)
    cw = _per_dispatch(a.write, "WRITE_SIZE", a.copy_kernel)
    if not (fetch and write and cf and cw):
        raise SystemExit("no matching dispatches for the kernel or the copy kernel")
    kib = a.copy_bytes / 1024.0
    # the largest of the copy's readings: its first launch may find part of the source in cache
    f_scale = kib / max(v for v, _ in cf.values())
    w_scale = kib / max(v for v, _ in cw.values())
    f_kib = sum(v for v, _ in fetch.values()) / len(fetch)
    w_kib = sum(v for v, _ in write.values()) / len(write)
    rows = [f"| dispatches of `{kernels[0]}`{f' with {a.grid} work-items' if a.grid else ''} (fetch pass / write pass) "
            f"| {len(fetch)} / {len(write)} |",
            f"| FETCH_SIZE per dispatch, KiB | {f_kib:,.1f} |",
            f"| WRITE_SIZE per dispatch, KiB | {w_kib:,.1f} |"]
    for k in kernels[1:]:
        f2 = _per_dispatch(a.fetch, "FETCH_SIZE", k)
        w2 = _per_dispatch(a.write, "WRITE_SIZE", k)
        f2_kib = sum(v for v, _ in f2.values()) / len(fetch)   # per launch of the first kernel
        w2_kib = sum(v for v, _ in w2.values()) / len(write)
        rows += [f"| dispatches of `{k}` (fetch pass / write pass) | {len(f2)} / {len(w2)} |",
                 f"| its FETCH_SIZE per launch, KiB | {f2_kib:,.1f} |",
                 f"| its WRITE_SIZE per launch, KiB | {w2_kib:,.1f} |"]
        f_kib += f2_kib
        w_kib += w2_kib
    bytes_per_launch = (f_kib * f_scale + w_kib * w_scale) * 1024.0
    out = [f"# {a.title}", "", "commands (run from the repo root on an MI355X):", ""]
    out += [f"    {c}" for c in a.cmd]
    out += ["", "kernel regex: " + " + ".join(f"`{k}`" for k in kernels) + f"; copy kernel regex: `{a.copy_kernel}`, "
                f"{a.copy_bytes} bytes read and written per copy launch", "",
            "| figure | value |", "|---|---|"] + rows + [
            f"| copy FETCH_SIZE per dispatch, KiB (max of {len(cf)}) | {max(v for v, _ in cf.values()):,.1f} |",
            f"| copy WRITE_SIZE per dispatch, KiB (max of {len(cw)}) | {max(v for v, _ in cw.values()):,.1f} |",
            f"| fetch scale (copy bytes / copy counter) | {f_scale:.4f} |",
            f"| write scale (copy bytes / copy counter) | {w_scale:.4f} |",
            f"| HBM bytes read per launch (scaled) | {f_kib * f_scale * 1024:,.0f} |",
            f"| HBM bytes written per launch (scaled) | {w_kib * w_scale * 1024:,.0f} |", "",
            *([f"algorithmic bytes per launch: {a.alg_bytes:,.0f} (counted / algorithmic = "
               f"{bytes_per_launch / a.alg_bytes:.3f}); at the counted launches' mean duration "
               f"{_mean_us(fetch, write):.1f} us (under counter collection): {a.alg_bytes / _mean_us(fetch, write) / 1e3:,.0f} GB/s algorithmic, "
               f"{bytes_per_launch / _mean_us(fetch, write) / 1e3:,.0f} GB/s counted", ""] if a.alg_bytes else []),
            f"bytes_per_launch: {bytes_per_launch:.0f}",
            f"source_sha256: {source_digest(a.source)}",
            "sources: " + " ".join(os.path.relpath(p) for p in sorted(a.source))]
    return "\n".join(out) + "\n"


def grids(path: str, title: str, cmds, byte_specs, peak_gbs: float, include=None) -> str:
    rows = list(csv.DictReader(open(path)))
    inc = re.compile(include) if include else None
    dur = defaultdict(list)
    for r in rows:
        if inc and not inc.search(_short(r["Kernel_Name"])):
            continue
        key = (_short(r["Kernel_Name"]), int(r["Grid_Size_X"]), int(r["Grid_Size_Y"]), int(r["Grid_Size_Z"]))
        dur[key].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    nbytes = []
    for spec in byte_specs or ():
        rx, rest = spec.rsplit("@", 1)
        g, b = rest.split("=")
        nbytes.append((re.compile(rx), int(g), float(b)))
    out = [f"# {title}", "", "commands (run from the repo root on an MI355X):", ""]
    out += [f"    {c}" for c in cmds]
    out += ["", "rocprofv3 kernel durations per launch shape (grid in work-items), microseconds", "",
            "| kernel | grid | launches | median us | min us | mean us | algorithmic bytes | GB/s (median) | % of peak |",
            "|---|---|---|---|---|---|---|---|---|"]
    for key in sorted(dur, key=lambda k: (k[0], k[1] * k[2] * k[3])):
        v = sorted(dur[key])
        med = v[len(v) // 2]
        b = next((nb for rx, g, nb in nbytes if rx.search(key[0]) and g == key[1] * key[2] * key[3]), None)
        gbs = f"{b / (med * 1e-6) / 1e9:,.0f}" if b else ""
        frac = f"{b / (med * 1e-6) / 1e9 / peak_gbs * 100:.1f}" if b else ""
        out.append(f"| {key[0][:60]} | {key[1]}x{key[2]}x{key[3]} | {len(v)} | {med:.2f} | {v[0]:.2f} | "
                   f"{sum(v) / len(v):.2f} | {f'{b:,.0f}' if b else ''} | {gbs} | {frac} |")
    return "\n".join(out) + "\n"


def mfma(a) -> str:
    per = defaultdict(lambda: defaultdict(float))
    meta = {}
    for r in csv.DictReader(open(a.csv)):
        k = r["Dispatch_Id"]
        per[k][r["Counter_Name"]] += float(r["Counter_Value"])
        meta[k] = (_short(r["Kernel_Name"]), int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
    groups = defaultdict(list)
    for k, c in per.items():
        name, dur = meta[k]
        groups[(name, int(c["SQ_INSTS_MFMA"]))].append((dur, c))
    alg = []
    for spec in a.alg or ():
        label, rest = spec.split("@", 1)
        rx, fl = rest.rsplit("=", 1)
        alg.append((label, re.compile(rx), float(fl)))
    out = [f"# {a.title}", "", "commands (run from the repo root on an MI355X):", ""]
    out += [f"    {c}" for c in a.cmd]
    out += ["", f"one MFMA instruction = {a.flops_per_mfma} flops (v_mfma_f32_32x32x16_bf16, the only MFMA the kernels "
                f"issue); {a.simds} SIMDs; GRBM_GUI_ACTIVE summed over {a.xcds} XCDs; nominal peak {a.peak_tflops} TFLOP/s",
            "", "| kernel | step | launches | avg us | MFMA instructions | MFMA flops | algorithmic / MFMA flops | "
                "clock GHz | MFMA busy % of SIMD cycles | % of nominal peak |",
            "|---|---|---|---|---|---|---|---|---|---|"]
    for (name, n_mfma), L in sorted(groups.items(), key=lambda g: -g[0][1] * len(g[1])):
        if n_mfma == 0:
            continue
        dur_s = sum(d for d, _ in L) / len(L) * 1e-9
        busy = sum(c["SQ_VALU_MFMA_BUSY_CYCLES"] for _, c in L) / len(L)
        cyc = sum(c["GRBM_GUI_ACTIVE"] for _, c in L) / len(L) / a.xcds
        flops = n_mfma * a.flops_per_mfma
        lab = next(((l, f) for l, rx, f in alg if rx.search(name) and 0.85 <= f / flops <= 1.0001), None)
        ghz = cyc / dur_s / 1e9
        ok = ghz <= a.max_clock_ghz
        out.append(f"| {name[:48]} | {lab[0] if lab else ''} | {len(L)} | {dur_s * 1e6:.1f} | {n_mfma:,} | {flops:.4g} | "
                   f"{f'{lab[1] / flops:.3f}' if lab else ''} | {f'{ghz:.2f}' if ok else '—'} | "
                   f"{f'{100 * busy / (a.simds * cyc):.1f}' if ok else '—'} | "
                   f"{100 * (lab[1] if lab else flops) / dur_s / (a.peak_tflops * 1e12):.1f} |")
    out += ["", "% of nominal peak uses the algorithmic flops where the step is named, else the MFMA flops.",
            f"GRBM active cycles include time outside a launch's own timestamps, which overstates the clock of short",
            f"launches: where it comes out above {a.max_clock_ghz} GHz the clock and the busy share at it are not shown."]
    return "\n".join(out) + "\n"


def read_traffic(path: str, sources):
    """bytes_per_launch from a traffic summary, or None when it is missing or its
    recorded sources differ from `sources` (the kernel changed since the counters)."""
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"^bytes_per_launch: (\d+)", text, re.M)
    s = re.search(r"^source_sha256: ([0-9a-f]+)", text, re.M)
    if not (m and s) or s.group(1) != source_digest(sources):
        return None
    return float(m.group(1))


def main(argv=None):
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="what", required=True)
    s = sub.add_parser("stats")
    s.add_argument("csv")
    s.add_argument("--title", required=True)
    s.add_argument("--cmd", action="append", required=True)
    t = sub.add_parser("traffic")
    t.add_argument("--fetch", required=True)
    t.add_argument("--write", required=True)
    t.add_argument("--kernel", required=True, action="append",
                   help="kernel regex; repeat for kernels that follow it within one launch")
    t.add_argument("--grid", type=int, help="only launches of this many work-items")
    t.add_argument("--alg-bytes", type=float, help="algorithmic bytes of one launch, for comparison")
    t.add_argument("--copy-kernel", required=True)
    t.add_argument("--copy-bytes", type=int, required=True)
    t.add_argument("--source", nargs="+", required=True)
    t.add_argument("--title", required=True)
    t.add_argument("--cmd", action="append", required=True)
    mf = sub.add_parser("mfma")
    mf.add_argument("csv")
    mf.add_argument("--title", required=True)
    mf.add_argument("--cmd", action="append", required=True)
    mf.add_argument("--alg", action="append", help="LABEL@KERNEL_REGEX=FLOPS: algorithmic flops of one launch")
    mf.add_argument("--flops-per-mfma", type=int, default=32768)
    mf.add_argument("--simds", type=int, default=1024)
    mf.add_argument("--xcds", type=int, default=8)
    mf.add_argument("--peak-tflops", type=float, default=2500.0)
    mf.add_argument("--max-clock-ghz", type=float, default=2.4)
    gr = sub.add_parser("grids")
    gr.add_argument("csv")
    gr.add_argument("--title", required=True)
    gr.add_argument("--cmd", action="append", required=True)
    gr.add_argument("--bytes", action="append")
    gr.add_argument("--peak-gbs", type=float, default=8000.0)
    gr.add_argument("--include", help="only kernels whose short name matches this regex")
    a = ap.parse_args(argv)
    if a.what == "stats":
        sys.stdout.write(stats(a.csv, a.title, a.cmd))
    elif a.what == "mfma":
        sys.stdout.write(mfma(a))
    elif a.what == "grids":
        sys.stdout.write(grids(a.csv, a.title, a.cmd, a.bytes, a.peak_gbs, a.include))
    else:
        sys.stdout.write(traffic(a))


if __name__ == "__main__":
    main()
