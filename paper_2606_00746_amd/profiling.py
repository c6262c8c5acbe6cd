"""Summaries of rocprofv3 runs, for ``profiles/`` and the benchmark's traffic figure.

Kernel-trace summary (per-kernel call count and durations)::

    python -m paper_2606_00746_amd.profiling trace RESULTS_DB OUT.txt --command "..."

HBM traffic record from two counter runs of ``bench.py --copy-calibration MIB``,
one collecting ``FETCH_SIZE`` and one ``WRITE_SIZE`` (KiB per dispatch), each
making CALLS calls of the forward and of the backward (``--warmup 1 --steps 2``:
3)::

    python -m paper_2606_00746_amd.profiling traffic FETCH_CSV WRITE_CSV OUT.json \\
        --workload NAME --copy-mib MIB --calls CALLS --command "..."

Each counter is scaled by what it reads for the plain copy of known size that
the same run makes, so the record holds bytes.  The record carries a hash of
the kernel sources: the benchmark reports the figure only while the sources
are unchanged.

Where the waves' time goes, from one counter run collecting the SQ_ counters
in ``WAVE_COUNTERS`` (wave-cycles waiting, issuing, and by instruction kind)::

    python -m paper_2606_00746_amd.profiling waves COUNTERS_CSV OUT.txt --command "..."
"""
from __future__ import annotations

import argparse
import collections
import csv
import hashlib
import json
import os
import subprocess
import sys
import tempfile

_HERE = os.path.dirname(os.path.abspath(__file__))
_ROOT = os.path.dirname(_HERE)
COPY_KERNEL = "__amd_rocclr_copyBuffer"


# the source files of each kernel family, by a part of the kernel's name
_MED = ("scan_med.hpp", "scan_med.hip", "scan_med_64.hip", "scan_med_56.hip", "scan_med_48.hip",
        "scan_med_40_32_24.hip")
_FAMILY_SOURCES = (("_med_", _MED), ("dw_sum", _MED), ("_pm_", ("scan_pm.hip",)),
                   ("to_blocked", ("scan_pm.hip",)), ("_wide_", ("scan_wide.hip",)),
                   ("pieces_kernel", ("scan_wide.hip",)), ("_tiny_", ("scan_tiny.hip",)),
                   ("_small_", ("scan_small.hip",)), ("_general_", ("scan_general.hip",)),
                   ("norm", ("scan_norm.hip",)))
# kernels that run at the start of a call (re-layouts into the blocked order):
# they belong to the call whose scan kernel follows them
_PREPASS = ("to_blocked_kernel", "norm_to_blocked_kernel", "pieces_kernel")
# the normalization kernels of the _norm calls: forming the weights at the
# start of a call, or the logits' gradient at the end of a backward
_NORM = ("norm_kernel", "norm_pm_kernel")
# shared by every family: device helpers, launch declarations, the dispatch
# and the build flags
_COMMON_SOURCES = ("cdna.hpp", "device.hpp", "launch.hpp", "api.cpp")


def source_files(kernels=None) -> list:
    """The sources that decide what the named kernels do (all of them if None
    or if a name belongs to no known family)."""
    csrc = os.path.join(_HERE, "csrc")
    every = sorted(f for f in os.listdir(csrc) if f.endswith((".hip", ".hpp", ".cpp")))
    names = set(_COMMON_SOURCES)
    for k in kernels or ():
        hit = [f for part, fs in _FAMILY_SOURCES if part in k for f in fs]
        if not hit:
            return [os.path.join(csrc, f) for f in every] + [os.path.join(_HERE, "build.py")]
        names.update(hit)
    if not kernels:
        names = set(every)
    return [os.path.join(csrc, f) for f in sorted(names)] + [os.path.join(_HERE, "build.py")]


def source_hash(kernels=None) -> str:
    """sha256 over the sources of the named kernels (all sources if None) and
    the build flags."""
    h = hashlib.sha256()
    for f in source_files(kernels):
        h.update(os.path.basename(f).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def short_name(name: str) -> str:
    for pre in ("void ", "gspn::(anonymous namespace)::"):
        name = name.replace(pre, "")
    # enum template arguments print as "(gspn::(anonymous namespace)::Mode)1"
    name = name.replace("(Mode)0", "Plain").replace("(Mode)1", "Params")
    return name.split("(")[0]


def call_of(kernel: str) -> str | None:
    """Which library call a kernel belongs to ('fwd' or 'bwd'), None for others."""
    k = short_name(kernel)
    if k.startswith(("fwd_", "sum_")):
        return "fwd"
    if k.startswith(("bwd_", "dw_sum", "dw_reduce", "cast_")):
        return "bwd"
    return None


def trace_summary(db: str, out: str, command: str) -> str:
    with tempfile.TemporaryDirectory() as d:
        subprocess.run(["rocpd2summary", "-i", os.path.abspath(db), "-f", "csv", "-o", "s", "-d", d],
                       check=True, capture_output=True, cwd=d)
        rows = list(csv.DictReader(open(os.path.join(d, "s_kernels_summary.csv"))))
    lines = ["# rocprofv3 kernel-trace summary", f"# command: {command}",
             "# from: rocpd2summary of the run's results database (durations in ns)", "",
             f"{'kernel':<58} {'calls':>6} {'avg_ns':>11} {'min_ns':>10} {'max_ns':>10} {'pct':>6}"]
    for r in rows:
        lines.append(f"{short_name(r['Name'])[:58]:<58} {r['Calls']:>6} "
                     f"{float(r['Average (Nsec)']):>11.0f} {float(r['Min (Nsec)']):>10.0f} "
                     f"{float(r['Max (Nsec)']):>10.0f} {float(r['Percent (Inc)']):>6.1f}")
    text = "\n".join(lines) + "\n"
    with open(out, "w") as f:
        f.write(text)
    return text


def _counter(path: str) -> dict:
    vals = collections.defaultdict(list)
    for r in csv.DictReader(open(path)):
        vals[r["Kernel_Name"]].append(float(r["Counter_Value"]))
    return vals


def _dispatches(path: str) -> list:
    """(kernel, counter value) of every dispatch of a one-counter run, in
    dispatch order."""
    d = {}
    for r in csv.DictReader(open(path)):
        i = int(r["Dispatch_Id"])
        k, v = d.get(i, (r["Kernel_Name"], 0.0))
        d[i] = (k, v + float(r["Counter_Value"]))
    return [d[i] for i in sorted(d)]


def _calls_in_order(disp: list) -> list:
    """The library call of each dispatch, None for other kernels.  The
    library's dispatches come in runs between other kernels (the benchmark's
    cache flush before each step); within a run a scan kernel (call_of)
    names its call, a kernel before a scan kernel belongs to that scan's
    call (a re-layout or the weights' normalization at the start of a call),
    and one after the run's last scan kernel to that kernel's call (the
    transpose of a weight gradient, the logits' gradient at the end of a
    backward)."""
    def library(k):
        return call_of(k) is not None or k.startswith(_PREPASS) or k.startswith(_NORM)

    names = [short_name(k) for k, _ in disp]
    out = [None] * len(disp)
    n = 0
    while n < len(names):
        if not library(names[n]):
            n += 1
            continue
        m = n
        while m < len(names) and library(names[m]):
            m += 1
        nxt = None
        for i in range(m - 1, n - 1, -1):
            nxt = call_of(names[i]) or nxt
            out[i] = nxt
        last = None
        for i in range(n, m):
            last = call_of(names[i]) or last
            if out[i] is None:
                out[i] = last
        n = m
    return out


def traffic_record(fetch_csv: str, write_csv: str, workload: str, copy_mib: int,
                   command: str, calls: int = 3) -> dict:
    """Bytes per call of the library: every dispatch of its kernels counted,
    divided by the number of calls the run made (a call may dispatch a kernel
    several times, e.g. one scan per round of planes)."""
    fetch, write = _counter(fetch_csv), _counter(write_csv)
    fd, wd = _dispatches(fetch_csv), _dispatches(write_csv)
    if [k for k, _ in fd] != [k for k, _ in wd]:
        raise SystemExit("the two counter runs dispatched different kernels")
    calls_of = _calls_in_order(fd)
    copy = [k for k in fetch if short_name(k) == COPY_KERNEL]
    if not copy:
        raise SystemExit(f"no {COPY_KERNEL} dispatch in {fetch_csv}: run bench.py with "
                         "--copy-calibration")
    copy_bytes = copy_mib * (1 << 20)
    # the calibration copy is the copy dispatch that writes the most (small
    # input uploads may run the same kernel); both runs dispatch in one order
    wl = write[copy[0]]
    at = max(range(len(wl)), key=lambda i: wl[i])
    f_copy = fetch[copy[0]][at] * 1024.0
    w_copy = wl[at] * 1024.0
    scale_f, scale_w = copy_bytes / f_copy, copy_bytes / w_copy
    # per (kernel, call): dispatches and bytes (a re-layout kernel may serve
    # both calls)
    acc = collections.defaultdict(lambda: [0, 0.0, 0.0])
    for (k, fv), (_, wv), call in zip(fd, wd, calls_of):
        if call is None:
            continue
        a = acc[(short_name(k), call)]
        a[0] += 1
        a[1] += fv * 1024.0 * scale_f
        a[2] += wv * 1024.0 * scale_w
    kernels, per_call = {}, collections.defaultdict(float)
    for (k, call), (n, fb, wb) in acc.items():
        name = k if (k, "fwd" if call == "bwd" else "bwd") not in acc else f"{k} [{call}]"
        kernels[name] = {"call": call, "fetch_bytes": round(fb / n), "write_bytes": round(wb / n),
                         "dispatches": n, "dispatches_per_call": n / calls}
        per_call[call] += (fb + wb) / calls
    names = sorted({k.split(" [")[0] for k in kernels})
    return {"workload": workload, "source_hash": source_hash(names),
            "source_files": [os.path.basename(f) for f in source_files(names)],
            "command": command,
            "copy_calibration": {"bytes": copy_bytes, "fetch_kib": f_copy / 1024.0,
                                 "write_kib": w_copy / 1024.0, "fetch_scale": scale_f,
                                 "write_scale": scale_w},
            "calls": calls, "kernels": kernels,
            "bytes_per_call": {k: round(v) for k, v in per_call.items()}}


WAVE_COUNTERS = ("SQ_WAVE_CYCLES", "SQ_BUSY_CYCLES", "SQ_WAIT_ANY", "SQ_WAIT_INST_ANY",
                 "SQ_ACTIVE_INST_ANY", "SQ_ACTIVE_INST_VALU", "SQ_ACTIVE_INST_VMEM",
                 "SQ_ACTIVE_INST_LDS")


def waves_summary(csv_path: str, out: str, command: str) -> str:
    """Per kernel, the share of wave-cycles spent waiting and issuing by kind.

    SQ_WAVE_CYCLES counts the cycles of every resident wave; SQ_WAIT_ANY the
    wave-cycles a wave waited on anything (a dependency on an outstanding
    memory or LDS access, a barrier); SQ_WAIT_INST_ANY those it waited for an
    instruction to issue; the SQ_ACTIVE_INST_* those it spent issuing.  All
    are in the same unit, so their ratios are shares of wave time.
    """
    vals = collections.defaultdict(lambda: collections.defaultdict(list))
    for r in csv.DictReader(open(csv_path)):
        vals[short_name(r["Kernel_Name"])][r["Counter_Name"]].append(float(r["Counter_Value"]))
    lines = ["# rocprofv3 wave-time summary (SQ counters, mean over dispatches)",
             f"# command: {command}",
             "# shares of SQ_WAVE_CYCLES: wait = SQ_WAIT_ANY, issue-wait = SQ_WAIT_INST_ANY, "
             "busy = SQ_ACTIVE_INST_ANY, valu/vmem/lds = SQ_ACTIVE_INST_*", "",
             f"{'kernel':<44} {'disp':>4} {'wave_cyc':>12} {'wait':>6} {'iss_wt':>6} "
             f"{'busy':>6} {'valu':>6} {'vmem':>6} {'lds':>6}"]
    for k, cv in vals.items():
        if call_of(k) is None:
            continue
        m = {c: sum(v) / len(v) for c, v in cv.items()}
        wc = m.get("SQ_WAVE_CYCLES", 0.0)
        if wc <= 0:
            continue
        sh = lambda c: m.get(c, 0.0) / wc  # noqa: E731
        lines.append(f"{k[:44]:<44} {len(cv['SQ_WAVE_CYCLES']):>4} {wc:>12.4g} "
                     f"{sh('SQ_WAIT_ANY'):>6.3f} {sh('SQ_WAIT_INST_ANY'):>6.3f} "
                     f"{sh('SQ_ACTIVE_INST_ANY'):>6.3f} {sh('SQ_ACTIVE_INST_VALU'):>6.3f} "
                     f"{sh('SQ_ACTIVE_INST_VMEM'):>6.3f} {sh('SQ_ACTIVE_INST_LDS'):>6.3f}")
    text = "\n".join(lines) + "\n"
    with open(out, "w") as f:
        f.write(text)
    return text


def load_traffic(path: str, call: str) -> float | None:
    """Bytes per call from a traffic record, None if absent or made from other sources."""
    try:
        rec = json.load(open(path))
    except (OSError, ValueError):
        return None
    if rec.get("source_hash") != source_hash(sorted({k.split(" [")[0]
                                                     for k in rec.get("kernels", {})})):
        return None
    return rec.get("bytes_per_call", {}).get(call)


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    sub = ap.add_subparsers(dest="cmd", required=True)
    t = sub.add_parser("trace")
    t.add_argument("db")
    t.add_argument("out")
    t.add_argument("--command", required=True)
    c = sub.add_parser("traffic")
    c.add_argument("fetch_csv")
    c.add_argument("write_csv")
    c.add_argument("out")
    c.add_argument("--workload", required=True)
    c.add_argument("--copy-mib", type=int, required=True)
    c.add_argument("--calls", type=int, default=3,
                   help="calls of each kind in the counter runs (warmup + steps)")
    c.add_argument("--command", required=True)
    v = sub.add_parser("waves")
    v.add_argument("csv")
    v.add_argument("out")
    v.add_argument("--command", required=True)
    a = ap.parse_args(argv)
    if a.cmd == "trace":
        sys.stdout.write(trace_summary(a.db, a.out, a.command))
    elif a.cmd == "waves":
        sys.stdout.write(waves_summary(a.csv, a.out, a.command))
    else:
        rec = traffic_record(a.fetch_csv, a.write_csv, a.workload, a.copy_mib, a.command, a.calls)
        with open(a.out, "w") as f:
            json.dump(rec, f, indent=1)
            f.write("\n")
        print(json.dumps(rec, indent=1))
    return 0


if __name__ == "__main__":
    sys.exit(main())
