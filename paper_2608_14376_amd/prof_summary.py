"""Summaries of rocprofv3 output for the decode benchmark, as short text.

Run on the CSV files of the profiler runs (see each subcommand's "command"
line in the summaries it writes):

  python -m paper_2608_14376_amd.prof_summary kernels  --trace T.csv --out F --title ... --command ...
  python -m paper_2608_14376_amd.prof_summary traffic  --fetch F.csv --write W.csv [--rdreq R.csv]
                                                       --kernel k_attn_split --first N --algorithmic BYTES ...
  python -m paper_2608_14376_amd.prof_summary mfma     --pmc P.csv --trace T.csv ...
  python -m paper_2608_14376_amd.prof_summary fetch    --pmc P.csv --trace T.csv ...
  python -m paper_2608_14376_amd.prof_summary prefill  --pmc P.csv --trace T.csv --call 1 --op qkv=FLOPS ...

Dispatch windows follow bench.py's order for the headline batch: `warmup`
graph steps, `steps` graph steps, one more step, `profile_steps` eagerly
launched steps timed kernel by kernel (the roofline's in-step durations),
then the dominant kernel's isolated launches.  Counter values are averaged
per dispatch; FETCH_SIZE and WRITE_SIZE (KiB) are scaled by what they read
for the run's last dispatch, a plain 1 GiB device copy (bench.py
--calibrate-copy)."""
from __future__ import annotations

import argparse
import collections
import csv
import hashlib
import os

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CLOCK_GHZ = 2.4
SIMDS = 1024


def source_sha() -> str:
    h = hashlib.sha256()
    for f in ("kernels.hip", "kernels.h"):
        h.update(open(os.path.join(HERE, "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def short(name: str) -> str:
    return name.split("(")[0].split("<")[0].strip()


def read(path):
    with open(path) as f:
        return list(csv.DictReader(f))


def grid(r) -> str:
    """The dispatch's grid size in work-items (x * y * z): the kernel trace
    lists the dimensions, the counter runs the product."""
    if "Grid_Size_X" in r:
        return str(int(r["Grid_Size_X"]) * int(r.get("Grid_Size_Y") or 1) * int(r.get("Grid_Size_Z") or 1))
    return str(int(float(r.get("Grid_Size", "0"))))


def trace_dispatches(path):
    """(name, grid, start_ns, end_ns) of every kernel dispatch, in start order."""
    out = []
    for r in read(path):
        out.append((short(r["Kernel_Name"]), grid(r), int(r["Start_Timestamp"]), int(r["End_Timestamp"])))
    out.sort(key=lambda d: d[2])
    return out


def pmc_dispatches(path, counters):
    """{dispatch id: (name, grid, {counter: value})} in dispatch order."""
    by = collections.OrderedDict()
    for r in read(path):
        did = int(r["Dispatch_Id"])
        name = short(r["Kernel_Name"])
        g = grid(r)
        by.setdefault(did, (name, g, {}))[2][r["Counter_Name"]] = float(r["Counter_Value"])
    return [by[k] for k in sorted(by)]


def header(a) -> list[str]:
    return [f"# {a.title}", f"# command: {a.command}", f"# kernel_source_sha256_16: {source_sha()}"]


def cmd_kernels(a):
    ds = [d for d in trace_dispatches(a.trace) if d[0].startswith("k_")]
    lines = header(a)
    per = collections.defaultdict(list)
    for n, g, s, e in ds:
        per[n].append((e - s) / 1e3)
    lines.append("")
    lines.append("# corun kernels by total time (all dispatches of the run)")
    lines.append(f"{'kernel':34s} {'calls':>7s} {'avg_us':>9s} {'min_us':>9s} {'max_us':>9s} {'total_ms':>9s}")
    for n, v in sorted(per.items(), key=lambda kv: -sum(kv[1])):
        lines.append(f"{n:34s} {len(v):7d} {sum(v) / len(v):9.2f} {min(v):9.2f} {max(v):9.2f} {sum(v) / 1e3:9.2f}")
    L = a.layers
    if a.kernel:
        k = [(e - s) / 1e3 for n, g, s, e in ds if n == a.kernel]
        graph = k[:(a.warmup + a.steps) * L]
        prof = k[(a.warmup + a.steps + 1) * L:(a.warmup + a.steps + 1 + a.profile_steps) * L]
        iso = k[(a.warmup + a.steps + 1 + a.profile_steps) * L:][:a.kernel_iters + 1][1:]
        lines.append("")
        lines.append(f"# {a.kernel} of the headline batch, by phase of bench.py (dispatch order)")
        if graph:
            lines.append(f"graph_steps_mean_us: {sum(graph) / len(graph):.2f}  ({len(graph)} dispatches)")
        if prof:
            lines.append(f"in_step_eager_mean_us: {sum(prof) / len(prof):.2f}  ({len(prof)} dispatches; "
                         f"bench.py's roofline duration)")
        if iso:
            lines.append(f"isolated_mean_us: {sum(iso) / len(iso):.2f}  ({len(iso)} dispatches)")
    if a.step_kernel:
        # one timed graph step: dispatches between consecutive launches of the step's first kernel
        starts = [i for i, d in enumerate(ds) if d[0] == a.step_kernel]
        spans = []
        for i0, i1 in zip(starts[a.warmup:a.warmup + a.steps], starts[a.warmup + 1:a.warmup + a.steps + 1]):
            seg = ds[i0:i1]
            spans.append((seg[-1][3] - seg[0][2], sum(e - s for _, _, s, e in seg), len(seg), seg))
        if spans:
            spans.sort(key=lambda x: x[0])
            span, busy, cnt, seg = spans[len(spans) // 2]
            lines.append("")
            lines.append(f"# one timed graph step (the median of {len(spans)}): span {span / 1e3:.1f} us, "
                         f"{cnt} kernels, kernel time {busy / 1e3:.1f} us")
            agg = collections.defaultdict(list)
            for n, g, s, e in seg:
                agg[f"{n} grid={g}"].append((e - s) / 1e3)
            lines.append(f"{'kernel':44s} {'launches':>8s} {'total_us':>9s} {'avg_us':>8s}")
            for n, v in sorted(agg.items(), key=lambda kv: -sum(kv[1])):
                lines.append(f"{n:44s} {len(v):8d} {sum(v):9.1f} {sum(v) / len(v):8.2f}")
    for ln in a.note or []:
        lines.append(f"# {ln}")
    open(a.out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def copy_scale(ds, counter, known_kib):
    n, g, c = ds[-1]
    if not n.startswith("__amd") and "copy" not in n.lower() and "elementwise" not in n:
        raise SystemExit(f"the run's last dispatch ({n}) is not the calibration copy")
    return known_kib / c[counter], c[counter]


def cmd_traffic(a):
    f = pmc_dispatches(a.fetch, ["FETCH_SIZE"])
    w = pmc_dispatches(a.write, ["WRITE_SIZE"])
    fs, fraw = copy_scale(f, "FETCH_SIZE", 1 << 20)
    ws, wraw = copy_scale(w, "WRITE_SIZE", 1 << 20)
    fk = [c["FETCH_SIZE"] for n, g, c in f if n == a.kernel][:a.first]
    wk = [c["WRITE_SIZE"] for n, g, c in w if n == a.kernel][:a.first]
    fmean, wmean = sum(fk) / len(fk), sum(wk) / len(wk)
    traffic = (fmean * fs + wmean * ws) * 1024
    lines = header(a)
    lines += [
        f"# calibration: the last dispatch of each run is a plain 1 GiB device copy (bench.py --calibrate-copy)",
        f"# dispatches used: the first {a.first} of {a.kernel} (the headline batch's graph steps and the step",
        f"# after them); later batch mixes decoded by bench.py's bit-exact check are excluded",
        f"copy_fetch_kib: {fraw:.1f}",
        f"copy_write_kib: {wraw:.1f}",
        f"fetch_scale: {fs:.4f}",
        f"write_scale: {ws:.4f}",
        f"dispatches_fetch: {len(fk)}",
        f"dispatches_write: {len(wk)}",
        f"fetch_kib_per_dispatch_raw: {fmean:.1f}",
        f"write_kib_per_dispatch_raw: {wmean:.1f}",
        f"traffic_bytes_per_launch: {traffic:.0f}",
        f"algorithmic_bytes_per_launch: {a.algorithmic}",
        f"traffic_over_algorithmic: {traffic / a.algorithmic:.4f}",
    ]
    if a.rdreq:
        r = pmc_dispatches(a.rdreq, [])
        names = ("TCC_EA0_RDREQ_32B_sum", "TCC_EA0_RDREQ_64B_sum", "TCC_EA0_RDREQ_128B_sum")
        size = dict(zip(names, (32, 64, 128)))
        copy = r[-1][2]
        kr = [c for n, g, c in r if n == a.kernel][:a.first]
        mean = {k: sum(c.get(k, 0.0) for c in kr) / len(kr) for k in names}
        cb = sum(copy.get(k, 0.0) * size[k] for k in names)
        kb = sum(mean[k] * size[k] for k in names)
        lines += [
            "",
            "# cross-check: L2-to-fabric read requests resolved by size (a third run)",
            f"copy_read_bytes_by_request_size: {cb:.0f}  (1 GiB = {1 << 30})",
            f"kernel_requests_per_dispatch: { {k: round(v, 1) for k, v in mean.items()} }",
            f"kernel_read_bytes_by_request_size: {kb:.0f}",
            f"kernel_read_over_algorithmic: {kb / a.algorithmic:.4f}",
        ]
    for ln in a.note or []:
        lines.append(f"# {ln}")
    open(a.out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def durations_by_grid(trace, kernels):
    out = collections.defaultdict(list)
    for n, g, s, e in trace_dispatches(trace):
        if n in kernels:
            out[g].append((e - s) / 1e3)
    return out


def cmd_mfma(a):
    p = pmc_dispatches(a.pmc, [])
    ks = set(a.kernel.split(","))
    dur = durations_by_grid(a.trace, ks)
    lines = header(a)
    lines += ["# SQ_VALU_MFMA_BUSY_CYCLES: the dispatch's MFMA busy cycles summed over SIMDs; busy fraction =",
              f"# that / (duration x {CLOCK_GHZ} GHz x {SIMDS} SIMDs), mean durations from the kernel trace run",
              "", f"{'projection (grid)':34s} {'dispatches':>10s} {'MFMA busy Mcyc':>15s} {'us':>9s} {'busy':>7s}"]
    agg = collections.defaultdict(list)
    for n, g, c in p:
        if n in ks:
            agg[g].append(c.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0))
    for g, v in sorted(agg.items(), key=lambda kv: -sum(kv[1]) / len(kv[1])):
        d = dur.get(g)
        if not d:
            continue
        us = sum(d) / len(d)
        busy = sum(v) / len(v)
        frac = busy / (us * 1e-6 * CLOCK_GHZ * 1e9 * SIMDS)
        label = a.labels.get(g, g) if a.labels else g
        lines.append(f"{label:34s} {len(v):10d} {busy / 1e6:15.2f} {us:9.2f} {100 * frac:6.1f}%")
    for ln in a.note or []:
        lines.append(f"# {ln}")
    open(a.out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def cmd_fetch(a):
    p = pmc_dispatches(a.pmc, ["FETCH_SIZE"])
    fs, fraw = copy_scale(p, "FETCH_SIZE", 1 << 20)
    ks = set(a.kernel.split(","))
    dur = durations_by_grid(a.trace, ks)
    lines = header(a)
    lines += [f"# calibration: the run's last dispatch copies 1 GiB; FETCH_SIZE read {fraw:.1f} KiB, scale x{fs:.4f}",
              "", f"{'projection (grid)':34s} {'dispatches':>10s} {'fetched MB':>11s} {'weights MB':>11s} "
                  f"{'ratio':>6s} {'us':>8s} {'TB/s':>6s} {'of 8 TB/s':>9s}"]
    agg = collections.defaultdict(list)
    for n, g, c in p:
        if n in ks:
            agg[g].append(c["FETCH_SIZE"])
    for g, v in sorted(agg.items(), key=lambda kv: -sum(kv[1])):
        if g not in (a.labels or {}):
            continue
        label, wbytes = a.labels[g]
        mb = sum(v) / len(v) * fs * 1024 / 1e6
        d = dur.get(g, [])
        us = sum(d) / len(d) if d else float("nan")
        lines.append(f"{label:34s} {len(v):10d} {mb:11.1f} {wbytes / 1e6:11.1f} {mb * 1e6 / wbytes:6.3f} "
                     f"{us:8.2f} {wbytes / us / 1e6:6.2f} {100 * wbytes / us / 1e6 / 8:8.1f}%")
    for ln in a.note or []:
        lines.append(f"# {ln}")
    open(a.out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def prefill_window(disp, call):
    """The dispatches of the call-th prefill of the run (0-based): from its
    k_embed to the next one (each prefill call starts with the embedding)."""
    starts = [i for i, d in enumerate(disp) if d[0] == "k_embed"]
    if call >= len(starts):
        raise SystemExit(f"the run has {len(starts)} prefill calls, not {call + 1}")
    end = starts[call + 1] if call + 1 < len(starts) else len(disp)
    return disp[starts[call]:end]


def label_prefill(window, ops, layers):
    """Name each dispatch of one prefill: the projections cycle through `ops`
    per layer (the last is lm_head), k_prefill_attn is attention."""
    out, j = [], 0
    for d in window:
        n = d[0]
        if n.startswith("k_gemm"):
            out.append(ops[j % len(ops)] if j < len(ops) * layers else "lm_head")
            j += 1
        elif n.startswith("k_prefill_attn"):
            out.append("attention")
        else:
            out.append(n)
    return out


def cmd_prefill(a):
    ops = [x.split("=")[0] for x in a.op]
    flops = {x.split("=")[0]: float(x.split("=")[1]) for x in a.op}
    flops["attention"] = a.attn_flops
    tw = prefill_window(trace_dispatches(a.trace), a.call)
    pw = prefill_window(pmc_dispatches(a.pmc, []), a.call)
    if [d[0] for d in tw] != [d[0] for d in pw]:
        raise SystemExit("the trace and counter runs launched different kernels in this prefill")
    names = label_prefill(tw, ops, a.layers)
    dur, cnt, kern = collections.defaultdict(list), collections.defaultdict(list), {}
    for nm, t, c in zip(names, tw, pw):
        dur[nm].append((t[3] - t[2]) / 1e3)
        cnt[nm].append(c[2])
        kern[nm] = t[0]
    lines = header(a)
    lines += [f"# busy = SQ_VALU_MFMA_BUSY_CYCLES / (duration x {CLOCK_GHZ} GHz x {SIMDS} SIMDs) (32 cycles per "
              "32x32x16 bf16 MFMA);",
              "# VALU / MFMA and LDS / MFMA are instruction-count ratios (SQ_INSTS_VALU counts the MFMAs too);",
              "# durations from the kernel-trace run, counters from the counter run, matched dispatch by dispatch",
              "", f"{'op':12s} {'kernel':16s} {'dispatches':>10s} {'us':>9s} {'busy':>6s} {'TFLOP/s':>8s} "
                  f"{'VALU/MFMA':>9s} {'LDS/MFMA':>8s} {'conflicts/LDS':>13s}"]
    total_us = sum(sum(v) for v in dur.values())
    for nm in ops + ["attention", "lm_head"]:
        if nm not in dur:
            continue
        us = sum(dur[nm]) / len(dur[nm])
        mean = lambda k: sum(c.get(k, 0.0) for c in cnt[nm]) / len(cnt[nm])
        mf = mean("SQ_INSTS_MFMA")
        busy = mean("SQ_VALU_MFMA_BUSY_CYCLES") / (us * 1e-6 * CLOCK_GHZ * 1e9 * SIMDS)
        tf = flops.get(nm, 0.0) / us / 1e6
        lds = mean("SQ_INSTS_LDS")
        lines.append(f"{nm:12s} {kern[nm]:16s} {len(dur[nm]):10d} {us:9.2f} {100 * busy:5.1f}% {tf:8.1f} "
                     f"{mean('SQ_INSTS_VALU') / mf if mf else 0:9.2f} {lds / mf if mf else 0:8.2f} "
                     f"{mean('SQ_LDS_BANK_CONFLICT') / lds if lds else 0:13.3f}")
    rest = sorted(((nm, sum(v)) for nm, v in dur.items() if nm not in ops + ["attention", "lm_head"]),
                  key=lambda kv: -kv[1])
    lines += ["", f"# the prefill's {len(tw)} dispatches take {total_us / 1e3:.2f} ms of kernel time; "
                  "the other kernels: " + ", ".join(f"{nm} {v / 1e3:.2f} ms" for nm, v in rest)]
    for ln in a.note or []:
        lines.append(f"# {ln}")
    open(a.out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    for name in ("kernels", "traffic", "mfma", "fetch", "prefill"):
        s = sub.add_parser(name)
        s.add_argument("--out", required=True)
        s.add_argument("--title", required=True)
        s.add_argument("--command", required=True)
        s.add_argument("--note", action="append")
        if name == "kernels":
            s.add_argument("--trace", required=True)
            s.add_argument("--kernel", default="")
            s.add_argument("--step-kernel", default="")
            s.add_argument("--layers", type=int, default=36)
            s.add_argument("--warmup", type=int, default=2)
            s.add_argument("--steps", type=int, default=8)
            s.add_argument("--profile-steps", type=int, default=3)
            s.add_argument("--kernel-iters", type=int, default=10)
        elif name == "traffic":
            s.add_argument("--fetch", required=True)
            s.add_argument("--write", required=True)
            s.add_argument("--rdreq", default="")
            s.add_argument("--kernel", required=True)
            s.add_argument("--first", type=int, required=True)
            s.add_argument("--algorithmic", type=int, required=True)
        elif name == "prefill":
            s.add_argument("--pmc", required=True)
            s.add_argument("--trace", required=True)
            s.add_argument("--call", type=int, default=1, help="which prefill call of the run (0-based)")
            s.add_argument("--layers", type=int, default=36)
            s.add_argument("--op", action="append", default=[],
                           help="name=flops of each projection, in launch order within a layer")
            s.add_argument("--attn-flops", type=float, default=0.0)
        else:
            s.add_argument("--pmc", required=True)
            s.add_argument("--trace", required=True)
            s.add_argument("--kernel", default="k_gemm_dma", help="kernel name(s), comma-separated")
            s.add_argument("--label", action="append", default=[],
                           help="grid=name (mfma) or grid=name=weight_bytes (fetch)")
    a = ap.parse_args()
    if a.cmd in ("mfma", "fetch"):
        a.labels = {}
        for item in a.label:
            parts = item.split("=")
            a.labels[parts[0]] = parts[1] if a.cmd == "mfma" else (parts[1], int(parts[2]))
    {"kernels": cmd_kernels, "traffic": cmd_traffic, "mfma": cmd_mfma, "fetch": cmd_fetch,
     "prefill": cmd_prefill}[a.cmd](a)


if __name__ == "__main__":
    main()
