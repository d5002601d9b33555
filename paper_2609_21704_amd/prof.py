"""Summaries of rocprofv3 output for the SpecQuant kernels.

    python -m paper_2609_21704_amd.prof stats <rocprofv3 output dir> [--match SUBSTR]
        per-kernel dispatch count and duration (avg / min / max), kernels grouped
        by name and grid size
    python -m paper_2609_21704_amd.prof traffic <FETCH_SIZE dir> <WRITE_SIZE dir> --copy-bytes N
            [--variant int4|fp8] [--calls C]
        HBM bytes per draft-GEMV call from the FETCH_SIZE / WRITE_SIZE
        counters, each divided by what the same counter reads, per byte, for the
        plain copy pass over N bytes (read once, written once) that the profiled
        command dispatches last; the draft-GEMV dispatches of the variant are
        summed and divided by C calls (default: one call per dispatch)
    python -m paper_2609_21704_amd.prof gemv <rocprofv3 output dir> --variant int4|fp8 [--calls C]
        the draft-GEMV dispatches of the variant: count, total and average
        duration (per call when C is given)
    python -m paper_2609_21704_amd.prof verify <MfmaUtil/MfmaFlopsF16 dir> <FETCH_SIZE dir> <WRITE_SIZE dir>
            --copy-bytes N --m M --layers L --shapes NAME:NxK,... [--lm NxK]
        per verify projection (the verify dispatches of one round, in their
        order: the L layers' shapes in turn, then the LM head): duration,
        executed matrix-core flops, matrix-core busy fraction, HBM bytes

    python -m paper_2609_21704_amd.prof rounds <rocprofv3 output dir> --end SUBSTR [--rounds R]
        the last R rounds of a trace, each ending with a dispatch whose name
        contains SUBSTR (the decoder rounds end with sq::commit_kernel): time
        per round, busy time per kernel and the gaps between dispatches

The inputs are the rocpd SQLite databases rocprofv3 writes (*.db).
"""
from __future__ import annotations

import argparse
import collections
import glob
import hashlib
import os
import re
import sqlite3

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_21704_amd", "csrc")
# the sources of each draft GEMV variant's kernels, and its dispatches: the
# GEMV kernels with the variant's weight kind (second template argument: fp8
# or not), and for FP8 the matrix-core streaming instance (kind 1) that takes
# the large matrices at m >= 3
GEMV_SOURCES = {"int4": ["gemv.hip"], "fp8": ["gemv.hip", "linear.hip"]}


def is_draft_gemv(name: str, variant: str) -> bool:
    if name.startswith(("sq::gemv_kernel<", "sq::gemv_rows_kernel<")):
        fp8 = name.split(",")[1].strip() == "true"
        return fp8 == (variant == "fp8")
    return variant == "fp8" and name.startswith("sq::linear_kernel<1,")


def sources_sha(variant: str) -> str:
    h = hashlib.sha256()
    for f in GEMV_SOURCES[variant]:
        h.update(open(os.path.join(CSRC, f), "rb").read())
    return h.hexdigest()


def _dbs(path):
    return sorted(glob.glob(os.path.join(path, "**", "*.db"), recursive=True))


def short_name(name: str) -> str:
    name = name.replace("(anonymous namespace)::", "")
    if name.startswith("void "):
        name = name[5:]
    depth = 0
    for i, ch in enumerate(name):  # cut the argument list (the first '(' outside template brackets)
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0:
            return name[:i].strip()
    return name.strip()


def kernel_rows(path):
    for db in _dbs(path):
        con = sqlite3.connect(db)
        for row in con.execute("select name, grid_x, grid_y, workgroup_x, duration from kernels order by start"):
            yield row


def stats(path, match=None):
    groups = collections.OrderedDict()
    for name, gx, gy, wx, dur in kernel_rows(path):
        sn = short_name(name)
        if match and match not in sn:
            continue
        key = (sn, gx // max(wx, 1), gy, wx)
        groups.setdefault(key, []).append(dur)
    lines = [f"{'kernel':58s} {'grid':>12s} {'wg':>4s} {'calls':>7s} {'avg_us':>9s} {'min_us':>9s} {'max_us':>9s}"]
    by_name = collections.OrderedDict()
    for (sn, gx, gy, wx), d in groups.items():
        lines.append(f"{sn[:58]:58s} {f'{gx}x{gy}':>12s} {wx:>4d} {len(d):>7d} {sum(d) / len(d) / 1e3:>9.2f} "
                     f"{min(d) / 1e3:>9.2f} {max(d) / 1e3:>9.2f}")
        by_name.setdefault(sn, []).extend(d)
    if match and by_name:
        alld = [x for d in by_name.values() for x in d]
        lines.append(f"all kernels matching '{match}': calls {len(alld)}, avg_us {sum(alld) / len(alld) / 1e3:.2f}")
    lines.append("")
    lines.append(f"{'kernel (all grids)':58s} {'calls':>7s} {'avg_us':>9s} {'total_ms':>10s}")
    for sn, d in by_name.items():
        lines.append(f"{sn[:58]:58s} {len(d):>7d} {sum(d) / len(d) / 1e3:>9.2f} {sum(d) / 1e6:>10.3f}")
    return "\n".join(lines)


def counter_values(path, counter):
    """(dispatch_id, short kernel name, value) of every dispatch, in dispatch order."""
    rows = []
    for db in _dbs(path):
        con = sqlite3.connect(db)
        for d, k, c, v in con.execute("select dispatch_id, kernel_name, counter_name, value from counters_collection"):
            if c == counter:
                rows.append((d, short_name(k), v))
    rows.sort()
    return rows


def traffic(fetch_dir, write_dir, copy_bytes, variant="int4", calls=None):
    fetch = counter_values(fetch_dir, "FETCH_SIZE")
    write = counter_values(write_dir, "WRITE_SIZE")
    copy_key = fetch[-1][1]
    f_scale = fetch[-1][2] * 1024.0 / copy_bytes   # counters are in KiB
    w_scale = write[-1][2] * 1024.0 / copy_bytes
    f_g = [v * 1024.0 for _, k, v in fetch if is_draft_gemv(k, variant)]
    w_g = [v * 1024.0 for _, k, v in write if is_draft_gemv(k, variant)]
    n = calls or len(f_g)
    f_mean = sum(f_g) / n / f_scale
    w_mean = sum(w_g) / n / w_scale if w_g else 0.0
    return "\n".join([
        f"copy_kernel = {copy_key}",
        f"copy_bytes = {copy_bytes}",
        f"fetch_counter_bytes_per_copied_byte = {f_scale:.6f}",
        f"write_counter_bytes_per_copied_byte = {w_scale:.6f}",
        f"variant = {variant}",
        f"gemv_dispatches = {len(f_g)}",
        f"gemv_calls = {n}",
        f"fetch_bytes_per_launch_raw = {sum(f_g) / n:.1f}",
        f"write_bytes_per_launch_raw = {sum(w_g) / n:.1f}",
        f"hbm_read_bytes_per_launch = {f_mean:.1f}",
        f"hbm_write_bytes_per_launch = {w_mean:.1f}",
        f"hbm_bytes_per_launch = {f_mean + w_mean:.1f}",
        f"gemv_source_sha256 = {sources_sha(variant)}",
    ])


def gemv_trace(path, variant, calls=None):
    d = [dur for name, _, _, _, dur in kernel_rows(path) if is_draft_gemv(short_name(name), variant)]
    n = calls or len(d)
    return "\n".join([
        f"variant = {variant}",
        f"gemv_dispatches = {len(d)}",
        f"gemv_calls = {n}",
        f"total_ms = {sum(d) / 1e6:.3f}",
        f"avg_us_per_call = {sum(d) / n / 1e3:.3f}",
    ])


# the FP16 verification kernels (linear_kernel<2, ...> is the FP16 instance; the
# INT4 / FP8 instances serve draft projections)
VERIFY_KERNELS = ("sq::linear_kernel<2,", "sq::gemm_rows_kernel", "sq::gemm_f16_kernel")
REDUCE_KERNEL = "sq::slice_reduce_kernel"


def dispatch_counters(path):
    """{dispatch_id: (short kernel name, duration ns, {counter: value})}."""
    out = {}
    for db in _dbs(path):
        con = sqlite3.connect(db)
        for d, k, c, v, dur in con.execute(
                "select dispatch_id, kernel_name, counter_name, value, duration from counters_collection"):
            e = out.setdefault(d, [short_name(k), dur, {}])
            e[2][c] = v
    return out


def verify(mfma_dir, fetch_dir, write_dir, copy_bytes, m, layers, shapes, lm):
    mf = dispatch_counters(mfma_dir)
    fe = dispatch_counters(fetch_dir)
    wr = dispatch_counters(write_dir)
    # the copy pass is the last dispatch of every run: counter bytes per copied byte
    f_scale = fe[max(fe)][2]["FETCH_SIZE"] * 1024.0 / copy_bytes
    w_scale = wr[max(wr)][2]["WRITE_SIZE"] * 1024.0 / copy_bytes

    def seq(runs):
        # verify dispatches in order, each K-slice reduction that directly follows one attached to it
        out, prev = [], False
        for d in sorted(runs):
            name = runs[d][0]
            if name.startswith(VERIFY_KERNELS) or (prev and name.startswith(REDUCE_KERNEL)):
                out.append(runs[d])
                prev = not name.startswith(REDUCE_KERNEL)
            else:
                prev = False
        return out

    vm, vf, vw = seq(mf), seq(fe), seq(wr)
    labels = [name for _ in range(layers) for name, _, _ in shapes] + (["lm_head"] if lm else [])
    dims = {name: (n, k) for name, n, k in shapes}
    if lm:
        dims["lm_head"] = lm
    # a projection may take two dispatches (a K-slice reduction follows); attach those to the previous one
    groups = []
    for i, e in enumerate(vm):
        if e[0].startswith(REDUCE_KERNEL) and groups:
            groups[-1].append(i)
        else:
            groups.append([i])
    if len(groups) != len(labels):
        raise SystemExit(f"{len(groups)} verify calls in the profile, {len(labels)} expected")
    rows = collections.OrderedDict()
    for name, idx in zip(labels, groups):
        r = rows.setdefault(name, {"calls": 0, "dur": 0.0, "flops": 0.0, "busy": 0.0, "hbm": 0.0, "kernels": set()})
        r["calls"] += 1
        for i in idx:
            r["kernels"].add(vm[i][0].replace("sq::", ""))
            r["dur"] += vm[i][1]
            r["flops"] += vm[i][2].get("MfmaFlopsF16", 0.0)
            # busy fraction weighted by duration over the projection's dispatches
            r["busy"] += vm[i][2].get("MfmaUtil", 0.0) / 100.0 * vm[i][1]
            r["hbm"] += vf[i][2]["FETCH_SIZE"] * 1024.0 / f_scale + vw[i][2]["WRITE_SIZE"] * 1024.0 / w_scale
    lines = [f"{'projection':10s} {'n x k':>14s} {'calls':>5s} {'us/call':>8s} {'alg MB':>8s} {'HBM MB':>8s} "
             f"{'HBM/alg':>7s} {'TB/s':>6s} {'MFMA TF/s':>9s} {'MFMA busy':>9s}  kernels"]
    for name, r in rows.items():
        n, k = dims[name]
        c = r["calls"]
        alg = 2.0 * n * k + 2.0 * m * k + 4.0 * m * n
        dur = r["dur"] / c
        hbm = r["hbm"] / c
        lines.append(f"{name:10s} {f'{n}x{k}':>14s} {c:>5d} {dur / 1e3:>8.2f} {alg / 1e6:>8.2f} {hbm / 1e6:>8.2f} "
                     f"{hbm / alg:>7.3f} {alg / dur / 1e3:>6.2f} {r['flops'] / c / dur / 1e3:>9.1f} "
                     f"{r['busy'] / r['dur']:>9.4f}  {','.join(sorted(r['kernels']))}")
    lines.append(f"fetch_counter_bytes_per_copied_byte = {f_scale:.6f}")
    lines.append(f"write_counter_bytes_per_copied_byte = {w_scale:.6f}")
    return "\n".join(lines)


def rounds(path, end, count=20):
    rows = []
    for db in _dbs(path):
        con = sqlite3.connect(db)
        rows += list(con.execute("select name, start, end from kernels order by start"))
    rows.sort(key=lambda r: r[1])
    ends = [i for i, r in enumerate(rows) if end in short_name(r[0])]
    if len(ends) < 2:
        return f"fewer than two dispatches matching '{end}'"
    sel = ends[-(count + 1):]
    n = len(sel) - 1
    busy = collections.Counter()
    calls = collections.Counter()
    total = gaps = 0
    for a, b in zip(sel[:-1], sel[1:]):
        total += rows[b][2] - rows[a][2]
        prev = rows[a][2]
        for name, st, en in rows[a + 1:b + 1]:
            sn = re.sub(r"<.*", "", short_name(name))
            busy[sn] += en - st
            calls[sn] += 1
            gaps += max(0, st - prev)
            prev = max(prev, en)
    lines = [f"rounds: {n} (ending with '{end}'); {total / n / 1e3:.1f} us per round, dispatches "
             f"{sum(calls.values()) / n:.0f} per round, busy {sum(busy.values()) / n / 1e3:.1f} us, gaps "
             f"{gaps / n / 1e3:.1f} us",
             f"{'kernel':44s} {'calls/round':>11s} {'us/round':>10s} {'avg_us':>8s}"]
    for sn, t in busy.most_common():
        lines.append(f"{sn[:44]:44s} {calls[sn] / n:>11.0f} {t / n / 1e3:>10.1f} {t / calls[sn] / 1e3:>8.2f}")
    return "\n".join(lines)


def _nk(s):
    n, k = s.lower().split("x")
    return int(n), int(k)


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    a = sub.add_parser("stats")
    a.add_argument("path")
    a.add_argument("--match")
    b = sub.add_parser("traffic")
    b.add_argument("fetch_dir")
    b.add_argument("write_dir")
    b.add_argument("--copy-bytes", type=int, required=True)
    b.add_argument("--variant", default="int4", choices=["int4", "fp8"])
    b.add_argument("--calls", type=int)
    g = sub.add_parser("gemv")
    g.add_argument("path")
    g.add_argument("--variant", default="int4", choices=["int4", "fp8"])
    g.add_argument("--calls", type=int)
    c = sub.add_parser("verify")
    c.add_argument("mfma_dir")
    c.add_argument("fetch_dir")
    c.add_argument("write_dir")
    c.add_argument("--copy-bytes", type=int, required=True)
    c.add_argument("--m", type=int, required=True)
    c.add_argument("--layers", type=int, required=True)
    c.add_argument("--shapes", required=True, help="name:NxK,... in the order of one layer's verify calls")
    c.add_argument("--lm", type=_nk, help="NxK of the LM head, verified after the layers")
    r = sub.add_parser("rounds")
    r.add_argument("path")
    r.add_argument("--end", required=True)
    r.add_argument("--rounds", type=int, default=20)
    args = ap.parse_args()
    if args.cmd == "rounds":
        print(rounds(args.path, args.end, args.rounds))
    elif args.cmd == "stats":
        print(stats(args.path, args.match))
    elif args.cmd == "traffic":
        print(traffic(args.fetch_dir, args.write_dir, args.copy_bytes, args.variant, args.calls))
    elif args.cmd == "gemv":
        print(gemv_trace(args.path, args.variant, args.calls))
    else:
        shapes = [(part.split(":")[0],) + _nk(part.split(":")[1]) for part in args.shapes.split(",")]
        print(verify(args.mfma_dir, args.fetch_dir, args.write_dir, args.copy_bytes, args.m, args.layers, shapes,
                     args.lm))


if __name__ == "__main__":
    main()
