#!/usr/bin/env python3
"""Summarise rocprofv3 runs of ``bench.py`` into a short Markdown profile.

Inputs are rocprofv3 SQLite outputs (``*_results.db``):

* ``--trace``: a ``--kernel-trace --stats`` run of bench.py, with the JSON
  line that run printed (``--bench``);
* ``--fetch`` / ``--write``: one ``--pmc FETCH_SIZE`` and one
  ``--pmc WRITE_SIZE`` run of the same workload (``--no-profile``);
* ``--calib-fetch`` / ``--calib-write``: the same two counters read on
  ``bench.py --copy-calib`` (three plain copies of 1 GiB), which turn the
  counters' KiB into bytes.

The summary lists the per-kernel trace statistics, the library's own
HIP-event timing of the same run, and the calibrated HBM bytes per dispatch
of each kernel variant.  It ends with a ``traffic`` block (one JSON object
per variant) that bench.py reads to fill ``roofline.traffic``, stamped with
a hash of the kernel sources: once any source changes, bench.py ignores the
record and reports null.

Usage (after the rocprofv3 runs):
    python bench_profile.py --bench B.json --trace T.db --fetch F.db --write W.db \
        --calib-fetch CF.db --calib-write CW.db --title "..." --cmd "..." [--cmd ...] \
        --out profiles/NAME.md
"""

import argparse
import collections
import json
import re
import sqlite3

COPY_BYTES = 16384 * 16384 * 4   # one --copy-calib copy: 1 GiB read, 1 GiB written


def short(name):
    """`gemm_kernel<true, false, ...>` from a demangled kernel symbol."""
    m = re.search(r"gist::\(anonymous namespace\)::(\w+)(<[^()]*>)?", name)
    return (m.group(1) + (m.group(2) or "")) if m else name[:60]


def variant_symbol(variant):
    """Regex over short kernel names that a library profiler variant launches."""
    b = lambda s: "true" if s else "false"
    m = re.fullmatch(r"gemm_(f32|bf16)_([KR])([KR])_([vs])([vs])(_n)?", variant)
    if m:
        dt, ak, bk, av, bv, nar = m.groups()
        args = ", ".join([b(ak == "K"), b(bk == "K"), b(av == "v"), b(bv == "v"), b(dt == "bf16"),
                          b(nar is not None)])
        return re.escape(f"gemm_kernel<{args}>") + "$"
    m = re.fullmatch(r"gemm_bf16_direct_([KR])([KR])", variant)
    if m:
        ak, bk = m.groups()
        return re.escape(f"gemm_bf16_direct_kernel<{b(ak == 'K')}, {b(bk == 'K')},")
    m = re.fullmatch(r"spmm_v(\d+)_l(\d+)", variant)
    if m:
        v, l = m.groups()
        return (re.escape(f"spmm_wide_kernel<{v}>") if l == "64"
                else re.escape(f"spmm_kernel<{v}, {l}>")) + "$"
    table = {
        "gemm_bf16_packed": r"gemm_bf16_kernel<", "gemm_bf16_fixup": r"fixup_bf16_kernel",
        "cvt_bf16_K": r"cvt_bf16_kernel<true,", "cvt_bf16_R": r"cvt_bf16_kernel<false,",
        "gemm_streamk_fixup": r"streamk_fixup", "subagg_gather_rows": r"subagg_gather_rows_kernel<",
        "spmm_tile": r"spmm_tile_kernel",
        "subagg_gather": r"subagg_gather_kernel<", "gather_slice": r"gather_kernel",
        "subagg_scatter": r"scatter_kernel", "sgd_update": r"sgd_kernel",
        "relu_mask": r"relu_mask_kernel", "subagg_mean": r"subagg_mean_kernel",
        "gat_scores": r"gat_scores_kernel", "gat_softmax": r"gat_softmax_kernel",
        "gat_edge_grad": r"gat_edge_grad_kernel<", "gat_mirror": r"gat_mirror_kernel",
        "gat_mirror_sums": r"gat_mirror_sums_kernel", "gat_rank2": r"gat_rank2_kernel",
        "gat_gemv_t": r"gat_gemv_partial_kernel",
    }
    return "^" + table[variant] if variant in table else None


def top_kernels(db):
    """(short name, calls, total ms, average us, percent); rocpd reports us."""
    c = sqlite3.connect(db)
    rows = c.execute("select name, total_calls, total_duration, average, percentage "
                     "from top_kernels").fetchall()
    return [(short(n), k, t / 1e3, a, p) for n, k, t, a, p in rows]


def counter_values(db):
    """short kernel name -> per-dispatch counter values (KiB), dispatch order."""
    c = sqlite3.connect(db)
    out = collections.defaultdict(list)
    for name, val in c.execute("select kernel_name, value from counters_collection "
                               "order by dispatch_id"):
        out[short(name)].append(val)
    return out


def calib_factor(db):
    vals = counter_values(db)
    v = [x for k, xs in vals.items() if k.startswith("gather_kernel") for x in xs]
    if not v:
        raise SystemExit(f"{db}: no copy dispatches")
    return COPY_BYTES / (sum(v) / len(v))   # bytes per counter unit


def variant_bytes(variant, vals, per_step):
    """Mean counter value over the last `per_step` dispatches of a variant's
    kernels (the timed rounds' launch mix, not the warm-up's)."""
    pat = variant_symbol(variant)
    if pat is None:
        return None, 0
    rx = re.compile(pat)
    seq = [x for k, xs in vals.items() if rx.search(k) for x in xs]
    if not seq:
        return None, 0
    seq = seq[-per_step:] if per_step else seq
    return sum(seq) / len(seq), len(seq)


def main():
    ap = argparse.ArgumentParser()
    for k in ("bench", "trace", "fetch", "write", "calib_fetch", "calib_write", "title", "out"):
        ap.add_argument("--" + k.replace("_", "-"), required=True)
    ap.add_argument("--cmd", action="append", default=[])
    ap.add_argument("--workload", required=True, help="config name the run used (c1..c7)")
    a = ap.parse_args()
    res = json.load(open(a.bench))
    steps = res["steps"]
    kf, kw = calib_factor(a.calib_fetch), calib_factor(a.calib_write)
    fv, wv = counter_values(a.fetch), counter_values(a.write)
    L = [f"# {a.title}", "", "Commands (rocprofv3 runs, then this summary):", "", "```"]
    L += a.cmd + ["```", ""]
    L += [f"Bench line of the trace run: value {res['value']} {res['unit']} per sub-GCN step, "
          f"{res['ms_per_step']} ms per step, dtype {res['dtype']}, {steps} timed steps.", ""]
    rf = res.get("roofline")
    if rf:
        L += [f"Roofline kernel: `{rf['kernel']}`, {rf['achieved']} {rf['unit']} of {rf['peak']} "
              f"({100 * rf['frac']:.1f}%), mean launch {rf['avg_launch_us']} us (library HIP events).", ""]
    L += ["rocprofv3 kernel statistics (all dispatches of the run, warm-up included):", "",
          "| kernel | calls | total ms | avg us | % |", "|---|---|---|---|---|"]
    for n, k, t, av, p in top_kernels(a.trace)[:16]:
        L.append(f"| `{n}` | {k} | {t:.2f} | {av:.1f} | {p:.1f} |")
    L += ["", "Library HIP-event timing (timed steps only) and calibrated HBM traffic per dispatch:",
          "", "| variant | launches | avg us | TFLOP/s | GB/s algorithmic | fetched MB | written MB |",
          "|---|---|---|---|---|---|---|"]
    records = []
    for var, v in list(res["kernels"].items())[:14]:
        per_step = max(1, round(v["launches"] / steps))
        f, nf = variant_bytes(var, fv, per_step)
        w, nw = variant_bytes(var, wv, per_step)
        fm = f"{f * kf / 1e6:.1f}" if f is not None else ""
        wm = f"{w * kw / 1e6:.1f}" if w is not None else ""
        L.append(f"| {var} | {v['launches']} | {v['avg_us']} | {v.get('tflops', '')} | "
                 f"{v.get('gbs', '')} | {fm} | {wm} |")
        if f is not None and w is not None:
            records.append({"variant": var, "workload": a.workload, "dtype": res["dtype"],
                            "fetch_bytes": round(f * kf), "write_bytes": round(w * kw),
                            "dispatches": min(nf, nw), "src_sha256": res["kernel_src_sha256"]})
    L += ["", f"Counter calibration: a 1 GiB copy reads {COPY_BYTES / kf:.0f} units of "
              f"FETCH_SIZE and {COPY_BYTES / kw:.0f} of WRITE_SIZE, so one unit is "
              f"{kf:.1f} bytes fetched and {kw:.1f} bytes written (counters averaged over the "
              "last step's dispatches of each variant).", "",
          "Traffic records read by bench.py (valid while the kernel sources hash as stated):", "",
          "```traffic"]
    L += [json.dumps(r) for r in records] + ["```"]
    open(a.out, "w").write("\n".join(L) + "\n")
    print("\n".join(L))


if __name__ == "__main__":
    main()
