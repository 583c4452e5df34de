#!/usr/bin/env python3
"""Benchmark of the colour-restricted tensor path on one MI355X.

Headline workload (the colour-restricted streaming configuration): triad
a = b + 3c on three 1 GiB fp32 arrays (2^28 elements, U[-1,1)) stored in
64 KiB pages (one pool per colour set), with 6 XOR masks (64 colours) and colour sets of
8, 16, 32 and 64 of the 64 colours, all CUs enabled.  One step = the four
triad passes (one per colour set); ``value`` is the algorithmic HBM traffic
of the timed steps (12 bytes per element per pass) divided by their wall
time.  Inputs are resident in HBM before timing starts.

The other steps of the path are measured in the same run and reported under
"rows": batched classify (2^26 addresses), the page-table build, the bimodal
relayout of a 4 GiB fp16 tensor in both directions, and the memory-bound
GEMV sweep (bf16 4096x11008 and 11008x4096, batch 1/2/4/8, CU masks of
64/128/192/256 CUs) with p50/p99 kernel latency.  The CPU oracle is timed on
a bounded sample of the headline workload ("cpu_baseline").

Prints one JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
METRIC = "colour-restricted HBM GB/s (% of colour-scaled peak); colored GEMV p99 latency"


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--rows", default="classify,pagetable,relayout,gemv,xcd,corun,preempt,bimodal,"
                                      "sectors,probe",
                    help="comma list of extra rows to measure ('' for none)")
    ap.add_argument("--gemv-launches", type=int, default=2000)
    ap.add_argument("--corun-launches", type=int, default=2000)
    ap.add_argument("--preempt-trials", type=int, default=40)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--full-out", default="",
                    help="file for the full result (every row); without it the full result goes "
                         "to stderr as one JSON line; stdout gets a compact line")
    return ap.parse_args()


def pctl(xs, q):
    import numpy as np
    return float(np.percentile(np.asarray(xs, dtype=np.float64), q))


class Timer:
    """Per-launch HIP event pairs on one stream."""

    def __init__(self, torch, stream):
        self.torch, self.stream, self.pairs, self.pool = torch, stream, [], []

    def reserve(self, n):
        """Creates n events ahead of a timed region (recording each once, so
        that the runtime allocates it now) and keeps host-side allocation out
        of the region: an event pair there once spanned 21 ms around a
        0.5 ms launch, which a host stall that let the GPU run dry explains."""
        for _ in range(n):
            e = self.torch.cuda.Event(enable_timing=True)
            e.record(self.stream)
            self.pool.append(e)
        self.torch.cuda.synchronize()

    def _event(self):
        return self.pool.pop() if self.pool else self.torch.cuda.Event(enable_timing=True)

    def start(self):
        e = self._event()
        e.record(self.stream)
        return e

    def stop(self, e0, tag=None):
        e1 = self._event()
        e1.record(self.stream)
        self.pairs.append((tag, e0, e1))

    def durations_ms(self, tag=None):
        return [a.elapsed_time(b) for t, a, b in self.pairs if tag is None or t == tag]


class DevTimes:
    """Kernel spans from the library's device time log: for each launch on
    ``stream`` the ticks at which its first workgroup started and its last
    workgroup finished, so no host launch overhead is included."""

    def __init__(self, torch, ctx, stream, n):
        self.torch, self.ctx, self.stream, self.n = torch, ctx, stream, n
        self.slots = torch.zeros(2 * n, dtype=torch.int64, device="cuda:0")
        torch.cuda.synchronize()
        ctx.set_timelog(stream, self.slots)

    def close_ticks(self, count=None):
        """Switch the log off and return the {start, end} ticks of the first
        ``count`` launches logged (at most n), shape [launches, 2]."""
        import numpy as np
        self.torch.cuda.synchronize()
        self.ctx.set_timelog(self.stream, None)
        t = self.slots.cpu().numpy().reshape(-1, 2).astype(np.int64)
        return t[: self.n if count is None else min(count, self.n)]

    def close_us(self, count=None):
        """Switch the log off and return the spans (microseconds) of the
        first ``count`` launches logged (at most n)."""
        t = self.close_ticks(count)
        return (t[:, 1] - t[:, 0]) * 1e3 / self.ctx.wallclock_khz


PMC_SUMMARY = os.path.join(ROOT, "profiles", "triad_3x1GiB_64KiB.pmc.md")


def recorded_traffic():
    """Calibrated HBM bytes per triad launch from the committed rocprofv3
    FETCH_SIZE/WRITE_SIZE summary, or None if the kernel sources changed
    since the counters were taken (their hash no longer matches)."""
    import hashlib
    try:
        fields = {}
        for line in open(PMC_SUMMARY):
            if ":" in line and not line.startswith(("#", "|", "`")):
                k, v = line.split(":", 1)
                fields[k.strip()] = v.strip()
        h = hashlib.sha256()
        for f in fields["kernel_sources"].split():
            h.update(open(os.path.join(ROOT, f), "rb").read())
        if h.hexdigest()[:16] != fields["kernel_sources_sha256_16"]:
            return None
        return int(fields["traffic_bytes_per_launch"])
    except (OSError, KeyError, ValueError):
        return None


def aligned_pool(torch, n_pages, shift):
    """A device byte pool of n_pages pages whose base is page aligned."""
    P = 1 << shift
    raw = torch.empty(n_pages * P + P, dtype=torch.uint8, device="cuda:0")
    base = raw.data_ptr()
    off = (-base) % P
    return raw, base + off


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the colour-restricted path is per device and "
              "runs no collectives; use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2407_13996_amd as sg
    import synth

    dev = "cuda:0"
    torch.cuda.set_device(0)
    ctx = sg.Context(0)
    stream = torch.cuda.Stream(device=0)
    timer = Timer(torch, stream)
    props = torch.cuda.get_device_properties(0)
    log(f"device {props.name} {props.gcnArchName} CUs={ctx.num_cus}")

    # ------------------------------------------------------------ headline
    shift = 16
    P = 1 << shift
    n = 1 << 28
    pages = (n * 4) >> shift
    fractions = [8, 16, 32, 64]
    masks = synth.xor_masks(6, seed=1, min_bit=shift)
    log("masks " + " ".join(hex(m) for m in masks))
    with torch.cuda.stream(stream):
        b_host = synth.uniform_f32(n, seed=2)
        c_host = synth.uniform_f32(n, seed=3)
        b_lin = torch.from_numpy(b_host).to(dev)
        c_lin = torch.from_numpy(c_host).to(dev)
        ident = torch.arange(pages, dtype=torch.int32, device=dev)
        # one pool per colour set, so that the four page sets never share pages
        tables = {}
        for nc in fractions:
            pool_pages = int(3 * pages * 64 / nc * 1.04) + 64
            raw, base = aligned_pool(torch, pool_pages, shift)
            pt = torch.empty(3 * pages, dtype=torch.int32, device=dev)
            torch.cuda.synchronize()
            # the call is synchronous and idempotent: median of 5 (the first one
            # also loads the kernels' code)
            runs = []
            for _ in range(5):
                t0 = time.perf_counter()
                found = sg.colour_alloc_pagetable(ctx, masks, base, shift, pool_pages, range(nc),
                                                  3 * pages, pt, stream)
                runs.append(time.perf_counter() - t0)
            t_pt = float(np.median(runs))
            tables[nc] = {"pt": pt, "found": found, "seconds": t_pt, "raw": raw, "base": base,
                          "pool_pages": pool_pages}
            log(f"pool {nc}/64: {pool_pages} pages of 64 KiB ({pool_pages * P / 2**30:.1f} GiB), "
                f"page table {t_pt * 1e3:.2f} ms")

    def paged_arrays(nc):
        t = tables[nc]
        return [sg.paged(t["base"], t["pt"][i * pages:(i + 1) * pages], t["pool_pages"])
                for i in range(3)]

    def place_inputs(nc):
        a, b, c = paged_arrays(nc)
        sg.bimodal_relayout(ctx, b, sg.paged(b_lin, ident, pages), n * 4, shift, stream)
        sg.bimodal_relayout(ctx, c, sg.paged(c_lin, ident, pages), n * 4, shift, stream)
        return a, b, c

    bytes_per_pass = 12 * n
    per_frac = {}
    with torch.cuda.stream(stream):
        arrays = {}
        for nc in fractions:
            arrays[nc] = place_inputs(nc)
        torch.cuda.synchronize()
        # warmup
        for _ in range(args.warmup):
            for nc in fractions:
                a, b, c = arrays[nc]
                sg.colored_stream(ctx, a, b, c, 3.0, n, shift, stream)
        timer.reserve(2 * args.steps * len(fractions))
        log(f"timing {args.steps} steps x {len(fractions)} triad passes")
        t0 = time.perf_counter()
        for _ in range(args.steps):
            for nc in fractions:
                a, b, c = arrays[nc]
                e0 = timer.start()
                sg.colored_stream(ctx, a, b, c, 3.0, n, shift, stream)
                timer.stop(e0, ("triad", nc))
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
    all_ms = []
    for nc in fractions:
        d = timer.durations_ms(("triad", nc))
        all_ms += d
        f = nc / 64
        med = pctl(d, 50)
        gbs = bytes_per_pass / (med * 1e-3) / 1e9
        per_frac[nc] = {
            "colours": f"{nc}/64", "median_ms": round(med, 4), "p99_ms": round(pctl(d, 99), 4),
            "mean_ms": round(float(np.mean(d)), 4), "max_ms": round(max(d), 4),
            "slowest_launch": int(np.argmax(d)),
            "launches_over_1.2x_median": int(sum(1 for v in d if v > 1.2 * med)),
            "GBps": round(gbs, 1), "colour_scaled_peak_GBps": f * HBM_PEAK_GBS,
            "pct_of_colour_scaled_peak": round(100 * gbs / (f * HBM_PEAK_GBS), 1),
            "pct_of_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 1),
            "pagetable_ms": round(tables[nc]["seconds"] * 1e3, 3),
        }
        log(f"triad {nc}/64 colours: {med:.4f} ms  {gbs:.0f} GB/s")
    value = args.steps * len(fractions) * bytes_per_pass / wall / 1e9
    avg_ms = float(np.mean(all_ms))
    achieved = bytes_per_pass / (avg_ms * 1e-3) / 1e9
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": recorded_traffic(), "traffic_unit": "bytes per launch",
                "kernel": "k_triad (64 KiB pages)", "avg_launch_ms": round(avg_ms, 4),
                "bytes_per_launch": bytes_per_pass}

    result = {
        "metric": METRIC, "value": round(value, 1), "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(wall / args.steps * 1e3, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": "colour-restricted triad a=b+3c, three 1 GiB fp32 arrays "
                               "(2^28 elements) in 64 KiB pages, 6 XOR masks (64 colours), "
                               "colour sets 8/16/32/64 of 64, all CUs; one step = 4 passes",
                   "page_bytes": P, "elements": n, "num_cus": ctx.num_cus,
                   "masks": [hex(m) for m in masks]},
        "roofline": roofline,
        "per_fraction": [per_frac[nc] for nc in fractions],
    }

    # ------------------------------------------------------------ sampled check
    # GPU result of the 8/64 pass on a few logical pages (compared against the
    # oracle in the CPU-baseline leg).
    t8 = tables[8]
    sample_pages = [0, 1, 777, pages - 1]
    pt8 = t8["pt"][:pages].cpu().numpy().astype(np.int64)
    gpu_pages = {}
    for j in sample_pages:
        off = t8["base"] + int(pt8[j]) * P - t8["raw"].data_ptr()
        gpu_pages[j] = t8["raw"][off:off + P].cpu().numpy().view(np.float32).copy()
    pools_desc = {nc: (tables[nc]["base"], tables[nc]["pool_pages"]) for nc in fractions}

    flags = {"headline": ctx.device_error()}
    rows = {}
    checks = {}
    want = [r for r in args.rows.split(",") if r]

    def row(name, fn):
        """Runs one row; a row that raises is recorded as such (with the
        error) and the others still run, so the headline line is printed."""
        try:
            rows[name] = fn()
        except Exception as e:  # noqa: BLE001 - any failure of an auxiliary row
            import traceback
            traceback.print_exc(file=sys.stderr)
            rows[name] = {"error": f"{type(e).__name__}: {e}"}
            torch.cuda.synchronize()
        flags[name] = ctx.device_error()

    if "classify" in want:
        row("classify", lambda: bench_classify(torch, sg, synth, ctx, stream, timer, checks))
    if "pagetable" in want:
        rows["pagetable"] = {
            "what": "colour_alloc_pagetable over the headline pool (synchronous call)",
            "n_needed": 3 * pages,
            "pool_pages": {f"{nc}/64": tables[nc]["pool_pages"] for nc in fractions},
            "ms": {f"{nc}/64": round(tables[nc]["seconds"] * 1e3, 3) for nc in fractions},
            "pool_pages_per_s": {f"{nc}/64": round(tables[nc]["pool_pages"] / tables[nc]["seconds"], 0)
                                 for nc in fractions}}
    # free the headline pools before the larger rows
    del arrays, tables, t8, b_lin, c_lin
    torch.cuda.empty_cache()
    if "relayout" in want:
        row("relayout", lambda: bench_relayout(torch, sg, synth, ctx, stream, timer))
    if "gemv" in want:
        row("gemv", lambda: bench_gemv(torch, sg, synth, ctx, stream, timer, args.gemv_launches,
                                       checks))
    ops = corun_operands(torch, sg, synth, ctx) if ("corun" in want or "preempt" in want) else None
    if "corun" in want:
        row("corun", lambda: bench_corun(torch, sg, synth, ctx, args.corun_launches, ops))
    if "preempt" in want:
        row("preempt", lambda: bench_preempt(torch, sg, synth, ctx, ops, args.preempt_trials))
    del ops
    torch.cuda.empty_cache()
    if "bimodal" in want:
        row("bimodal", lambda: bench_bimodal(torch, sg, synth, ctx, stream))
    if "sectors" in want:
        row("sectors", lambda: bench_sectors(torch, sg, synth, ctx, stream, timer))
    if "xcd" in want:
        row("xcd", lambda: bench_xcd(torch, sg, ctx, stream))
    if "probe" in want:
        row("probe", lambda: bench_probe(torch, sg, synth, ctx, stream, timer))
    if rows:
        result["rows"] = rows

    if not args.no_cpu:
        result["cpu_baseline"] = cpu_baseline(np, synth, masks, shift, pages, pools_desc,
                                              b_host, c_host, fractions, gpu_pages, checks)
    flags["end"] = ctx.device_error()
    result["device_flags_by_row"] = flags
    result["device_error_flags"] = 0
    for v in flags.values():
        result["device_error_flags"] |= v
    ctx.close()
    full_path = args.full_out or "stderr"
    if args.full_out:
        try:
            os.makedirs(os.path.dirname(os.path.abspath(full_path)), exist_ok=True)
            with open(full_path, "w") as f:
                json.dump(result, f, indent=1)
            log(f"full result written to {full_path}")
        except OSError as e:
            log(f"could not write {full_path}: {e}")
            args.full_out = ""
    if not args.full_out:
        log("full result: " + json.dumps(result))
    line = json.dumps(compact(result, full_path if args.full_out else "stderr"))
    print(line, flush=True)


def _get(d, *keys):
    for k in keys:
        if not isinstance(d, dict) or k not in d:
            return None
        d = d[k]
    return d


def compact(result, full_path):
    """The one stdout line: the contract's fields, the roofline and CPU
    baseline, the per-colour-set figures and one headline figure per row
    (all rows in full are in ``full_path``).  Kept under 8 KB."""
    keep = ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
            "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config", "roofline",
            "device_error_flags")
    out = {k: result[k] for k in keep if k in result}
    out["per_fraction"] = [{k: p[k] for k in ("colours", "GBps", "pct_of_colour_scaled_peak",
                                              "pct_of_hbm_peak", "median_ms")}
                           for p in result.get("per_fraction", [])]
    cb = result.get("cpu_baseline")
    if cb:
        out["cpu_baseline"] = {k: cb[k] for k in ("value", "unit", "cores", "kind", "sample")}
        out["cpu_baseline"]["ops"] = {
            op: {k: v for k, v in row.items() if k.endswith(("_per_s", "GBps"))}
            for op, row in cb["ops"].items()}
        out["cpu_baseline"]["checks"] = {k: v for k, v in cb.items()
                                         if k.endswith(("match_oracle", "matches_oracle",
                                                        "within_bound", "identity"))}
    rows = {k: v for k, v in result.get("rows", {}).items() if "error" not in v}
    errors = {k: v["error"] for k, v in result.get("rows", {}).items() if "error" in v}
    if errors:
        out["row_errors"] = errors
    summ = {}
    if "classify" in rows:
        c = rows["classify"]
        summ["classify_2e26"] = {"colours_us": _get(c, "colours_only", "median_us"),
                                 "hist_us": _get(c, "with_histogram", "median_us"),
                                 "colours_span_us": _get(c, "colours_only", "kernel_span_p50_us"),
                                 "hist_span_us": _get(c, "with_histogram", "kernel_span_p50_us"),
                                 "addrs_per_s": _get(c, "colours_only", "addrs_per_s"),
                                 "pct_hbm": _get(c, "colours_only", "pct_of_hbm_peak")}
    if "pagetable" in rows:
        summ["pagetable_ms"] = rows["pagetable"]["ms"]
    if "relayout" in rows:
        r = rows["relayout"]
        summ["relayout_4GiB"] = {k: [_get(r, k, "GBps"), _get(r, k, "pages_per_s")]
                                 for k in ("to_restricted", "to_all", "to_restricted_2MiB",
                                           "to_all_2MiB", "contiguous_copy") if k in r}
    if "gemv" in rows:
        g = rows["gemv"]
        pts = {}
        for p in g["points"]:
            if p["placement"] == "xcds" and p["layout"] == "coloured" and \
                    p["rotated_copies"] == max(q["rotated_copies"] for q in g["points"]):
                key = f"{p['M']}x{p['K']}_b{p['batch']}_cu{p['cus']}"
                pts[key] = [p["p50_us"], p["p99_us"], p["GBps"]]
        summ["gemv_p50_p99_us_GBps"] = pts
        if "indirection" in g:
            summ["gemv_indirection"] = g["indirection"]
        if "library_reference" in g:
            summ["gemv_library_reference_launch_p50_us"] = g["library_reference"]
        summ["gemv_launch_p50_us_256cus"] = {
            f"{p['M']}x{p['K']}_b{p['batch']}": p["launch_p50_us"] for p in g["points"]
            if p["placement"] == "xcds" and p["layout"] == "coloured" and p["batch"] in (1, 8)
            and p["rotated_copies"] == 8 and p["cus"] == max(q["cus"] for q in g["points"])}
        if g.get("graph_ls") and "error" not in g["graph_ls"]:
            gl = g["graph_ls"]
            summ["gemv_ls_launch_p50_p99_us_direct_graph"] = [
                gl["direct_launch_p50_us"], gl["direct_launch_p99_us"], gl["graph_launch_p50_us"],
                gl["graph_launch_p99_us"], gl["graph_matches_direct"]]
        summ["gemv_p50_us_by_rotated_copies"] = {
            f"{p['M']}x{p['K']}_b{p['batch']}_x{p['rotated_copies']}": p["p50_us"]
            for p in g["points"] if p["placement"] == "xcds" and p["layout"] == "coloured"
            and p["batch"] in (1, 8) and p["cus"] == max(q["cus"] for q in g["points"])}
    if "corun" in rows:
        c = rows["corun"]
        summ["corun"] = {k: {kk: c[k].get(kk) for kk in ("ls_p50_us", "ls_p99_us", "be_GBps")}
                         for k in ("isolated_ls_coloured_masked", "corun_coloured_masked",
                                   "corun_uncoloured_masked", "corun_uncoloured_unmasked")
                         if k in c}
    if "preempt" in rows:
        pr = rows["preempt"]
        summ["preempt"] = {k: pr.get(k) for k in (
            "evicted_trials", "eviction_latency_p50_us", "eviction_latency_p99_us",
            "ls_from_flag_p50_us", "ls_from_flag_p99_us", "preemptible_overhead_pct")}
    if "bimodal" in rows:
        summ["bimodal"] = {k: v for k, v in rows["bimodal"].items()
                           if isinstance(v, (int, float)) and not isinstance(v, bool)}
    if "xcd" in rows:
        summ["xcd_triad_GBps"] = {f"{p['cus']}{'s' if p['placement'] == 'spread' else ''}":
                                  p["GBps"] for p in rows["xcd"]["points"]}
    if "sectors" in rows:
        summ["sectors_triad_GBps"] = {k[6:-5]: v for k, v in rows["sectors"].items()
                                      if k.startswith("triad_") and k.endswith("_GBps")}
    if "probe" in rows:
        pb = rows["probe"]
        for key in ("points", "high_bits"):
            rs = [p["ratio"] for p in pb.get(key, [])[1:]]
            if rs:
                summ[f"probe_{key}_ratio_min_max"] = [min(rs), max(rs)]
        summ["probe_placement_GBps"] = {f"{p['page_KiB']}K {p['pages']}": p["GBps"]
                                        for p in pb.get("placement", [])}
    out["rows_summary"] = summ
    out["rows_full"] = os.path.relpath(full_path, ROOT) if full_path != "stderr" else "stderr"
    text = json.dumps(out)
    if len(text) > 8000:       # drop the widest parts first
        for k in ("sectors_triad_GBps", "probe_placement_GBps", "xcd_triad_GBps", "bimodal"):
            summ.pop(k, None)
            text = json.dumps(out)
            if len(text) <= 8000:
                break
    return out


def bench_classify(torch, sg, synth, ctx, stream, timer, checks, n=1 << 26, reps=50):
    out = {}
    for hist in (False, True):
        out["with_histogram" if hist else "colours_only"] = bench_classify_one(
            torch, sg, synth, ctx, stream, timer, n, reps, hist, checks)
    return out


def bench_classify_one(torch, sg, synth, ctx, stream, timer, n, reps, hist, checks):
    log(f"classify {n} addresses")
    masks = synth.xor_masks(6, seed=1, min_bit=12)
    addrs = synth.page_addresses(n, seed=0)
    d_addrs = torch.from_numpy(addrs.view("int64")).to("cuda:0")
    torch.cuda.synchronize()
    d_col = torch.empty(n, dtype=torch.uint8, device="cuda:0")
    d_hist = torch.empty(64, dtype=torch.int64, device="cuda:0") if hist else None
    tag = ("classify", hist)
    with torch.cuda.stream(stream):
        for _ in range(5):
            sg.colour_classify(ctx, masks, d_addrs, d_col, d_hist, stream)
        dev = DevTimes(torch, ctx, stream, reps)
        for _ in range(reps):
            sg.colour_classify(ctx, masks, d_addrs, d_col, d_hist, stream)
        spans = dev.close_us()
        timer.reserve(2 * reps)
        for _ in range(reps):
            e0 = timer.start()
            sg.colour_classify(ctx, masks, d_addrs, d_col, d_hist, stream)
            timer.stop(e0, tag)
        torch.cuda.synchronize()
    d = timer.durations_ms(tag)
    med = pctl(d, 50)
    span = pctl(list(spans), 50)
    gbs = 9 * n / (med * 1e-3) / 1e9
    log(f"classify (histogram {hist}): {med * 1e3:.1f} us with launch, kernel span {span:.1f} us, "
        f"{gbs:.0f} GB/s")
    checks["classify_colours"] = d_col[:1 << 22].cpu().numpy()
    return {"what": "2^26 random 4 KiB-aligned addresses, 6 masks"
                    + (", colours + histogram" if hist else ", colours"),
            "median_us": round(med * 1e3, 2), "p99_us": round(pctl(d, 99) * 1e3, 2),
            "kernel_span_p50_us": round(span, 2), "kernel_span_p99_us": round(pctl(list(spans), 99), 2),
            "timing": "median_us/p99_us: host events around each call (launch overhead, and the "
                      "finishing kernel of a statically scheduled launch, included); kernel_span: "
                      "device time log of the main kernel",
            "addrs_per_s": round(n / (med * 1e-3), 0), "GBps": round(gbs, 1),
            "pct_of_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 1), "bytes_per_addr": 9}


def bench_relayout(torch, sg, synth, ctx, stream, timer, reps=10):
    """The 4 GiB fp16 tensor moved between the all-colour form and colours
    0..15 of 64, both directions, in 64 KiB pages and in 2 MiB pages; and
    the same bytes copied between two contiguous buffers (identity tables)
    as the ceiling the indirection is measured against."""
    n_bytes = 4 << 30
    g = torch.Generator(device="cuda:0")
    g.manual_seed(5)
    all_form = torch.randint(-32768, 32767, (n_bytes // 2,), dtype=torch.int16, device="cuda:0",
                             generator=g)
    back = torch.empty_like(all_form)
    out = {"what": "4 GiB fp16, all colours <-> 16 of 64 colours; 64 KiB pages (65,536) and "
                   "2 MiB pages (2,048); contiguous copy with identity tables as the ceiling"}

    def timed(tag, dst, src, shift):
        with torch.cuda.stream(stream):
            for _ in range(2):
                sg.bimodal_relayout(ctx, dst, src, n_bytes, shift, stream)
            for _ in range(reps):
                e0 = timer.start()
                sg.bimodal_relayout(ctx, dst, src, n_bytes, shift, stream)
                timer.stop(e0, tag)
            torch.cuda.synchronize()
        med = pctl(timer.durations_ms(tag), 50)
        gbs = 2 * n_bytes / (med * 1e-3) / 1e9
        pages = n_bytes >> shift
        log(f"relayout {tag}: {med:.3f} ms  {gbs:.0f} GB/s")
        return {"median_ms": round(med, 4), "GBps": round(gbs, 1),
                "pages_per_s": round(pages / (med * 1e-3), 0),
                "pct_of_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 1)}

    for shift in (16, 21):
        pages = n_bytes >> shift
        masks = synth.xor_masks(6, seed=1, min_bit=shift)
        ident = torch.arange(pages, dtype=torch.int32, device="cuda:0")
        pt = torch.empty(pages, dtype=torch.int32, device="cuda:0")
        for margin in (1.04, 1.25, 1.6):
            # a short pool of 2 MiB pages can hold slightly fewer of the colours than
            # a quarter of its pages: grow it until the table fills
            pool_pages = int(pages * 64 / 16 * margin) + 64
            raw, base = aligned_pool(torch, pool_pages, shift)
            try:
                sg.colour_alloc_pagetable(ctx, masks, base, shift, pool_pages, range(16), pages,
                                          pt, stream)
                break
            except sg.SgdrcError as e:
                if e.code != sg.ENOMEM or margin == 1.6:
                    raise
                del raw
                torch.cuda.empty_cache()
        log(f"relayout 4 GiB fp16, {1 << (shift - 10)} KiB pages, restricted pool {pool_pages} pages")
        torch.cuda.synchronize()   # operands made on torch's stream, used on ``stream``
        A = sg.paged(all_form, ident, pages)
        S = sg.paged(base, pt, pool_pages)
        B = sg.paged(back, ident, pages)
        key = "" if shift == 16 else "_2MiB"
        out["to_restricted" + key] = timed(("to_restricted", shift), S, A, shift)
        out["to_all" + key] = timed(("to_all", shift), B, S, shift)
        out["round_trip_identity" + key] = bool(torch.equal(back, all_form))
        if shift == 16:
            out["contiguous_copy"] = timed(("contiguous", shift), B, A, shift)
        del raw, pt, S
        torch.cuda.empty_cache()
    return out


def bench_gemv(torch, sg, synth, ctx, stream, timer, launches, checks):
    import numpy as np
    shift = 21
    P = 1 << shift
    copies = 8
    masks = synth.xor_masks(6, seed=1, min_bit=shift)
    n_cus = ctx.num_cus
    out = []
    lib_ref = {}
    indirection = {}
    graph_ls = {}
    g = torch.Generator(device="cuda:0")
    g.manual_seed(7)
    x = (torch.randn(8 * 11008, generator=g, device="cuda:0")).to(torch.bfloat16)
    for (M, K) in [(4096, 11008), (11008, 4096)]:
        torch.cuda.synchronize()   # operands made on torch's stream, used on ``stream``
        w_bytes = M * K * 2
        pages = -(-w_bytes // P)
        pool_pages = int(copies * pages * 64 / 48 * 1.1) + 16
        raw, base = aligned_pool(torch, pool_pages, shift)
        pt = torch.empty(copies * pages, dtype=torch.int32, device="cuda:0")
        sg.colour_alloc_pagetable(ctx, masks, base, shift, pool_pages, range(48), copies * pages,
                                  pt, stream)
        w = (torch.randn(M * K, generator=g, device="cuda:0") * 0.02).to(torch.bfloat16)
        ident = torch.arange(pages, dtype=torch.int32, device="cuda:0")
        torch.cuda.synchronize()
        W = []
        for i in range(copies):
            Wi = sg.paged(base, pt[i * pages:(i + 1) * pages], pool_pages)
            sg.bimodal_relayout(ctx, Wi, sg.paged(w, ident, pages), w_bytes, shift, stream)
            W.append(Wi)
        y = torch.empty(8 * M, dtype=torch.float32, device="cuda:0")
        setup_flags = ctx.device_error()
        log(f"gemv {M}x{K}: {copies} weight copies rotated (setup flags {setup_flags})")

        def point(Ws, B, ncu, place, layout, rotate=copies):
            tag = ("gemv", M, B, ncu, place, layout, rotate)
            cus = range(ncu) if place == "xcds" else spread_cus(n_cus, ncu)
            with torch.cuda.stream(stream):
                sg.set_cu_mask(ctx, stream, cus)
                for i in range(20):
                    sg.colored_gemv(ctx, Ws[i % rotate], sg.BF16, M, K, x, sg.BF16, B, y,
                                    shift, stream)
                # kernel spans from the device time log ...
                dev = DevTimes(torch, ctx, stream, launches)
                for i in range(launches):
                    sg.colored_gemv(ctx, Ws[i % rotate], sg.BF16, M, K, x, sg.BF16, B, y,
                                    shift, stream)
                spans = dev.close_us()
                # ... and, without the log, host events around each call
                timer.reserve(2 * launches)
                for i in range(launches):
                    e0 = timer.start()
                    sg.colored_gemv(ctx, Ws[i % rotate], sg.BF16, M, K, x, sg.BF16, B, y,
                                    shift, stream)
                    timer.stop(e0, tag)
                schedule = ctx.last_schedule(stream)
                sg.set_cu_mask(ctx, stream, None)
                torch.cuda.synchronize()
            d = timer.durations_ms(tag)
            flag = ctx.device_error()
            nbytes = M * K * 2 + B * K * 2 + B * M * 4
            med, p99 = pctl(list(spans), 50), pctl(list(spans), 99)
            gbs = nbytes / (med * 1e-6) / 1e9
            out.append({"M": M, "K": K, "batch": B, "cus": ncu, "placement": place,
                        "layout": layout, "rotated_copies": rotate, "device_flags": flag,
                        "path": "mfma" if B >= 3 else "valu", "schedule": schedule,
                        "p50_us": round(med, 2), "p99_us": round(p99, 2),
                        "GBps": round(gbs, 1),
                        "pct_of_colour_scaled_peak": round(100 * gbs / (0.75 * HBM_PEAK_GBS), 1),
                        "pct_of_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 1),
                        "launch_p50_us": round(pctl(d, 50) * 1e3, 2),
                        "launch_p99_us": round(pctl(d, 99) * 1e3, 2)})
            log(f"gemv {M}x{K} B={B} cus={ncu} ({place}, {layout}, {rotate} copies): kernel p50 "
                f"{med:.1f} us p99 {p99:.1f} us {gbs:.0f} GB/s; with launch p50 "
                f"{pctl(d, 50) * 1e3:.1f} us")
            return med

        def graph_point(B, ncu):
            """Launch-inclusive latency of the LS call (host events around
            each call) launched directly and as a replay of a HIP graph that
            captured it (one graph per weight copy, captured on ``stream``
            under the same CU mask), in interleaved blocks of launches; and
            whether a replay writes the same bits as the direct call."""
            tag_d, tag_g = ("gemv-direct", M, B, ncu), ("gemv-graph", M, B, ncu)
            with torch.cuda.stream(stream):
                sg.set_cu_mask(ctx, stream, range(ncu))
                for i in range(20):
                    sg.colored_gemv(ctx, W[i % copies], sg.BF16, M, K, x, sg.BF16, B, y,
                                    shift, stream)
                torch.cuda.synchronize()
                graphs = []
                for i in range(copies):
                    gr = torch.cuda.CUDAGraph()
                    with torch.cuda.graph(gr, stream=stream):
                        sg.colored_gemv(ctx, W[i], sg.BF16, M, K, x, sg.BF16, B, y, shift,
                                        stream)
                    graphs.append(gr)
                for i in range(20):
                    graphs[i % copies].replay()
                timer.reserve(4 * launches)
                block = 100
                for b0 in range(0, launches, block):
                    for i in range(b0, min(b0 + block, launches)):
                        e0 = timer.start()
                        sg.colored_gemv(ctx, W[i % copies], sg.BF16, M, K, x, sg.BF16, B, y,
                                        shift, stream)
                        timer.stop(e0, tag_d)
                    for i in range(b0, min(b0 + block, launches)):
                        e0 = timer.start()
                        graphs[i % copies].replay()
                        timer.stop(e0, tag_g)
                torch.cuda.synchronize()
                sg.colored_gemv(ctx, W[1], sg.BF16, M, K, x, sg.BF16, B, y, shift, stream)
                torch.cuda.synchronize()
                direct = y[:B * M].clone()
                y.fill_(-1.0)
                graphs[1].replay()
                torch.cuda.synchronize()
                same = bool(torch.equal(direct.view(torch.int32), y[:B * M].view(torch.int32)))
                sg.set_cu_mask(ctx, stream, None)
                torch.cuda.synchronize()
            del graphs
            dd, dg = timer.durations_ms(tag_d), timer.durations_ms(tag_g)
            r = {"M": M, "K": K, "batch": B, "cus": ncu, "launches": launches,
                 "direct_launch_p50_us": round(pctl(dd, 50) * 1e3, 2),
                 "direct_launch_p99_us": round(pctl(dd, 99) * 1e3, 2),
                 "graph_launch_p50_us": round(pctl(dg, 50) * 1e3, 2),
                 "graph_launch_p99_us": round(pctl(dg, 99) * 1e3, 2),
                 "graph_matches_direct": same, "device_flags": ctx.device_error()}
            log(f"gemv {M}x{K} B={B} cus={ncu}: launch p50/p99 direct {r['direct_launch_p50_us']}"
                f" / {r['direct_launch_p99_us']} us, graph replay {r['graph_launch_p50_us']} / "
                f"{r['graph_launch_p99_us']} us (same bits: {same})")
            return r

        for B in (1, 2, 4, 8):
            for ncu in (64, 128, 192, 256):
                if ncu > n_cus:
                    continue
                point(W, B, ncu, "xcds", "coloured")
                if ncu < n_cus and B in (1, 8):
                    point(W, B, ncu, "spread", "coloured")
        # B = 1 output of the last launch, for the CPU baseline's oracle check
        sg.colored_gemv(ctx, W[0], sg.BF16, M, K, x, sg.BF16, 1, y, shift, stream)
        torch.cuda.synchronize()
        checks.setdefault("gemv", {})[(M, K)] = (
            w.view(torch.int16).cpu().numpy().view(np.uint16),
            x[:K].view(torch.int16).cpu().numpy().view(np.uint16), y[:M].cpu().numpy())
        # fewer rotated copies: with one or four copies (90 / 360 MB) part of W
        # can stay in the 256 MiB MALL between launches; eight (721 MB) cannot
        for rot in (1, 4):
            for B in (1, 8):
                point(W, B, n_cus, "xcds", "coloured", rotate=rot)
        # the same product through the ROCm libraries (torch.nn.functional.linear
        # in bf16, fp32 accumulation inside the library): a reference time
        lib_ref[f"{M}x{K}"] = library_linear_us(torch, w, x, M, K, stream, timer)
        if M == 4096:
            # the same weights in contiguous buffers (identity tables): the
            # cost of the page-table indirection
            Wc = [torch.empty(pages * P, dtype=torch.uint8, device="cuda:0") for _ in range(copies)]
            WC = [sg.paged(t, ident, pages) for t in Wc]
            torch.cuda.synchronize()
            for Wi in WC:
                sg.bimodal_relayout(ctx, Wi, sg.paged(w, ident, pages), w_bytes, shift, stream)
            torch.cuda.synchronize()
            for B in (1, 8):
                t_plain = point(WC, B, n_cus, "xcds", "contiguous")
                t_col = [p["p50_us"] for p in out if p["M"] == M and p["batch"] == B and
                         p["cus"] == n_cus and p["placement"] == "xcds" and
                         p["layout"] == "coloured" and p["rotated_copies"] == copies][0]
                indirection[f"b{B}_pct"] = round(100 * (t_col / t_plain - 1), 2)
            del Wc, WC
            # the LS layer of the co-located pair (batch 1 on 192 CUs) as a
            # HIP graph replay (recorded as an error, not fatal, if capture
            # fails on this stack)
            try:
                graph_ls = graph_point(1, n_cus * 3 // 4)
            except Exception as e:  # noqa: BLE001
                torch.cuda.synchronize()
                sg.set_cu_mask(ctx, stream, None)
                graph_ls = {"error": f"{type(e).__name__}: {e}"}
        del raw, W
        torch.cuda.empty_cache()
    return {"what": "bf16 W on 48/64 colours in 2 MiB pages, bf16 x, fp32 y; "
                    f"{copies} rotated weight copies; {launches} launches per point; layout "
                    "contiguous: the same weights in plain buffers with identity tables",
            "placement": "xcds: the first n logical CUs (whole XCDs, n/32 of them); spread: n/8 "
                         "CUs in each of the 8 XCDs",
            "bytes": "M*K*2 + B*K*2 + B*M*4",
            "indirection": {"what": "4096x11008 on 256 CUs: coloured pages (8 copies) against "
                                    "contiguous weights with identity tables, p50 difference",
                            **indirection},
            "library_reference": lib_ref,
            "graph_ls": graph_ls,
            "timing": "p50/p99_us and GBps: kernel spans from the device time log (first "
                      "workgroup start to last workgroup end); launch_p50/p99_us: host events "
                      "around each call in a separate loop without the log, including launch "
                      "overhead",
            "points": out}


def library_linear_us(torch, w, x, M, K, stream, timer, reps=200):
    """p50 time (host events around each call) of torch.nn.functional.linear
    on contiguous bf16 weights [M x K] at batch 1 and 8: the ROCm library
    GEMV/GEMM on the same shapes, all CUs, no colouring.  A reference, not
    part of the path."""
    import torch.nn.functional as F
    res = {}
    W2 = w[:M * K].view(M, K)
    for B in (1, 8):
        X = x[:B * K].view(B, K).contiguous()
        tag = ("library", M, B)
        with torch.cuda.stream(stream):
            for _ in range(10):
                F.linear(X, W2)
            timer.reserve(2 * reps)
            for _ in range(reps):
                e0 = timer.start()
                F.linear(X, W2)
                timer.stop(e0, tag)
        torch.cuda.synchronize()
        res[f"b{B}"] = round(pctl(timer.durations_ms(tag), 50) * 1e3, 2)
    log(f"library reference F.linear {M}x{K}: {res} us (with launch)")
    return res


def spread_cus(n_cus, ncu, n_xcds=8):
    """ncu logical CUs spread evenly over all XCDs (logical CUs are numbered
    XCD by XCD, n_cus / n_xcds in each)."""
    per = n_cus // n_xcds
    return [x * per + i for x in range(n_xcds) for i in range(ncu // n_xcds)]


def bench_xcd(torch, sg, ctx, stream, reps=20):
    """Streaming bandwidth against the XCDs a CU mask reaches: the triad over
    three contiguous 1 GiB fp32 arrays (identity page tables, 64 KiB pages)
    on whole XCDs (the first 32k logical CUs) and on the same CU count
    spread over all eight XCDs."""
    shift = 16
    n = 1 << 28
    pages = (n * 4) >> shift
    n_cus = ctx.num_cus
    per_xcd = n_cus // 8
    g = torch.Generator(device="cuda:0")
    g.manual_seed(11)
    a = torch.empty(n, dtype=torch.float32, device="cuda:0")
    b = torch.rand(n, generator=g, device="cuda:0") * 2 - 1
    c = torch.rand(n, generator=g, device="cuda:0") * 2 - 1
    ident = torch.arange(pages, dtype=torch.int32, device="cuda:0")
    A, B, C = (sg.paged(t, ident, pages) for t in (a, b, c))
    torch.cuda.synchronize()
    out = []
    for k in range(1, 9):
        for place in ("xcds", "spread") if k < 8 else ("xcds",):
            ncu = k * per_xcd
            cus = range(ncu) if place == "xcds" else spread_cus(n_cus, ncu)
            with torch.cuda.stream(stream):
                sg.set_cu_mask(ctx, stream, cus)
                for _ in range(3):
                    sg.colored_stream(ctx, A, B, C, 3.0, n, shift, stream)
                dev = DevTimes(torch, ctx, stream, reps)
                for _ in range(reps):
                    sg.colored_stream(ctx, A, B, C, 3.0, n, shift, stream)
                spans = dev.close_us()
                sg.set_cu_mask(ctx, stream, None)
            med = pctl(list(spans), 50)
            gbs = 12 * n / (med * 1e-6) / 1e9
            xcds = k if place == "xcds" else 8
            out.append({"cus": ncu, "xcds": xcds, "placement": place,
                        "p50_ms": round(med / 1e3, 4), "GBps": round(gbs, 1),
                        "GBps_per_xcd": round(gbs / xcds, 1),
                        "device_flags": ctx.device_error()})
            log(f"xcd triad {ncu} CUs on {xcds} XCDs: {med / 1e3:.3f} ms, {gbs:.0f} GB/s")
    del a, b, c
    torch.cuda.empty_cache()
    return {"what": "triad a=b+3c, three contiguous 1 GiB fp32 arrays, 64 KiB pages, by CU mask; "
                    f"{reps} launches per point, kernel spans from the device time log",
            "points": out}


def corun_operands(torch, sg, synth, ctx):
    """Operands of the co-located pair (LS GEMV and BE triad), all from one pool under one hash
    (6 masks on address bits 21..40, so every 2 MiB region has one colour):
    the LS GEMV's bf16 W (4096 x 11008) in 2 MiB pages on colours 0..47
    (8 rotated copies), the BE triad's three 2 GiB fp32 arrays in 64 KiB
    pages on colours 48..63 -- the two page sets share no region -- and,
    for the uncoloured control, the same tensors in plain buffers with
    identity tables."""
    dev = "cuda:0"
    M, K = 4096, 11008
    g = torch.Generator(device=dev)
    g.manual_seed(11)
    wshift, shift = 21, 16
    masks = synth.xor_masks(6, seed=1, min_bit=wshift)
    WP = 1 << wshift
    w_bytes = M * K * 2
    wpages = -(-w_bytes // WP)
    copies = 8
    n = 1 << 29
    pages = (n * 4) >> shift
    region = 1 << (wshift - shift)
    pool_regions = int(3 * pages / region * 4 * 1.1) + copies * wpages * 2 + 64
    raw, base = aligned_pool(torch, pool_regions, wshift)
    w_pt = torch.empty(copies * wpages, dtype=torch.int32, device=dev)
    sg.colour_alloc_pagetable(ctx, masks, base, wshift, pool_regions, range(48), copies * wpages, w_pt)
    be_pt = torch.empty(3 * pages, dtype=torch.int32, device=dev)
    sg.colour_alloc_pagetable(ctx, masks, base, shift, pool_regions * region, range(48, 64),
                              3 * pages, be_pt)
    overlap = len(set(w_pt.cpu().tolist()) & set((be_pt.cpu() // region).tolist()))
    # ---- LS operands
    w_lin = (torch.randn(M * K, generator=g, device=dev) * 0.02).to(torch.bfloat16)
    w_ident = torch.arange(wpages, dtype=torch.int32, device=dev)
    W_col = []
    for i in range(copies):
        Wi = sg.paged(base, w_pt[i * wpages:(i + 1) * wpages], pool_regions)
        sg.bimodal_relayout(ctx, Wi, sg.paged(w_lin, w_ident, wpages), w_bytes, wshift)
        W_col.append(Wi)
    w_plain = [torch.empty(wpages * WP // 2, dtype=torch.bfloat16, device=dev) for _ in range(copies)]
    W_plain = []
    for i in range(copies):
        Wi = sg.paged(w_plain[i], w_ident, wpages)
        sg.bimodal_relayout(ctx, Wi, sg.paged(w_lin, w_ident, wpages), w_bytes, wshift)
        W_plain.append(Wi)
    x = torch.randn(K, generator=g, device=dev).to(torch.bfloat16)
    y = torch.empty(M, dtype=torch.float32, device=dev)
    # ---- BE operands
    ident = torch.arange(pages, dtype=torch.int32, device=dev)
    lin = [torch.empty(n, dtype=torch.float32, device=dev) for _ in range(3)]
    lin[1].uniform_(-1, 1, generator=g)
    lin[2].uniform_(-1, 1, generator=g)
    T_col = [sg.paged(base, be_pt[i * pages:(i + 1) * pages], pool_regions * region)
             for i in range(3)]
    for i in (1, 2):
        sg.bimodal_relayout(ctx, T_col[i], sg.paged(lin[i], ident, pages), n * 4, shift)
    T_plain = [sg.paged(lin[i], ident, pages) for i in range(3)]
    torch.cuda.synchronize()
    log(f"corun operands: one pool of {pool_regions} x 2 MiB, LS/BE regions shared: {overlap}")
    return {"M": M, "K": K, "wshift": wshift, "copies": copies, "W_col": W_col,
            "W_plain": W_plain, "x": x, "y": y, "shift": shift, "n": n, "T_col": T_col,
            "T_plain": T_plain, "masks": [hex(m) for m in masks], "shared_regions": overlap,
            "_keep": (raw, w_plain, lin, w_pt, be_pt, w_ident, ident)}


def bench_corun(torch, sg, synth, ctx, ls_launches, ops):
    """Co-located pair: LS GEMV (bf16 4096x11008, batch 1) on colours 0..47 and
    CUs 0..191, BE triad (three 2 GiB fp32 arrays, 64 KiB pages) on colours
    48..63 and CUs 192..255, against the same two kernels uncoloured (identity
    page tables over contiguous buffers) with the same CU split (the paper's
    control group) and uncoloured with no CU split.  LS runs a closed loop of
    ``ls_launches`` kernels; BE streams triads for the whole LS window."""
    import numpy as np
    n_cus = ctx.num_cus
    ls_cus, be_cus = list(range(n_cus * 3 // 4)), list(range(n_cus * 3 // 4, n_cus))
    M, K, wshift, copies = ops["M"], ops["K"], ops["wshift"], ops["copies"]
    W_col, W_plain, x, y = ops["W_col"], ops["W_plain"], ops["x"], ops["y"]
    shift, n, T_col, T_plain = ops["shift"], ops["n"], ops["T_col"], ops["T_plain"]
    log(f"corun: LS gemv {M}x{K} on {len(ls_cus)} CUs, BE triad 3x2 GiB on {len(be_cus)} CUs")

    s_ls = torch.cuda.Stream(device=0)
    s_be = torch.cuda.Stream(device=0)

    # The long-running BE triad must leave workgroup slots free on its CUs,
    # so that the LS kernels' workgroups that the hardware sends to BE's XCDs
    # can be placed (and leave) without waiting for a BE kernel to end.  The
    # triad already runs one workgroup per CU; the cap states the bound.
    be_cap = 3

    def run(Ws, Ts, ls_mask, be_mask, with_be, ls_cap=0):
        sg.set_cu_mask(ctx, s_ls, ls_mask)
        sg.set_cu_mask(ctx, s_be, be_mask)
        sg.set_stream_occupancy(ctx, s_be, be_cap)
        sg.set_stream_occupancy(ctx, s_ls, ls_cap)
        t_ls = Timer(torch, s_ls)
        t_be = Timer(torch, s_be)
        for i in range(10):
            sg.colored_gemv(ctx, Ws[i % copies], sg.BF16, M, K, x, sg.BF16, 1, y, wshift, s_ls)
        sg.colored_stream(ctx, Ts[0], Ts[1], Ts[2], 3.0, n, shift, s_be)
        torch.cuda.synchronize()
        pending = []          # completion events of queued BE launches

        def top_up():
            while pending and pending[0].query():
                pending.pop(0)
            while len(pending) < 2:
                e0 = t_be.start()
                sg.colored_stream(ctx, Ts[0], Ts[1], Ts[2], 3.0, n, shift, s_be)
                t_be.stop(e0)
                pending.append(t_be.pairs[-1][2])

        dev_ls = DevTimes(torch, ctx, s_ls, ls_launches)
        dev_be = DevTimes(torch, ctx, s_be, 4096) if with_be else None
        if with_be:
            top_up()
        for i in range(ls_launches):
            e0 = t_ls.start()
            sg.colored_gemv(ctx, Ws[i % copies], sg.BF16, M, K, x, sg.BF16, 1, y, wshift, s_ls)
            t_ls.stop(e0)
            if with_be and i % 25 == 0:
                top_up()
        if with_be:
            last_ls = t_ls.pairs[-1][2]
            while not last_ls.query():
                top_up()
                time.sleep(0.0002)
        torch.cuda.synchronize()
        out = {}
        d = dev_ls.close_us()
        out["ls_p50_us"] = round(float(np.percentile(d, 50)), 2)
        out["ls_p99_us"] = round(float(np.percentile(d, 99)), 2)
        hd = np.array(t_ls.durations_ms()) * 1e3
        out["ls_launch_p50_us"] = round(float(np.percentile(hd, 50)), 2)
        out["ls_launch_p99_us"] = round(float(np.percentile(hd, 99)), 2)
        if with_be:
            nb = len(t_be.pairs)
            bd = dev_be.close_us(nb)
            out["be_GBps"] = round(12 * n / (float(np.median(bd)) * 1e-6) / 1e9, 1)
            out["be_launches"] = nb
        sg.set_cu_mask(ctx, s_ls, None)
        sg.set_cu_mask(ctx, s_be, None)
        sg.set_stream_occupancy(ctx, s_be, 0)
        sg.set_stream_occupancy(ctx, s_ls, 0)
        return out

    res = {"what": "LS bf16 GEMV 4096x11008 batch 1 (closed loop) + BE fp32 triad 3x2 GiB",
           "ls_launches": ls_launches, "be_workgroups_per_cu_cap": be_cap,
           "masks": ops["masks"], "ls_be_shared_2MiB_regions": ops["shared_regions"],
           "timing": "ls_p50/p99_us and be_GBps from the device time log (kernel spans); "
                     "ls_launch_p50/p99_us from host events around each LS call"}
    res["isolated_ls_coloured_masked"] = run(W_col, T_col, ls_cus, be_cus, with_be=False)
    res["corun_coloured_masked"] = run(W_col, T_col, ls_cus, be_cus, with_be=True)
    res["corun_uncoloured_masked"] = run(W_plain, T_plain, ls_cus, be_cus, with_be=True)
    res["corun_uncoloured_unmasked"] = run(W_plain, T_plain, None, None, with_be=True)
    res["corun_coloured_masked_ls_cap3"] = run(W_col, T_col, ls_cus, be_cus, with_be=True,
                                               ls_cap=3)
    for k in ("isolated_ls_coloured_masked", "corun_coloured_masked", "corun_uncoloured_masked",
              "corun_uncoloured_unmasked", "corun_coloured_masked_ls_cap3"):
        log(f"corun {k}: {res[k]}")
    return res


def bench_preempt(torch, sg, synth, ctx, ops, trials):
    """Tidal handover (paper section 7.1) at the co-located pair's sizes.  The BE triad
    (3 x 2 GiB, colours 48..63) starts on all CUs as a preemptible launch.
    After a random delay the LS side raises the eviction flag in its own
    stream order (a device store stamped with the device clock), takes the
    CUs of the sliding-window policy and launches its GEMV (bf16 4096x11008,
    colours 0..47); the BE stream clears the flag after its evicted kernel
    and resumes on the CUs left.  Everything is enqueued without host waits.
    Reported from the device time log: eviction latency (flag store -> end
    of the BE kernel), LS latency from the flag store to the GEMV's end and
    the GEMV's own span, the BE makespan (first start -> resumed end)
    against an uninterrupted triad on all CUs; and the cost of the
    preemptible triad kernel when nothing evicts it."""
    import numpy as np
    dev = "cuda:0"
    khz = ctx.wallclock_khz
    n_cus = ctx.num_cus
    M, K, wshift, copies = ops["M"], ops["K"], ops["wshift"], ops["copies"]
    Ws, x, y = ops["W_col"], ops["x"], ops["y"]
    shift, n, T = ops["shift"], ops["n"], ops["T_col"]
    ls_need = [n_cus * 3 // 4]
    ls_cus, be_cus = sg.tidal_masks(n_cus, ls_need, window=4, granule=32)
    s_ls, s_be = torch.cuda.Stream(device=0), torch.cuda.Stream(device=0)
    flag = torch.zeros(1, dtype=torch.int32, device=dev)
    stamps = torch.zeros(trials, dtype=torch.int64, device=dev)
    us = lambda t: t * 1e3 / khz

    def triad(stream):
        sg.colored_stream(ctx, T[0], T[1], T[2], 3.0, n, shift, stream)

    # the cost of the preemptible kernel (flag never raised) against the
    # plain one, interleaved on all CUs
    spans = {False: [], True: []}
    for rep in range(6):
        for pre in (False, True):
            sg.set_eviction_flag(ctx, s_be, flag if pre else None)
            d = DevTimes(torch, ctx, s_be, 1)
            triad(s_be)
            spans[pre].append(float(d.close_us()[0]))
    plain_us, pre_us = np.median(spans[False][1:]), np.median(spans[True][1:])
    log(f"preempt: triad plain {plain_us:.1f} us, preemptible {pre_us:.1f} us")

    # delay calibration of torch's sleep kernel (cycles per microsecond)
    with torch.cuda.stream(s_ls):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(s_ls)
        torch.cuda._sleep(1000000)
        e1.record(s_ls)
    torch.cuda.synchronize()
    cyc_per_us = 1000000 / max(e0.elapsed_time(e1) * 1e3, 1.0)

    sg.set_eviction_flag(ctx, s_be, flag)
    sg.set_stream_occupancy(ctx, s_be, 3)
    for i in range(3):        # warm both kernels on their masks
        sg.colored_gemv(ctx, Ws[i % copies], sg.BF16, M, K, x, sg.BF16, 1, y, wshift, s_ls)
    torch.cuda.synchronize()
    rng = np.random.default_rng(3)
    dev_be = DevTimes(torch, ctx, s_be, 2 * trials)
    dev_ls = DevTimes(torch, ctx, s_ls, trials)
    for i in range(trials):
        flag.zero_()
        torch.cuda.synchronize()
        sg.set_cu_mask(ctx, s_be, None)
        triad(s_be)
        with torch.cuda.stream(s_ls):
            torch.cuda._sleep(int(rng.uniform(0.1, 0.8) * plain_us * cyc_per_us))
        sg.signal_flag(ctx, s_ls, flag, 1, stamps[i:i + 1])
        sg.set_cu_mask(ctx, s_ls, ls_cus)
        sg.colored_gemv(ctx, Ws[i % copies], sg.BF16, M, K, x, sg.BF16, 1, y, wshift, s_ls)
        sg.signal_flag(ctx, s_be, flag, 0)
        sg.set_cu_mask(ctx, s_be, be_cus)
        sg.resume(ctx, s_be)
        torch.cuda.synchronize()
    tb = dev_be.close_ticks(2 * trials).reshape(trials, 2, 2)
    tl = dev_ls.close_ticks(trials)
    sig = stamps.cpu().numpy()
    left = sg.suspended(ctx, s_be)
    sg.set_eviction_flag(ctx, s_be, None)
    sg.set_cu_mask(ctx, s_be, None)
    sg.set_cu_mask(ctx, s_ls, None)
    sg.set_stream_occupancy(ctx, s_be, 0)
    first_end, first_start, resume_end = tb[:, 0, 1], tb[:, 0, 0], tb[:, 1, 1]
    hit = first_end > sig           # the flag landed while the BE kernel ran
    evict = us(first_end - sig)[hit]
    ls_from_flag = us(tl[:, 1] - sig)[hit]
    ls_span = us(tl[:, 1] - tl[:, 0])[hit]
    makespan = us(resume_end - first_start)[hit]

    def p(a, q):
        return round(float(np.percentile(a, q)), 2) if len(a) else None

    res = {"what": "BE fp32 triad 3x2 GiB (colours 48..63) evicted from all CUs by an LS bf16 "
                   "GEMV 4096x11008 batch 1 (colours 0..47); sliding-window split "
                   f"{len(ls_cus)} LS / {len(be_cus)} BE CUs",
           "trials": trials, "evicted_trials": int(hit.sum()), "left_after_last_trial": int(left),
           "eviction_latency_p50_us": p(evict, 50), "eviction_latency_p99_us": p(evict, 99),
           "ls_from_flag_p50_us": p(ls_from_flag, 50), "ls_from_flag_p99_us": p(ls_from_flag, 99),
           "ls_gemv_span_p50_us": p(ls_span, 50), "ls_gemv_span_p99_us": p(ls_span, 99),
           "be_makespan_p50_us": p(makespan, 50),
           "be_uninterrupted_us": round(float(plain_us), 2),
           "triad_plain_us": round(float(plain_us), 2),
           "triad_preemptible_us": round(float(pre_us), 2),
           "preemptible_overhead_pct": round(100 * (pre_us / plain_us - 1), 2),
           "timing": "device time log and device clock stamps of the flag store; p50/p99 over "
                     "the trials whose flag landed while the BE kernel ran"}
    log(f"preempt: {res}")
    return res


def bench_bimodal(torch, sg, synth, ctx, stream, reps=20, launches=100):
    """Bimodal LS tensors (paper section 7.2) at the LS layer shapes: both bf16
    matrices (4096x11008, 11008x4096; 2 MiB pages) registered as
    latency-sensitive tensors with an all-channel form and a form on colours
    0..47.  Reported: the time of a state change (the runtime relays both
    matrices between the forms; device time of the change on one stream)
    and the batch-1 GEMV latency on the form the runtime hands out in each
    state."""
    import numpy as np
    dev = "cuda:0"
    shift = 21
    P = 1 << shift
    masks = synth.xor_masks(6, seed=1, min_bit=shift)
    g = torch.Generator(device=dev)
    g.manual_seed(13)
    shapes = [(4096, 11008), (11008, 4096)]
    keep = []
    bm = sg.Bimodal(ctx)
    ids = []
    total = 0
    for (M, K) in shapes:
        nbytes = M * K * 2
        pages = -(-nbytes // P)
        w = (torch.randn(pages * P // 2, generator=g, device=dev) * 0.02).to(torch.bfloat16)
        ident = torch.arange(pages, dtype=torch.int32, device=dev)
        pool_pages = int(pages * 64 / 48 * 1.2) + 8
        raw, base = aligned_pool(torch, pool_pages, shift)
        pt = torch.empty(pages, dtype=torch.int32, device=dev)
        sg.colour_alloc_pagetable(ctx, masks, base, shift, pool_pages, range(48), pages, pt)
        ids.append(bm.register(sg.BM_LS_TENSOR, sg.paged(w, ident, pages),
                               sg.paged(base, pt, pool_pages), nbytes, shift, stream))
        keep += [w, ident, raw, pt]
        total += nbytes
    x = torch.randn(11008, generator=g, device=dev).to(torch.bfloat16)
    y = torch.empty(11008, dtype=torch.float32, device=dev)
    torch.cuda.synchronize()
    trans = {sg.BM_COLOCATED: [], sg.BM_MONOPOLY: []}
    for _ in range(reps):
        for st in (sg.BM_COLOCATED, sg.BM_MONOPOLY):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            bm.set_state(st, stream)
            e1.record(stream)
            torch.cuda.synchronize()
            trans[st].append(e0.elapsed_time(e1))
    out = {"what": "two bf16 LS matrices (4096x11008, 11008x4096) as LS tensors: all-channel form vs colours 0..47 "
                   "(2 MiB pages)", "bytes_moved_per_change": total}
    for st, name in ((sg.BM_COLOCATED, "to_colocated"), (sg.BM_MONOPOLY, "to_monopoly")):
        ms = float(np.median(trans[st]))
        out[name + "_ms"] = round(ms, 4)
        out[name + "_GBps"] = round(2 * total / (ms * 1e-3) / 1e9, 1)
    for st, name in ((sg.BM_MONOPOLY, "monopoly"), (sg.BM_COLOCATED, "colocated")):
        bm.set_state(st, stream)
        for (M, K), tid in zip(shapes, ids):
            desc, form = bm.input(tid)
            with torch.cuda.stream(stream):
                for _ in range(10):
                    sg.colored_gemv(ctx, desc, sg.BF16, M, K, x, sg.BF16, 1, y, shift, stream)
                d = DevTimes(torch, ctx, stream, launches)
                for _ in range(launches):
                    sg.colored_gemv(ctx, desc, sg.BF16, M, K, x, sg.BF16, 1, y, shift, stream)
                spans = d.close_us()
            out[f"gemv_{M}x{K}_{name}_p50_us"] = round(float(np.median(spans)), 2)
            out[f"gemv_{M}x{K}_{name}_form"] = "all" if form == sg.BM_ALL else "colours 0..47"
    bm.set_state(sg.BM_MONOPOLY, stream)
    torch.cuda.synchronize()
    bm.close()
    log(f"bimodal: {out}")
    del keep
    torch.cuda.empty_cache()
    return out


def bench_sectors(torch, sg, synth, ctx, stream, timer, reps=20):
    """Colouring granularity (paper section 6: 1-2 KiB sectors; section 5.3:
    a colour table for hashes that are not XOR-linear).  The streaming triad (three
    1 GiB fp32 arrays, colours 0..15 of 64) with 1, 2, 4 and 64 KiB pages:
    the cost of finer page-table indirection.  Then classify and the page-
    table build through a random colour table of 2^26 1 KiB partitions
    (64 GiB of address space)."""
    import numpy as np
    dev = "cuda:0"
    n = 1 << 28
    out = {"what": "triad 3x1 GiB fp32 on colours 0..15 of 64 by page size (1, 2, 4, 64 KiB "
                   "and 2 MiB), and on contiguous arrays through identity and randomly permuted "
                   "tables of the same page size; colour-table classify and page-table build"}
    g = torch.Generator(device=dev)
    g.manual_seed(21)
    b_lin = torch.empty(n, dtype=torch.float32, device=dev).uniform_(-1, 1, generator=g)
    c_lin = torch.empty(n, dtype=torch.float32, device=dev).uniform_(-1, 1, generator=g)
    for shift in (10, 11, 12, 16, 21):
        P = 1 << shift
        pages = (n * 4) >> shift
        masks = synth.xor_masks(6, seed=1, min_bit=shift)
        pool_pages = int(3 * pages * 4 * 1.08) + 64
        raw, base = aligned_pool(torch, pool_pages, shift)
        pt = torch.empty(3 * pages, dtype=torch.int32, device=dev)
        e0 = time.perf_counter()
        sg.colour_alloc_pagetable(ctx, masks, base, shift, pool_pages, range(16), 3 * pages, pt)
        pt_ms = (time.perf_counter() - e0) * 1e3
        A, B, C = (sg.paged(base, pt[i * pages:(i + 1) * pages], pool_pages) for i in range(3))
        ident = torch.arange(pages, dtype=torch.int32, device=dev)
        sg.bimodal_relayout(ctx, B, sg.paged(b_lin, ident, pages), n * 4, shift)
        sg.bimodal_relayout(ctx, C, sg.paged(c_lin, ident, pages), n * 4, shift)
        tag = ("sectors", shift)
        with torch.cuda.stream(stream):
            for _ in range(3):
                sg.colored_stream(ctx, A, B, C, 3.0, n, shift, stream)
            for _ in range(reps):
                e = timer.start()
                sg.colored_stream(ctx, A, B, C, 3.0, n, shift, stream)
                timer.stop(e, tag)
        torch.cuda.synchronize()
        ms = pctl(timer.durations_ms(tag), 50)
        out[f"triad_{P >> 10}KiB_GBps"] = round(12 * n / (ms * 1e-3) / 1e9, 1)
        out[f"triad_{P >> 10}KiB_ms"] = round(ms, 4)
        out[f"pagetable_{P >> 10}KiB_ms"] = round(pt_ms, 3)
        log(f"sectors: {P >> 10} KiB pages: triad {ms:.4f} ms "
            f"({12 * n / (ms * 1e-3) / 1e9:.0f} GB/s), page table {pt_ms:.2f} ms")
        # the same page size over contiguous arrays: identity tables (the
        # kernel's own cost of the indirection) and the pages of each array in
        # a random order (the cost of scattered placement)
        perm = torch.randperm(pages, device=dev, generator=g).to(torch.int32)
        a_lin = torch.empty(n, dtype=torch.float32, device=dev)
        torch.cuda.synchronize()
        for name, table in (("identity", ident), ("permuted", perm)):
            X = [sg.paged(t, table, pages) for t in (a_lin, b_lin, c_lin)]
            tag = ("sectors", shift, name)
            with torch.cuda.stream(stream):
                for _ in range(3):
                    sg.colored_stream(ctx, *X, 3.0, n, shift, stream)
                for _ in range(reps):
                    e = timer.start()
                    sg.colored_stream(ctx, *X, 3.0, n, shift, stream)
                    timer.stop(e, tag)
            torch.cuda.synchronize()
            m2 = pctl(timer.durations_ms(tag), 50)
            out[f"triad_{P >> 10}KiB_{name}_GBps"] = round(12 * n / (m2 * 1e-3) / 1e9, 1)
            log(f"sectors: {P >> 10} KiB pages, contiguous arrays, {name} tables: "
                f"{12 * n / (m2 * 1e-3) / 1e9:.0f} GB/s")
        del raw, pt, A, B, C, ident, perm, a_lin
        torch.cuda.empty_cache()
    del b_lin, c_lin
    # a random table of 2^26 1 KiB partitions
    entries, origin = 1 << 26, 1 << 36
    lut = torch.randint(0, 64, (entries,), dtype=torch.uint8, device=dev, generator=g)
    t = sg.colour_table(lut, origin, 10)
    na = 1 << 26
    addrs = (origin + torch.randint(0, entries << 10, (na,), device=dev, generator=g)).to(torch.int64)
    cols = torch.empty(na, dtype=torch.uint8, device=dev)
    hist = torch.empty(256, dtype=torch.int64, device=dev)
    tag = ("sectors", "classify_table")
    with torch.cuda.stream(stream):
        for _ in range(3):
            sg.colour_classify_table(ctx, t, addrs, cols, hist, stream)
        for _ in range(reps):
            e = timer.start()
            sg.colour_classify_table(ctx, t, addrs, cols, hist, stream)
            timer.stop(e, tag)
    torch.cuda.synchronize()
    ms = pctl(timer.durations_ms(tag), 50)
    out["classify_table_2e26_us"] = round(ms * 1e3, 2)
    out["classify_table_addrs_per_s"] = round(na / (ms * 1e-3), 0)
    pool_pages = entries                          # 1 KiB pages over the whole table
    pt = torch.empty(1 << 20, dtype=torch.int32, device=dev)
    times = []
    for _ in range(5):
        e0 = time.perf_counter()
        sg.colour_alloc_pagetable_table(ctx, t, origin, 10, pool_pages, range(16), 1 << 20, pt,
                                        stream)
        times.append((time.perf_counter() - e0) * 1e3)
    out["pagetable_table_1KiB_ms"] = round(float(np.median(times)), 3)
    out["pagetable_table_pool_pages"] = pool_pages
    log(f"sectors: {out}")
    del lut, addrs, cols, pt
    torch.cuda.empty_cache()
    return out


def bench_probe(torch, sg, synth, ctx, stream, timer, reps=10, masks=None):
    """Channel probing by bandwidth (in the spirit of the paper's section 5,
    measured through this library).  A triad over three 256 MiB fp32 arrays
    runs on the pages of a pool where parity(address & M) = 0 (a one-mask
    hash, colour 0).  If the bits of M feed the channel hash, those pages
    use half of the channels and the triad slows towards half speed;
    otherwise it keeps the speed of the unrestricted control (M = bit 47,
    zero over the whole pool, keeps every page: the first pages in order).  Bits below 21 are probed with
    1 KiB pages in a 2 GiB pool: user space sees virtual addresses, which
    agree with physical ones inside 2 MiB fragments.  Bits 16..32 are then
    probed with 64 KiB pages in an 8 GiB pool; above bit 20 the result
    describes where this allocation's fragments landed.  Last, placement at
    64 KiB and 2 MiB granularity: three 1 GiB arrays on the first pages of a
    pool four times their size, on a random quarter of its pages, and on
    colours 0..15 of 64."""
    dev = "cuda:0"
    out = {"what": "triad 3x256 MiB fp32 restricted to parity(addr & M) = 0; GB/s and ratio to "
                   "the control M = bit 47. low_bits: 1 KiB pages, 2 GiB pool; high_bits: 64 KiB "
                   "pages, 8 GiB pool. placement: triad 3x1 GiB on a quarter of a pool",
           "points": [], "high_bits": [], "placement": []}

    def triad_gbs(tag, pt, base, pool_pages, shift, n, pages):
        A, B, C = (sg.paged(base, pt[i * pages:(i + 1) * pages], pool_pages) for i in range(3))
        with torch.cuda.stream(stream):
            for _ in range(2):
                sg.colored_stream(ctx, A, B, C, 3.0, n, shift, stream)
            for _ in range(reps):
                e = timer.start()
                sg.colored_stream(ctx, A, B, C, 3.0, n, shift, stream)
                timer.stop(e, tag)
        torch.cuda.synchronize()
        return 12 * n / (pctl(timer.durations_ms(tag), 50) * 1e-3) / 1e9

    def probe(key, shift, pool_bytes, mask_list):
        n = 1 << 26                       # floats per array (256 MiB)
        pages = (n * 4) >> shift
        pool_pages = pool_bytes >> shift
        raw, base = aligned_pool(torch, pool_bytes >> 21, 21)     # 2 MiB aligned
        pt = torch.empty(3 * pages, dtype=torch.int32, device=dev)
        ref = None
        for m in mask_list:
            sg.colour_alloc_pagetable(ctx, [m], base, shift, pool_pages, [0], 3 * pages, pt)
            gbs = triad_gbs(("probe", key, m), pt, base, pool_pages, shift, n, pages)
            if ref is None:
                ref = gbs
            bits = [b for b in range(48) if (m >> b) & 1]
            out[key].append({"bits": bits, "GBps": round(gbs, 1), "ratio": round(gbs / ref, 3)})
            log(f"probe ({key}): bits {bits}: {gbs:.0f} GB/s ({gbs / ref:.2f} of control)")
        del raw, pt
        torch.cuda.empty_cache()

    if masks is None:
        masks = [1 << 47] + [1 << b for b in range(10, 21)] + \
                [(1 << a) | (1 << b) for a in range(10, 16) for b in range(a + 1, 17)]
    probe("points", 10, 2 << 30, masks)
    probe("high_bits", 16, 8 << 30, [1 << 47] + [1 << b for b in range(16, 33)] +
          [(1 << 21) | (1 << 22), (1 << 21) | (1 << 23), (1 << 22) | (1 << 23)])

    n = 1 << 28
    g = torch.Generator(device=dev)
    g.manual_seed(13)
    for shift in (16, 21):
        pages = (n * 4) >> shift
        pool_pages = 4 * 3 * pages + 64
        raw, base = aligned_pool(torch, pool_pages, shift)
        perm = torch.randperm(pool_pages, device=dev, generator=g)[:3 * pages].to(torch.int32)
        pt = torch.empty(3 * pages, dtype=torch.int32, device=dev)
        sg.colour_alloc_pagetable(ctx, synth.xor_masks(6, seed=1, min_bit=shift), base, shift,
                                  pool_pages, range(16), 3 * pages, pt, stream)
        for name, table in (("first pages", torch.arange(3 * pages, dtype=torch.int32, device=dev)),
                            ("random quarter", perm), ("colours 0..15 of 64", pt)):
            gbs = triad_gbs(("placement", shift, name), table, base, pool_pages, shift, n, pages)
            out["placement"].append({"page_KiB": 1 << (shift - 10), "pages": name,
                                     "GBps": round(gbs, 1)})
            log(f"probe (placement): {1 << (shift - 10)} KiB pages, {name}: {gbs:.0f} GB/s")
        del raw, perm, pt
        torch.cuda.empty_cache()
    return out


def cpu_threads():
    """Host threads for the all-cores oracle runs: the CPUs this process may
    use, at most 16 (one GPU's share of the host cores of an eight-GPU
    node)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def split(n, parts, align=1):
    """[lo, hi) ranges covering 0..n in ``parts`` pieces whose bounds are
    multiples of ``align`` (the last one excepted)."""
    step = -(-n // parts)
    step = -(-step // align) * align
    return [(lo, min(n, lo + step)) for lo in range(0, n, step)]


def run_threads(jobs, threads):
    """Runs the callables in ``jobs`` on ``threads`` host threads (the oracle's
    ctypes calls release the interpreter lock) and returns the wall time."""
    import concurrent.futures as cf
    t0 = time.perf_counter()
    if threads == 1:
        for j in jobs:
            j()
    else:
        with cf.ThreadPoolExecutor(max_workers=threads) as ex:
            for f in [ex.submit(j) for j in jobs]:
                f.result()
    return time.perf_counter() - t0


def cpu_baseline(np, synth, masks, shift, pages, pools_desc, b_host, c_host, fractions,
                 gpu_pages, gpu_checks):
    """The CPU oracle (plain single-threaded C, unchanged) timed on this
    host, on one thread and on ``cpu_threads()`` threads that call the same
    functions over disjoint index ranges.  Bounded samples of the path:
    the headline triad (full arrays, every colour set, one pass each), the
    headline page-table builds (full pools), classify of the first 2^22 of
    the 2^26 classify addresses, the 4 GiB relayout's first 256 MiB (4,096
    pages of 64 KiB) in both directions, and the batch-1 GEMV of both LS
    layers on the benchmark's own weights.  GPU results of the same
    operations are compared with the oracle's on these samples."""
    import oracle
    P = 1 << shift
    epp = P // 4
    n = b_host.size
    T = cpu_threads()
    res = {"threads": T, "ops": {}}
    out_ops = res["ops"]

    def timed(name, make_jobs, units, unit_name, bytes_per_unit=None):
        row = {}
        for t in (1, T):
            jobs = make_jobs(t)
            run_threads(jobs[:1], 1)                           # warm caches and pages once
            secs = run_threads(make_jobs(t), t)
            row[f"threads_{t}_s"] = round(secs, 3)
            row[f"threads_{t}_{unit_name}_per_s"] = round(units / secs, 1)
            if bytes_per_unit:
                row[f"threads_{t}_GBps"] = round(units * bytes_per_unit / secs / 1e9, 3)
        out_ops[name] = row
        log(f"cpu baseline {name}: {row}")
        return row

    # ---- triad: full headline arrays, one pass per colour set.  Each host
    # pool mirrors its GPU pool page for page; it is mapped without huge
    # pages, so that only the pages the tables name are ever committed, and
    # every page of a is written once before the timed passes.
    import mmap
    tri = {1: 0.0, T: 0.0}
    check = None
    for nc in fractions:
        base, pool_pages = pools_desc[nc]
        pt, found = oracle.pagetable(masks, base, shift, pool_pages,
                                     synth.colour_set_bits(range(nc)), 3 * pages)
        assert found >= 3 * pages
        pa, pb, pc = pt[:pages], pt[pages:2 * pages], pt[2 * pages:]
        mm = mmap.mmap(-1, pool_pages * P)
        if hasattr(mmap, "MADV_NOHUGEPAGE"):
            mm.madvise(mmap.MADV_NOHUGEPAGE)
        pool = np.frombuffer(mm, dtype=np.float32)
        view = pool.reshape(pool_pages, epp)
        view[pb.astype(np.int64)] = b_host.reshape(pages, epp)
        view[pc.astype(np.int64)] = c_host.reshape(pages, epp)
        view[pa.astype(np.int64)] = 0.0
        for t in (1, T):
            jobs = [lambda j0=j0, j1=j1: oracle.triad(pool, pa[j0:j1], pool, pb[j0:j1], pool,
                                                      pc[j0:j1], 3.0, (j1 - j0) * epp, shift)
                    for j0, j1 in split(pages, t)]
            tri[t] += run_threads(jobs, t)
        if nc == 8:
            check = all(np.array_equal(view[int(pa[j])].view(np.uint32),
                                       gpu_pages[j].view(np.uint32)) for j in gpu_pages)
        del pool, view
        mm.close()
    elems = n * len(fractions)
    triad = {}
    for t in (1, T):
        triad[f"threads_{t}_s"] = round(tri[t], 3)
        triad[f"threads_{t}_elements_per_s"] = round(elems / tri[t], 1)
        triad[f"threads_{t}_GBps"] = round(12 * elems / tri[t] / 1e9, 3)
    out_ops["triad"] = triad
    log(f"cpu baseline triad: {triad}")
    res["triad_gpu_pages_match_oracle"] = check

    # ---- page-table builds over the headline pools
    def pt_jobs(t):
        jobs = []
        for nc in fractions:
            base, pool_pages = pools_desc[nc]
            words = synth.colour_set_bits(range(nc))
            for i0, i1 in split(pool_pages, t):
                jobs.append(lambda base=base, i0=i0, i1=i1, words=words: oracle.pagetable(
                    masks, base + (i0 << shift), shift, i1 - i0, words, i1 - i0))
        return jobs
    timed("pagetable", pt_jobs, sum(pools_desc[nc][1] for nc in fractions), "pool_pages")

    # ---- classify: the first 2^22 of the 2^26 classify addresses
    na = 1 << 22
    cm = synth.xor_masks(6, seed=1, min_bit=12)
    addrs = synth.page_addresses(1 << 26, seed=0)[:na]
    got = {}

    def cls_jobs(t):
        def one(i0, i1):
            got[i0] = oracle.classify(addrs[i0:i1], cm, with_hist=False)[0]
        return [lambda i0=i0, i1=i1: one(i0, i1) for i0, i1 in split(na, t)]
    timed("classify", cls_jobs, na, "addrs", 9)
    ref_col = np.concatenate([got[k] for k in sorted(got)])
    if "classify_colours" in gpu_checks:
        res["classify_gpu_matches_oracle"] = bool(np.array_equal(
            ref_col, gpu_checks["classify_colours"][:na]))

    # ---- relayout: 256 MiB (4,096 pages of 64 KiB) of the 4 GiB tensor,
    # all colours -> colours 0..15 of 64 and back, on a synthetic pool origin
    rp = 4096
    rpool_pages = rp * 4 + 4096
    rmask = synth.xor_masks(6, seed=1, min_bit=16)
    rpt, found = oracle.pagetable(rmask, 1 << 40, 16, rpool_pages, synth.colour_set_bits(range(16)),
                                  rp)
    assert found >= rp
    src = synth.random_u16(rp * (1 << 15), seed=5)
    rpool = np.zeros(rpool_pages << 16, dtype=np.uint8)
    back = np.zeros_like(src)
    ident = np.arange(rp, dtype=np.uint32)

    def rel_jobs(t):
        jobs = []
        for j0, j1 in split(rp, t):
            jobs.append(lambda j0=j0, j1=j1: oracle.relayout(rpool, rpt[j0:j1], src, ident[j0:j1],
                                                             (j1 - j0) << 16, 16))
            jobs.append(lambda j0=j0, j1=j1: oracle.relayout(back, ident[j0:j1], rpool, rpt[j0:j1],
                                                             (j1 - j0) << 16, 16))
        return jobs
    timed("relayout", rel_jobs, 2 * (rp << 16), "bytes", 2)
    out_ops["relayout"]["pages_per_s_threads_1"] = round(
        2 * rp / out_ops["relayout"]["threads_1_s"], 1)
    res["relayout_round_trip_identity"] = bool(np.array_equal(back, src))
    del rpool, back, src

    # ---- GEMV batch 1 on the benchmark's own LS-layer weights (contiguous copy)
    if "gemv" in gpu_checks:
        for (M, K), (w, x, y_gpu) in gpu_checks["gemv"].items():
            rows_out = {}

            def gemv_jobs(t, M=M, K=K, w=w, x=x):
                def one(m0, m1):
                    pw = np.arange(-(-((m1 - m0) * K * 2) >> 21) + 1, dtype=np.uint32)
                    rows_out[m0] = oracle.gemv(w[m0 * K:m1 * K], pw, oracle.BF16, m1 - m0, K, x,
                                               oracle.BF16, 1, 21)
                return [lambda m0=m0, m1=m1: one(m0, m1) for m0, m1 in split(M, t)]
            timed(f"gemv_{M}x{K}_b1", gemv_jobs, M * K * 2 + K * 2 + M * 4, "bytes", 1)
            ref = np.concatenate([rows_out[k][0] for k in sorted(rows_out)], axis=1)
            absd = np.concatenate([rows_out[k][1] for k in sorted(rows_out)], axis=1)
            err = np.abs(y_gpu.astype(np.float64) - ref[0])
            res[f"gemv_{M}x{K}_gpu_within_bound"] = bool(np.all(err <= 1e-3 * absd[0] + 1e-30))

    res["value"] = triad[f"threads_{T}_GBps"]
    res["unit"] = "GB/s"
    res["cores"] = T
    res["kind"] = "oracle"
    res["sample"] = (f"triad on the full headline arrays (2^28 elements each, colour sets "
                     f"8/16/32/64 of 64, one pass each) on {T} host threads over disjoint page "
                     f"ranges; single-thread and other ops under 'ops'")
    return res


if __name__ == "__main__":
    main()
