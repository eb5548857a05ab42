"""Throughput of reachable-state weighted FST composition on one MI355X.

One step = one fstc_compose call over the whole workload (CSR build of both
inputs, every breadth-first level: join count, product merge or arc-pair
write + merge, visited-table insert, id assignment, result append), inputs
already resident in HBM.  Prints one JSON line.

Default workload: the HMM-like dense-inner-alphabet pair (|Q1| = |Q2| = 1000,
64 inner symbols, 4 (outer symbol, target) slots per state, 256 arcs per
state, seed 0), the configuration the HBM-fraction target is stated on.

The headline step is the library's default (product merge on).  Unless
--no-record-path is given, the same workload is also timed with every source
going through written records (opts.no_product_merge), and that step's
expand + merge kernels and their HBM roofline are reported as "record_path".
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "composed arcs/sec (pre- and post-merge) + HBM GB/s fraction, 1 MI355X"
HBM_PEAK_GBS = 8000.0
FP64_VECTOR_PEAK_TFLOPS = 78.6  # MI355X vector float64
FP64_MFMA_PEAK_TFLOPS = 78.6    # MI355X dense float64 matrix cores (the product merge's sums)
WORKLOAD_NAMES = {
    1: "tiny random pair: |Q|=200, |Sigma|=|Delta|=50, |Gamma|=100, 2,000 arcs each",
    2: "medium sparse pair: |Q|=10,000, 200,000 arcs each, inner Zipf(1.0) over 5,000, outer 2,000",
    3: "lexicon trie pair: 50,000 words (3-12 of 30 chars), |Gamma|=50,000, 1-5 translations Zipf(1.1) over 20,000",
    4: "HMM-like dense inner alphabet: |Q1|=|Q2|=1,000, m=64, 4 (outer, target) slots x 64 inner symbols = 256 arcs/state, |Sigma|=|Delta|=64",
    5: "large power-law pair: |Q|=1,000,000, 20M arcs each, degree ~ d^-2.1 on [4, 10^4], inner Zipf(1.0) over 10^5",
}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", type=int, default=4)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--max-levels", type=int, default=0)
    ap.add_argument("--oracle-levels", type=int, default=0,
                    help="depth cap of the CPU-oracle sample (0: the whole workload)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-reduction", action="store_true",
                    help="compose without merging identical arcs (every joined arc pair is an "
                         "arc; the setting of the paper's Table 2)")
    ap.add_argument("--fused", action="store_true",
                    help="fused expand + merge: tiles merge their composed arcs without "
                         "writing them first (opts.fused_merge)")
    ap.add_argument("--no-product", action="store_true",
                    help="send every source through written records (opts.no_product_merge): "
                         "the paper's count / write / sort-and-reduce path")
    ap.add_argument("--no-record-path", action="store_true",
                    help="skip the second timing with the product merge off")
    ap.add_argument("--paper-pair", default="",
                    help="SIZE-TARGET, e.g. 15k-de: instead of --config, the bigram-LM x "
                         "translation-model pair German -> English -> TARGET at a Table 1 size")
    ap.add_argument("--eps-pair", action="store_true",
                    help="instead of --config, a pair with the empty-string label 0 on every "
                         "tape (2,000 states and 40,000 arcs per side, 5%% empty labels), "
                         "composed under the three-state epsilon filter (fstc_compose_eps)")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="first run a plain device copy of this many MiB three times "
                         "(calibrates the FETCH_SIZE / WRITE_SIZE counters)")
    ap.add_argument("--stream-mib", type=int, default=2048,
                    help="size of each buffer of the STREAM-style probe of achievable HBM "
                         "bandwidth (copy, write-only fill, read-only sum), timed before the "
                         "workload; 0 skips it")
    return ap.parse_args()


def stream_probe(dev, mib: int, reps: int = 5) -> dict:
    """Achievable HBM bandwidth on this GPU with plain device kernels, timed
    with events on the current stream: copy (read + write), fill (write
    only) and a sum reduction (read only) of `mib` MiB buffers."""
    import torch
    n = (mib << 20) // 4
    a = torch.ones(n, dtype=torch.float32, device=dev)
    b = torch.empty_like(a)
    out = {"buffer_bytes": n * 4, "reps": reps}
    acc = torch.zeros((), dtype=torch.float32, device=dev)
    for name, fn, nbytes in (("copy", lambda: b.copy_(a), 2 * n * 4),
                             ("write", lambda: b.fill_(1.5), n * 4),
                             ("read", lambda: torch.sum(a, dim=0, out=acc), n * 4)):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        out[name + "_GBps"] = nbytes / (ms * 1e-3) / 1e9
    del a, b
    torch.cuda.empty_cache()
    return out


def kernel_source_digest(name: str) -> str:
    import hashlib
    path = os.path.join(ROOT, "paper_1805_06383_amd", "csrc", name)
    return hashlib.sha256(open(path, "rb").read()).hexdigest()[:16]


def recorded_traffic(kernel: str, workload: str):
    """HBM bytes per launch of `kernel` from the committed counter summary,
    or None when there is none or the kernel's source changed since."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_traffic.md")
    if not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if line.startswith("- ") and ":" in line:
            k, v = line[2:].split(":", 1)
            fields[k.strip()] = v.strip().strip("`")
    src = fields.get("source")
    if not src or kernel_source_digest(src) != fields.get("source_sha256"):
        return None
    try:
        return float(fields["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def product_flops(st: dict) -> float:
    """Float operations the product merge must do per compose: one float32
    multiply and one float64 add per joined arc pair it merges."""
    return 2.0 * st["total_product_records"]


def algorithmic_bytes(st: dict, R: int, unreduced: bool = False) -> dict:
    """Bytes each of the three tile kernels must move, per compose call.

    write (k_expand): every unmerged record written once (key + float32
      weight) plus one 24-byte match descriptor read per matched
      (source, symbol);
    merge (k_merge_dense) and sort (k_merge_tiles): every record of the tiles
      each merges read once, every merged run it produces written once
      (16 bytes: source, part-rank key, weight).
    """
    rec = st["record_key_bytes"] + 4
    R = R - st["total_product_records"]  # joined pairs written as records
    tile_records = R - st["total_big_records"]
    dense = st["total_dense_records"]
    # without reduction, product-form levels write their joined pairs as
    # result arcs (five 4-byte columns) in the write pass instead of records
    direct_out = st["total_product_records"] * 20 if unreduced else 0
    return {
        "write": R * rec + st["total_matches"] * 24 + direct_out,
        "merge": dense * rec + st["total_dense_runs"] * 16,
        "sort": (tile_records - dense) * rec + st["total_sort_runs"] * 16,
    }


def cpu_baseline(m1, m2, levels: int, reduce: bool = True, eps: bool = False) -> dict:
    import oracle
    if eps:
        r = oracle.compose_eps(m1, m2, 0, max_levels=levels, reduce=reduce)
    else:
        r = oracle.compose(m1, m2, max_levels=levels, reduce=reduce)
    return {
        "value": r.num_premerge / r.seconds,
        "unit": "arcs/s",
        "cores": 1,
        "kind": "oracle",
        "sample": ((f"same workload with the breadth-first search capped at depth {levels}: "
                    if levels else "the whole workload: ") +
                   f"{r.num_premerge} unmerged / {r.num_arcs} output arcs, "
                   f"{r.num_states} states, {r.seconds:.2f} s on 1 of {os.cpu_count()} host "
                   f"cores ({platform.processor() or platform.machine()}); value = unmerged arcs/s"),
        "post_merge_value": r.num_arcs / r.seconds,
    }


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU only (asked for --gpus {args.gpus}); "
              "the composition is not sharded across GPUs", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_1805_06383_amd import fstc
    from paper_1805_06383_amd import workloads as W

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = stream_probe(dev, args.stream_mib) if args.stream_mib else None
    if args.copy_probe_mib:
        nbytes = args.copy_probe_mib << 20
        a_ = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        b_ = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        for _ in range(3):
            b_.copy_(a_)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": nbytes, "launches": 3}), file=sys.stderr, flush=True)
        del a_, b_
    if args.eps_pair:
        h1, h2 = W.eps_pair(11 + args.seed, nq=2000, narcs=40000, nsym=1000, nouter=500,
                            eps_inner=0.05, eps_outer=0.05)
        workload = ("pair with epsilon transitions: 2,000 states and 40,000 arcs per side, "
                    "inner alphabet 1,000, outer 500, label 0 empty on 5% of each tape, "
                    f"three-state epsilon filter, seed {11 + args.seed}")
        traffic_key = None
    elif args.paper_pair:
        size, target = args.paper_pair.split("-")
        h1, h2 = W.paper_pair(size, target, args.seed)
        workload = (f"bigram-LM x translation-model pair, Table 1 size {size}, German -> English "
                    f"-> {target} ({h1.num_states} / {h2.num_states} states, {h1.num_arcs} / "
                    f"{h2.num_arcs} arcs), seed {args.seed}")
        traffic_key = None
    else:
        h1, h2 = W.make_config(args.config, args.seed)
        workload = f"config {args.config}: {WORKLOAD_NAMES[args.config]}, seed {args.seed}"
        traffic_key = "config%d" % args.config
    m1 = fstc.DeviceFST.from_host(h1, dev)
    m2 = fstc.DeviceFST.from_host(h2, dev)
    torch.cuda.synchronize()

    def timed(product: bool):
        """Warmup + K timed steps; returns (seconds, last result, summed stats)."""
        def step():
            if args.eps_pair:
                return fstc.fstc_compose_eps(m1, m2, 0, max_levels=args.max_levels,
                                             reduce=not args.no_reduction, fused=args.fused,
                                             product=product)
            return fstc.fstc_compose(m1, m2, max_levels=args.max_levels,
                                     reduce=not args.no_reduction, fused=args.fused,
                                     product=product)
        for _ in range(args.warmup):
            r = step()
            del r
        torch.cuda.synchronize()
        every = []  # each step's stats, summed after the timed region
        last = None
        t0 = time.perf_counter()
        for _ in range(args.steps):
            last = step()
            every.append(last.stats)
        torch.cuda.synchronize()
        secs = time.perf_counter() - t0
        sums = {}
        for st in every:
            for k, v in st.items():
                sums[k] = sums.get(k, 0) + v
        return secs, last, sums

    def phase_times(product: bool):
        if args.eps_pair:
            return None  # the per-phase events cover one composition of the two
        r = fstc.fstc_compose(m1, m2, max_levels=args.max_levels, reduce=not args.no_reduction,
                              fused=args.fused, product=product, phase_timing=True)
        torch.cuda.synchronize()
        return {k: r.stats[k] for k in ("ms_csr", "ms_count", "ms_expand", "ms_merge", "ms_assign")}

    def kernels_and_roofline(last, sums, traffic_key):
        R = last.num_premerge_arcs
        st = last.stats
        ab = algorithmic_bytes(st, R, args.no_reduction)
        kern = {}
        write_kernel = "k_expand" + (" / k_unreduced_product" if args.no_reduction else "")
        for name, kernel, ms_key, n_key in (("write", write_kernel, "ms_write_kernel", "write_launches"),
                                            ("merge", "k_merge_dense", "ms_merge_kernel", "merge_launches"),
                                            ("sort", "k_merge_listed" if st["merge_launches"]
                                             else "k_merge_tiles", "ms_sort_kernel", "sort_launches")):
            ms = sums[ms_key] / args.steps
            launches = max(1, st[n_key])
            gbs = ab[name] / (ms * 1e-3) / 1e9 if ms > 0 else 0.0
            kern[name] = {"kernel": kernel, "ms_per_step": ms, "launches_per_step": st[n_key],
                          "avg_launch_ms": ms / launches, "bytes_per_step": ab[name],
                          "bytes_per_launch": ab[name] / launches, "GBps": gbs}
        both_ms = sum(k["ms_per_step"] for k in kern.values())
        kern["expand+merge"] = {"ms_per_step": both_ms, "bytes_per_step": sum(ab.values()),
                                "GBps": sum(ab.values()) / (both_ms * 1e-3) / 1e9 if both_ms else 0.0}
        pms = sums["ms_product_kernel"] / args.steps
        pl = max(1, st["product_launches"])
        pf = product_flops(st)
        kern["product"] = {"kernel": "k_prod_quad + k_prod_sources", "ms_per_step": pms,
                           "launches_per_step": st["product_launches"], "avg_launch_ms": pms / pl,
                           "sources_per_step": st["total_product_sources"],
                           "joined_pairs_per_step": st["total_product_records"],
                           "mfma_sources_per_step": st["total_product_mfma_sources"],
                           "flops_per_step": pf,
                           "TFLOPps": pf / (pms * 1e-3) / 1e12 if pms > 0 else 0.0}
        rec_ms = {k: kern[k]["ms_per_step"] for k in ab}
        dom = max(rec_ms, key=rec_ms.get)
        exact = traffic_key and not args.max_levels and not args.no_reduction
        if pms == 0 and rec_ms[dom] == 0:
            # no per-level kernel ran: the one-workgroup kernels took every
            # level; their bytes are the result they write (20 B per arc, 9 B
            # per state), over the whole step
            step_ms = secs * 1e3 / args.steps
            nbytes = last.num_arcs * 20 + last.num_states * 9
            gbs = nbytes / (step_ms * 1e-3) / 1e9
            roof = {"bound": "hbm", "kernel": "k_small_levels",
                    "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": gbs / HBM_PEAK_GBS, "traffic": None,
                    "limiter": "one workgroup runs every level (a few dozen pairs each): the "
                               "latency of its dependent steps and the host's wait, not bandwidth"}
            return kern, roof
        if pms > rec_ms[dom]:
            # the product merge dominates: its arithmetic is one multiply and
            # one add per joined pair, in float64 on the matrix cores when every
            # source took that form (else vector float64); its bound in practice
            # is the per-source chain of dependent loads
            on_mfma = st["total_product_mfma_sources"] == st["total_product_sources"]
            peak = FP64_MFMA_PEAK_TFLOPS if on_mfma else FP64_VECTOR_PEAK_TFLOPS
            # counter bytes of the four-source kernel, which merges every
            # source of this workload (the one-per-wave kernel finds its list
            # empty); the launch time covers both kernels of the level
            traffic = recorded_traffic("k_prod_quad", traffic_key) if exact else None
            roof = {"bound": "mfma" if on_mfma else "alu", "kernel": "k_prod_quad + k_prod_sources",
                    "achieved": kern["product"]["TFLOPps"], "peak": peak,
                    "unit": "TFLOP/s", "frac": kern["product"]["TFLOPps"] / peak,
                    "traffic": traffic,
                    "limiter": "latency: each wave's chain of dependent loads (header, "
                               "symbols and arcs, visited-array claim), not arithmetic"}
            if traffic:
                gbs = traffic / (kern["product"]["avg_launch_ms"] * 1e-3) / 1e9
                roof["hbm_counter_GBps"] = gbs
                roof["hbm_counter_frac"] = gbs / HBM_PEAK_GBS
        else:
            kname = kern[dom]["kernel"]
            roof = {"bound": "hbm", "kernel": kname,
                    "achieved": kern[dom]["GBps"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": kern[dom]["GBps"] / HBM_PEAK_GBS,
                    "traffic": recorded_traffic(kname, traffic_key) if exact else None}
        return kern, roof

    product = not args.no_product
    secs, last, sums = timed(product)
    R, merged = last.num_premerge_arcs, last.num_arcs
    pre_rate = R * args.steps / secs
    post_rate = merged * args.steps / secs
    key = traffic_key if product else (traffic_key + "_records" if traffic_key else None)
    kern, roof = kernels_and_roofline(last, sums, key)

    out = {
        "metric": METRIC,
        "value": pre_rate,
        "unit": "arcs/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": secs * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": workload
                        + (f", depth cap {args.max_levels}" if args.max_levels else "")
                        + (", without reduction (every joined arc pair kept)"
                           if args.no_reduction else "")
                        + (", fused expand + merge" if args.fused else "")
                        + (", no product merge" if args.no_product else ""),
            "states": last.num_states,
            "premerge_arcs": R,
            "merged_arcs": merged,
            "levels": last.num_levels,
            "input_sha256": [h1.digest()[:16], h2.digest()[:16]],
        },
        "peak_device_GiB": last.stats["peak_device_bytes"] / 2**30,
        "post_merge_arcs_per_s": post_rate,
        # one more, untimed step with an event at every phase boundary (the
        # timed steps record events around the single-kernel phases only)
        "phase_ms_untimed_step": phase_times(product),
        "kernels": kern,
        "roofline": roof,
    }
    if product and not args.no_record_path and not args.no_reduction:
        rsecs, rlast, rsums = timed(False)
        rkern, rroof = kernels_and_roofline(rlast, rsums,
                                            traffic_key + "_records" if traffic_key else None)
        out["record_path"] = {
            "what": "same workload, every source through written records (opts.no_product_merge)",
            "value": rlast.num_premerge_arcs * args.steps / rsecs,
            "ms_per_step": rsecs * 1e3 / args.steps,
            "kernels": {k: rkern[k] for k in ("write", "merge", "sort", "expand+merge")},
            "roofline": rroof,
        }
        em = rkern["expand+merge"]
    else:
        em = kern["expand+merge"] if kern["expand+merge"]["ms_per_step"] else None
    if em:
        # the materialise-then-merge kernels (arc-pair write pass, tile merges)
        # against the HBM peak and the probe's achievable bandwidth
        out["expand_merge_hbm"] = {
            "kernels": "k_expand + k_merge_dense + sort-tile merge",
            "path": "record path (opts.no_product_merge)" if "record_path" in out else "this step",
            "GBps": em["GBps"], "frac_of_peak": em["GBps"] / HBM_PEAK_GBS,
            "frac_of_achievable": (em["GBps"] / stream["copy_GBps"]) if stream else None,
            "bytes": "algorithmic: records written and read once (key + float32 weight), 24 B "
                     "per match descriptor, 16 B per merged run written"}
    if stream:
        out["hbm_achievable"] = stream
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(h1, h2, args.oracle_levels, not args.no_reduction,
                                           args.eps_pair)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
