"""Benchmark: exact Top-2048 over the decode batch (64 ragged FP32 rows, L
uniform in [16384, 131072]) on one MI355X.

A step is one topk_ragged call over one batch already resident in HBM.  Calls
rotate over enough distinct copies of the batch (>= 512 MB in total) that the
256 MB last-level cache cannot serve repeats; they are captured in HIP graphs
(one call per graph node, as a serving loop would replay them) and replayed
back-to-back on one stream.  HIP events on that stream bracket exactly
`--steps` calls after exactly `--warmup` untimed ones; a busy kernel queued
just before the first event keeps the host's graph launch out of the timed
region.  `--rounds` more rounds of about 100 calls are timed separately and
their median is reported beside the main figure.  The line also carries the
time of the library's read-only ceiling kernel over the same rows (every valid
score read once with the same work items and loads, no selection): what a
single launch of this geometry can reach at all.

Metric: effective score-read bandwidth = 4 B x sum(L) per call / time per
call, the algorithmic bytes of an exact selector (one complete read of every
valid score), reported with the per-call time.  The JSON line also carries the
roofline of the kernel (HBM bound, 8 TB/s peak), route counts, and the CPU
oracle timed on the host cores on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, published
MALL_BYTES = 256 << 20
ROTATE_MIN_BYTES = 512 << 20
KERNEL_SRC = os.path.join(ROOT, "paper_2609_08450_amd", "csrc", "topk_ragged.hip")
WORKLOAD_NAMES = {1: "tiny", 2: "decode", 3: "chunked_prefill", 4: "long_split", 5: "adversarial"}


def traffic_file(config: int) -> str:
    return os.path.join(ROOT, "profiles", f"traffic_{WORKLOAD_NAMES[config]}.json")


def kernel_source_hash() -> str:
    with open(KERNEL_SRC, "rb") as fh:
        return hashlib.sha256(fh.read()).hexdigest()[:16]


def measured_traffic(config: int):
    """HBM bytes per launch from the committed rocprofv3 counter runs, or None
    when they are missing or were taken on a different kernel source."""
    try:
        with open(traffic_file(config)) as fh:
            t = json.load(fh)
    except (OSError, ValueError):
        return None
    if t.get("kernel_source_sha256_16") != kernel_source_hash() or t.get("config") != config:
        return None
    return t.get("hbm_bytes_per_launch")


def make_workload(config: int):
    from paper_2609_08450_amd import workloads as W

    return W.make(config)


def host_cpu():
    """CPU model and the cores this process may run on."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            for ln in fh:
                if ln.startswith("model name"):
                    model = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:
        avail = os.cpu_count() or 1
    return model, avail


def _time_oracle(wl, budget_s: float, threads: int):
    import oracle

    oracle.topk_ragged(wl.scores[:0], wl.row_offsets[:0], wl.row_lengths[:0], wl.K, threads)
    reps, t0 = 0, time.perf_counter()
    while True:
        oracle.topk_ragged(wl.scores, wl.row_offsets, wl.row_lengths, wl.K, threads)
        reps += 1
        el = time.perf_counter() - t0
        if el >= budget_s:
            break
    return reps, el


def cpu_baseline(wl, budget_s: float):
    """The oracle as it stands, on the host cores: whole copies of the batch
    until about budget_s seconds have passed with every available core (the
    OpenMP thread count is capped by OMP_NUM_THREADS when that is set), and a
    third of that with one thread."""
    model, avail = host_cpu()
    threads = avail
    env = os.environ.get("OMP_NUM_THREADS", "")
    if env.isdigit() and int(env) > 0:
        threads = min(threads, int(env))
    reps, el = _time_oracle(wl, budget_s, threads)
    reps1, el1 = _time_oracle(wl, budget_s / 3.0, 1)
    gbs = 4.0 * wl.total_len * reps / el / 1e9
    gbs1 = 4.0 * wl.total_len * reps1 / el1 / 1e9
    return {"value": round(gbs, 3), "unit": "GB/s", "cores": threads, "kind": "oracle",
            "sample": f"{reps} full batches ({wl.n_rows} rows, {wl.total_len} scores each) "
                      f"in {el:.1f} s on {threads} OpenMP threads; plain sort oracle",
            "us_per_call": round(el / reps * 1e6, 1),
            "single_thread": {"value": round(gbs1, 3), "unit": "GB/s",
                              "us_per_call": round(el1 / reps1 * 1e6, 1),
                              "sample": f"{reps1} full batches in {el1:.1f} s"},
            "cpu_model": model, "cpus_available": avail}


def copy_calibration(mib: int, steps: int, warmup: int):
    """A plain device-to-device copy of a known size (the runtime's copy
    kernel), timed with HIP events.  Run under rocprofv3 --pmc, its FETCH_SIZE
    and WRITE_SIZE readings calibrate the same counters taken on the Top-K
    kernel: each should read `bytes` per dispatch."""
    import torch

    dev = torch.device("cuda", 0)
    n = (mib << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device=dev)
    dst = torch.zeros_like(src)
    for _ in range(warmup):
        dst.copy_(src)
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(steps):
        dst.copy_(src)
    ev1.record()
    ev1.synchronize()
    us = ev0.elapsed_time(ev1) * 1e3 / max(1, steps)
    print(json.dumps({"calibration": "device-to-device copy", "bytes": 4 * n,
                      "us_per_copy": round(us, 3),
                      "read_plus_write_GBs": round(8.0 * n / (us * 1e-6) / 1e9, 1)}), flush=True)


def _pmc_mean_kib(csv_path: str, kernel_substr: str, counter: str, min_grid: int = 0):
    import csv

    vals = []
    with open(csv_path, newline="") as fh:
        for row in csv.DictReader(fh):
            if (kernel_substr in row["Kernel_Name"] and row["Counter_Name"] == counter
                    and int(row["Grid_Size"]) >= min_grid):
                vals.append(float(row["Counter_Value"]))
    if not vals:
        raise SystemExit(f"no {counter} rows for {kernel_substr!r} in {csv_path}")
    return sum(vals) / len(vals), len(vals)


def traffic_summary(paths, config: int, copy_mib: int, out_path: str):
    """Turns four rocprofv3 --pmc counter CSVs (kernel FETCH_SIZE, kernel
    WRITE_SIZE, copy FETCH_SIZE, copy WRITE_SIZE) into HBM bytes per launch of
    the Top-K kernel, each counter scaled by copy_bytes / copy_reading."""
    kf, kw, cf, cw = paths
    copy_bytes = copy_mib << 20
    f_kib, nf = _pmc_mean_kib(kf, "topk_ragged_kernel", "FETCH_SIZE")
    w_kib, nw = _pmc_mean_kib(kw, "topk_ragged_kernel", "WRITE_SIZE")
    cf_kib, _ = _pmc_mean_kib(cf, "copyBuffer", "FETCH_SIZE")
    cw_kib, _ = _pmc_mean_kib(cw, "copyBuffer", "WRITE_SIZE")
    sf = copy_bytes / (cf_kib * 1024.0)
    sw = copy_bytes / (cw_kib * 1024.0)
    wl = make_workload(config)
    fetch = f_kib * 1024.0 * sf
    write = w_kib * 1024.0 * sw
    out = {"config": config, "kernel": "topk_ragged_kernel",
           "kernel_source_sha256_16": kernel_source_hash(),
           "fetch_kib_per_dispatch": round(f_kib, 1), "write_kib_per_dispatch": round(w_kib, 1),
           "dispatches": [nf, nw],
           "copy_bytes": copy_bytes, "copy_fetch_kib": round(cf_kib, 1),
           "copy_write_kib": round(cw_kib, 1),
           "fetch_scale": round(sf, 4), "write_scale": round(sw, 4),
           "hbm_fetch_bytes_per_launch": round(fetch), "hbm_write_bytes_per_launch": round(write),
           "hbm_bytes_per_launch": round(fetch + write),
           "algorithmic_bytes_per_launch": 4 * wl.total_len,
           "traffic_over_algorithmic": round((fetch + write) / (4.0 * wl.total_len), 4)}
    with open(out_path, "w") as fh:
        json.dump(out, fh, indent=1)
        fh.write("\n")
    print(json.dumps(out))


SPACER_CYCLES = 20_000_000  # ~10 ms busy kernel ahead of a timed region


def upload_graph(g, stream) -> bool:
    """hipGraphUpload of a captured graph's executable on `stream`: the
    runtime's one-time copy of the graph to the device happens here rather
    than inside the first timed replay.  Runs no kernel."""
    import ctypes

    try:
        path = None
        with open("/proc/self/maps") as fh:
            for ln in fh:
                if "libamdhip64" in ln:
                    path = ln.split()[-1]
                    break
        hip = ctypes.CDLL(path or "libamdhip64.so")
        hip.hipGraphUpload.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        hip.hipGraphUpload.restype = ctypes.c_int
        rc = hip.hipGraphUpload(ctypes.c_void_p(g.raw_cuda_graph_exec()),
                                ctypes.c_void_p(stream.cuda_stream))
        stream.synchronize()
        return rc == 0
    except Exception:
        return False


def time_calls(wl, policy, steps, warmup, rotate=True, calls_per_graph=0, rounds=0,
               round_calls=100, ceiling=False):
    """Times exactly `steps` topk_ragged calls on workload wl (policy None =
    the production call) over rotated device copies, captured in HIP graphs
    and replayed on one stream between HIP events on that stream, after
    exactly `warmup` untimed calls.  A busy kernel is queued ahead of the
    first event so that the host's graph launch is not inside the timed
    region.  With rounds > 0, also times that many separate rounds of about
    round_calls calls each and reports their median.  ceiling: time the
    library's read-only ceiling kernel over the same rows instead of the
    selector.  Returns a dict."""
    import torch

    from paper_2609_08450_amd import topk

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    K, n = wl.K, wl.n_rows
    batch_bytes = 4 * wl.scores.size
    copies = max(1, -(-ROTATE_MIN_BYTES // batch_bytes)) if rotate else 1
    stream = torch.cuda.Stream(device=dev)

    with torch.cuda.stream(stream):
        host = torch.from_numpy(wl.scores)
        bufs = [host.to(dev) for _ in range(copies)]
        offs = torch.from_numpy(wl.row_offsets).to(dev)
        lens = torch.from_numpy(wl.row_lengths).to(dev)
        out_idx = torch.empty((n, K), dtype=torch.int32, device=dev)
        out_val = torch.empty((n, K), dtype=torch.float32, device=dev)
        out_max = torch.zeros(n, dtype=torch.int32, device=dev)
        ws = topk.alloc_workspace(n, K, dev, stream)
    stream.synchronize()

    def call(i, s):
        if ceiling:
            topk.debug_read_ceiling(bufs[i % copies], offs, lens, n, K, out_max, ws, s)
        elif policy is None:
            topk.topk_ragged(bufs[i % copies], offs, lens, n, K, out_idx, out_val, ws, s)
        else:
            topk.topk_ragged_ex(bufs[i % copies], offs, lens, n, K, out_idx, out_val, ws,
                                policy, None, s)

    # a graph of G consecutive calls over rotating copies, and a tail graph
    # for the remainder, so that exactly `steps` calls are timed
    G = calls_per_graph or copies
    G = max(1, min(G, steps)) if steps > 0 else 1

    def capture(ncalls):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            for j in range(ncalls):
                call(j, torch.cuda.current_stream())
        return g

    # warm-up: exactly `warmup` untimed calls (eager; the first loads the code)
    with torch.cuda.stream(stream):
        for i in range(warmup):
            call(i, stream)
    stream.synchronize()
    g_main = capture(G)
    rem = steps % G
    g_tail = capture(rem) if rem else None
    stream.synchronize()
    uploaded = upload_graph(g_main, stream) and (g_tail is None or upload_graph(g_tail, stream))

    def timed(fn):
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        with torch.cuda.stream(stream):
            torch.cuda._sleep(SPACER_CYCLES)
            ev0.record(stream)
            fn()
            ev1.record(stream)
        ev1.synchronize()
        torch.cuda.synchronize()
        return ev0.elapsed_time(ev1)

    def run(nsteps):
        reps, tail = divmod(nsteps, G)
        for _ in range(reps):
            g_main.replay()
        if tail:
            assert tail == rem
            g_tail.replay()

    ms = timed(lambda: run(steps))
    out = {"ms_per_call": ms / steps, "copies": copies, "copies_touched": min(copies, steps),
           "calls_per_graph": G, "warmup_calls": warmup, "graphs_uploaded": uploaded}

    if rounds > 0:
        reps = max(1, -(-round_calls // G))
        per = sorted(timed(lambda: [g_main.replay() for _ in range(reps)]) / (reps * G)
                     for _ in range(rounds))
        out["rounds"] = {"rounds": rounds, "calls_per_round": reps * G,
                         "ms_per_call_median": per[len(per) // 2],
                         "ms_per_call_min": per[0], "ms_per_call_max": per[-1]}

    # outside the timed region: route counts of one call
    if not ceiling:
        topk.read_stats(ws, stream)
        with torch.cuda.stream(stream):
            call(0, stream)
        out["routes"] = topk.read_stats(ws, stream)
    del bufs, g_main, g_tail
    torch.cuda.synchronize()
    return out


ABLATIONS = ("margin", "stride", "rescue", "crossover", "k", "recal", "recal-crossover", "batch",
             "ties")


def ablation(name, wl, steps, warmup):
    """The paper's policy ablations (Section 6: retention margin, sampling
    stride, conditional rescue, sampled-versus-exact crossover) and other K,
    on synthetic rows: per variant the time per call and the route counts."""
    from paper_2609_08450_amd import topk
    from paper_2609_08450_amd import workloads as W

    base = topk.default_policy()

    def pol(**kw):
        p = topk.Policy(**base.as_dict())
        for k, v in kw.items():
            setattr(p, k, v)
        return p

    def with_k(w, K):
        return W.Workload(f"{w.name} K={K}", w.scores, w.row_offsets, w.row_lengths, K,
                          w.description)

    variants = []
    if name == "margin":      # K~ = rho K at s = 128, primary only (rho1 = rho)
        for num, den in ((1, 1), (5, 4), (3, 2), (7, 4), (2, 1)):
            variants.append((f"rho={num}/{den}", wl,
                             pol(rho_num=num, rho_den=den, rho1_num=num, rho1_den=den)))
    elif name == "stride":    # s from 16 to 256 at rho = 3/2, primary only
        for sl in (4, 5, 6, 7, 8):
            variants.append((f"s={1 << sl}", wl, pol(s_log2=sl, rho1_num=3, rho1_den=2)))
    elif name == "rescue":    # nested band (rho1 = 7/4) against primary only
        variants = [("rescue rho1=7/4", wl, base), ("primary only", wl, pol(rho1_num=3, rho1_den=2))]
    elif name == "crossover": # fixed-length decode rows, sampled against exact route
        for L in (8192, 16384, 32768, 65536, 131072):
            rng = np.random.default_rng(260908450 + L)
            rows = [W.decode_mixture_row(rng, L).astype(np.float32) for _ in range(64)]
            lens = np.full(64, L, np.int32)
            offs = (np.arange(64, dtype=np.int64) * L)
            wlL = W.Workload(f"64 rows L={L}", np.concatenate(rows), offs, lens, 2048, "decode mixture")
            variants.append((f"L={L} sampled", wlL, pol(l_samp_min=0)))
            variants.append((f"L={L} exact", wlL, pol(l_samp_min=0x7FFFFFFF)))
    elif name == "k":         # the K = 2048 constants against the per-K policy
        for K in (256, 512, 1024, 2048, 4096, 8192):
            variants.append((f"K={K} evaluated constants", with_k(wl, K), base))
            variants.append((f"K={K} per-K policy", with_k(wl, K), topk.policy_for_k(K)))
    elif name == "recal":     # other K: stride and margins around the sample rank
        for K, pairs in ((256, ((3, 2, 7, 4), (2, 1, 5, 2), (3, 1, 4, 1))),
                         (512, ((3, 2, 7, 4), (2, 1, 5, 2), (3, 1, 4, 1))),
                         (1024, ((3, 2, 7, 4), (2, 1, 5, 2), (3, 1, 4, 1))),
                         (4096, ((5, 4, 11, 8), (4, 3, 3, 2), (3, 2, 7, 4)))):
            for sl in (4, 5, 6, 7):
                for rn, rd, r1n, r1d in pairs:
                    variants.append((f"K={K} s={1 << sl} rho={rn}/{rd} rho1={r1n}/{r1d}",
                                     with_k(wl, K),
                                     pol(s_log2=sl, rho_num=rn, rho_den=rd, rho1_num=r1n,
                                         rho1_den=r1d)))
    elif name == "batch":     # decode rows, more of them: where the latency chain amortises
        for n in (16, 32, 64, 128, 256, 512, 1024):
            variants.append((f"rows={n}", W.decode(n_rows=n), None))
    elif name == "ties":      # decode-shaped rows with heavy ties (exact route, re-read)
        variants = [("decode rows", W.decode(), None),
                    ("clustered 256-value codebook per row", W.decode_ties("clustered"), None),
                    ("8000 ties above the K-th score", W.decode_ties("block"), None)]
    elif name == "recal-crossover":  # per-K policy: sampled against exact on short rows
        for K in (256, 512, 1024, 2048, 4096):
            kp = topk.policy_for_k(K).as_dict()
            for m in (2, 4, 8, 16, 32):
                L = m * K
                if L > 131072:
                    continue
                rng = np.random.default_rng(260908450 + L + K)
                rows = [W.decode_mixture_row(rng, L).astype(np.float32) for _ in range(64)]
                lens = np.full(64, L, np.int32)
                offs = (np.arange(64, dtype=np.int64) * L)
                wlL = W.Workload(f"64 rows L={L}", np.concatenate(rows), offs, lens, K,
                                 "decode mixture")
                variants.append((f"K={K} L={L} sampled", wlL, pol(**dict(kp, l_samp_min=0))))
                variants.append((f"K={K} L={L} exact", wlL, pol(l_samp_min=0x7FFFFFFF)))
    for label, w, p in variants:
        t = time_calls(w, p, steps, warmup)
        ms, routes = t["ms_per_call"], t["routes"]
        print(json.dumps({"ablation": name, "variant": label, "rows": w.n_rows, "K": w.K,
                          "us_per_call": round(ms * 1e3, 3),
                          "gbs": round(4.0 * w.total_len / (ms * 1e-3) / 1e9, 2),
                          "routes": routes,
                          "policy": (p if p is not None else topk.policy_for_k(w.K)).as_dict()}),
              flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3000)
    ap.add_argument("--warmup", type=int, default=60)
    ap.add_argument("--config", type=int, default=2,
                    help="workload: 1 tiny, 2 decode (headline), 3 chunked prefill, 4 long split, 5 edge mix")
    ap.add_argument("--calls-per-graph", type=int, default=0, help="0 = number of rotated copies")
    ap.add_argument("--rounds", type=int, default=7,
                    help="after the timed steps, this many separately timed rounds of about 100 "
                         "calls (median reported); 0 = none")
    ap.add_argument("--no-rotate", action="store_true", help="reuse one copy (cache-resident input)")
    ap.add_argument("--no-ceiling", dest="ceiling", action="store_false",
                    help="skip timing the read-only ceiling kernel over the same rows")
    ap.add_argument("--cpu-budget", type=float, default=15.0,
                    help="seconds of all-core oracle time (plus a third of it on one thread); "
                         "0 = skip")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only time a plain device copy of MIB MiB (counter calibration)")
    ap.add_argument("--traffic-summary", nargs=4, metavar="CSV",
                    help="kernel FETCH_SIZE, kernel WRITE_SIZE, copy FETCH_SIZE, copy WRITE_SIZE "
                         "counter CSVs from rocprofv3 --pmc; writes the traffic file and exits")
    ap.add_argument("--copy-mib", type=int, default=1024, help="size of the calibration copy")
    ap.add_argument("--traffic-out", default=None,
                    help="where --traffic-summary writes (default: the config's traffic file "
                         "that the bench line reports)")
    ap.add_argument("--ablation", choices=ABLATIONS, default=None,
                    help="instead of the bench line, one JSON line per policy variant (the "
                         "paper's ablations on synthetic rows; --config picks the rows)")
    args = ap.parse_args()

    if args.traffic_summary:
        traffic_summary(args.traffic_summary, args.config, args.copy_mib,
                        args.traffic_out or traffic_file(args.config))
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on one GPU only: there is no multi-GPU launcher. Rows are "
              "independent, so a batch shards by rows, each GPU running the kernel on its "
              "own share.", file=sys.stderr)
        sys.exit(2)

    if args.copy_calibration:
        copy_calibration(args.copy_calibration, max(1, args.steps), args.warmup)
        return

    wl = make_workload(args.config)
    if args.ablation:
        ablation(args.ablation, wl, args.steps, args.warmup)
        return
    t = time_calls(wl, None, args.steps, args.warmup, not args.no_rotate, args.calls_per_graph,
                   rounds=args.rounds)
    ms_per_step = t["ms_per_call"]
    K, n = wl.K, wl.n_rows
    batch_bytes = 4 * wl.scores.size
    alg_bytes = 4.0 * wl.total_len
    gbs = alg_bytes / (ms_per_step * 1e-3) / 1e9

    traffic = measured_traffic(args.config)
    result = {
        "metric": "effective score-read GB/s, exact Top-2048 over ragged FP32 rows",
        "value": round(gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": t["warmup_calls"],
        "ms_per_step": round(ms_per_step, 6),
        "us_per_call": round(ms_per_step * 1e3, 3),
        "frac_of_hbm_peak": round(gbs / HBM_PEAK_GBS, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": wl.name + ": " + wl.description, "rows": n, "K": K,
                   "sum_len": wl.total_len, "bytes_per_call": int(alg_bytes),
                   "copies_touched": t["copies_touched"], "calls_per_graph": t["calls_per_graph"],
                   "touched_bytes": t["copies_touched"] * batch_bytes,
                   "graphs_uploaded": t["graphs_uploaded"]},
        "roofline": {"bound": "hbm", "achieved": round(gbs, 2), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4),
                     "traffic": traffic},
        "routes": t["routes"],
        "kernel": "topk_ragged_kernel",
        "kernel_source_sha256_16": kernel_source_hash(),
    }
    if "rounds" in t:
        rd = t["rounds"]
        result["rounds"] = {"rounds": rd["rounds"], "calls_per_round": rd["calls_per_round"],
                            "us_per_call_median": round(rd["ms_per_call_median"] * 1e3, 3),
                            "us_per_call_min": round(rd["ms_per_call_min"] * 1e3, 3),
                            "us_per_call_max": round(rd["ms_per_call_max"] * 1e3, 3),
                            "gbs_median": round(alg_bytes / (rd["ms_per_call_median"] * 1e-3) / 1e9, 2)}
    if args.ceiling:
        c = time_calls(wl, None, args.steps, args.warmup, not args.no_rotate, args.calls_per_graph,
                       rounds=args.rounds, ceiling=True)
        cms = c["rounds"]["ms_per_call_median"] if "rounds" in c else c["ms_per_call"]
        sms = t["rounds"]["ms_per_call_median"] if "rounds" in t else ms_per_step
        cgbs = alg_bytes / (cms * 1e-3) / 1e9
        result["ceiling"] = {"kernel": "read_ceiling_kernel",
                             "what": "every valid score read once, same work items and loads",
                             "us_per_call": round(cms * 1e3, 3), "gbs": round(cgbs, 2),
                             "frac_of_hbm_peak": round(cgbs / HBM_PEAK_GBS, 4),
                             "selector_frac_of_ceiling": round(cms / sms, 4)}
    if args.cpu_budget > 0:
        result["cpu_baseline"] = cpu_baseline(wl, args.cpu_budget)
    else:
        result["cpu_baseline"] = None
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
