"""Benchmark of the CMC two-tier decode hot path on one MI355X.

A "step" is one pass of the whole hot path over one batch of the workload:
Tier-1 selection (score GEMV + top-k) once, then `decode_steps` (3000)
decode iterations, each a ring-buffer append followed by two-tier decode
attention over [selected memory rows || window].  Throughput is
attention-only generated tokens/s: B * decode_steps * K / (time of K steps),
with every input already resident in HBM when the timed region starts.  No
decoder weights, MLPs or sampling run: the synthetic per-step queries and
K/V rows stand in for the frozen decoder's.

The default workload is one Llama-3-8B-shaped layer (B=1, Hq=32, Hkv=8,
Dh=128, N=2048 memory rows, k=256, W=512, bf16 K/V, 3000 steps).

The JSON line also carries:
  roofline      for the dominant kernel (two-tier decode): algorithmic bytes
                per launch / average launch duration, measured here with HIP
                events on the launch stream, against the 8 TB/s HBM peak;
                `traffic` comes from committed rocprofv3 counter data when it
                was taken on the current kernel source, else null;
  cpu_baseline  the fp64 CPU oracle timed on this host's cores on a bounded
                sample of the same workload (rank 0, one GPU only).
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
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
DECODE_SOURCES = ["paper_2609_25537_amd/csrc/decode.hip", "paper_2609_25537_amd/csrc/device_common.hpp"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "decode_traffic.json")


def decode_kernel_hash() -> str:
    h = hashlib.sha256()
    for f in DECODE_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5, help="timed passes (each = select + decode_steps)")
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="llama3_8b_layer")
    ap.add_argument("--decode-steps", type=int, default=None, help="override the workload's 3000")
    ap.add_argument("--step-pool", type=int, default=None,
                    help="distinct per-step input sets (rotated); default all steps up to 4096 rows of q")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="budget of the CPU oracle sample")
    ap.add_argument("--eager", action="store_true",
                    help="launch every kernel from Python instead of replaying a captured HIP graph")
    ap.add_argument("--out", default=None, help="also append the JSON line to this file")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only run plain device-to-device copies of MIB MiB (calibrates byte counters) and exit")
    ap.add_argument("--pmc-summary", nargs=4, metavar=("FETCH_DIR", "WRITE_DIR", "COPY_FETCH_DIR", "COPY_WRITE_DIR"),
                    help="turn rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE output directories (decode kernel of "
                         "--workload, and a --copy-probe run) into the per-launch HBM traffic record in "
                         "profiles/decode_traffic.json; runs on the CPU")
    ap.add_argument("--copy-probe-mib", type=int, default=1024, help="size the copy probe ran with")
    ap.add_argument("--launch-reps", type=int, default=500,
                    help="back-to-back decode launches timed for the roofline figure")
    return ap.parse_args()


def to_dev(x, dev):
    import torch
    x = np.ascontiguousarray(x)
    if x.dtype == np.uint16:
        return torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).to(dev)
    return torch.from_numpy(x).to(dev)


class Inputs:
    """Device-resident inputs of one workload (single layer)."""

    def __init__(self, w, steps, pool, dev):
        import torch
        from paper_2609_25537_amd import workloads as wl
        self.w = w
        self.keys = to_dev(wl.sel_keys(w), dev)
        self.qv = to_dev(wl.q_vecs(w), dev)
        pk, pv = wl.pool_kv(w)
        self.pk, self.pv = to_dev(pk, dev), to_dev(pv, dev)
        wk, wv, cnt = wl.window_kv(w)
        self.wk, self.wv, self.wc = to_dev(wk, dev), to_dev(wv, dev), to_dev(cnt, dev)
        self.wc0 = self.wc.clone()
        self.P = min(steps, pool)
        self.q = [to_dev(wl.step_q(w, t), dev) for t in range(self.P)]
        nkv = [wl.step_new_kv(w, t) for t in range(self.P)]
        self.nk = [to_dev(a, dev) for a, _ in nkv]
        self.nv = [to_dev(b, dev) for _, b in nkv]
        self.idx = torch.empty((w.B, w.k), dtype=torch.int32, device=dev)
        self.out = torch.empty((w.B, w.Hq, w.Dh), dtype=torch.float32, device=dev)
        from paper_2609_25537_amd import cmc
        self.sel_ws = torch.empty(max(1, cmc.cmc_select_workspace_bytes(w.B, w.N)), dtype=torch.uint8, device=dev)
        self.dec_ws = cmc.decode_workspace(w.B, w.Hq, w.Hkv, w.Dh, w.k, w.W, dev)


def run_pass(inp: Inputs, steps: int):
    """One pass of the hot path: select once, then `steps` decode iterations."""
    from paper_2609_25537_amd import cmc
    w = inp.w
    cmc.cmc_select_cmes(inp.keys, inp.qv, w.k, idx_out=inp.idx, workspace=inp.sel_ws)
    for t in range(steps):
        j = t % inp.P
        cmc.cmc_decode_step(inp.q[j], inp.pk, inp.pv, inp.idx, w.k, inp.wk, inp.wv, inp.wc, inp.nk[j], inp.nv[j],
                            w.scale, out=inp.out, workspace=inp.dec_ws)


def decode_bytes(w) -> int:
    """Algorithmic bytes of one decode-step launch: K and V of the k + W
    keys (ring full, the newest row read from the appended input), the
    appended row written into the ring, q, out and the index list."""
    kv = w.B * w.Hkv * (w.k + w.W) * w.Dh * w.kv_bytes * 2
    ring_write = w.B * w.Hkv * w.Dh * w.kv_bytes * 2
    return kv + ring_write + w.B * w.Hq * w.Dh * 4 * 2 + w.B * w.k * 4


def capture(fn):
    """Capture fn's launches into a HIP graph (after one warm-up run)."""
    import torch
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        fn()
    torch.cuda.current_stream().wait_stream(s)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


def time_decode_launch(inp: Inputs, reps: int = 500):
    """Average duration of one decode launch: `reps` back-to-back launches
    replayed from a graph, bracketed by HIP events on the replay stream."""
    import torch
    from paper_2609_25537_amd import cmc
    w = inp.w

    def launches():
        for r in range(reps):
            j = r % inp.P
            cmc.cmc_decode_step(inp.q[j], inp.pk, inp.pv, inp.idx, w.k, inp.wk, inp.wv, inp.wc, inp.nk[j],
                                inp.nv[j], w.scale, out=inp.out, workspace=inp.dec_ws)

    g = capture(launches)
    s = torch.cuda.current_stream()
    g.replay()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    s.synchronize()
    a.record(s)
    g.replay()
    b.record(s)
    b.synchronize()
    return a.elapsed_time(b) / reps * 1e-3  # seconds


def cpu_baseline(w, budget_s: float):
    """Time the fp64 CPU oracle on a bounded sample: one selection and as
    many decode iterations as fit in the budget; report tokens/s for a full
    pass (selection amortised over the workload's decode steps)."""
    import oracle
    from paper_2609_25537_amd import workloads as wl
    orc = oracle.default()
    keys, qv = wl.sel_keys(w), wl.q_vecs(w)
    t0 = time.perf_counter()
    idx, _, _ = orc.select(keys, qv, w.k)
    t_sel = time.perf_counter() - t0
    pk, pv = wl.pool_kv(w)
    wk, wv, cnt = wl.window_kv(w)
    n, t_dec = 0, 0.0
    while (n < 8 or t_dec < budget_s) and n < w.steps:
        nk, nv = wl.step_new_kv(w, n)
        q = wl.step_q(w, n)
        t0 = time.perf_counter()
        orc.window_append(wk, wv, cnt, nk, nv)
        orc.two_tier_decode(q, pk, pv, idx, w.k, wk, wv, cnt, w.W, w.scale)
        t_dec += time.perf_counter() - t0
        n += 1
    per_step = t_dec / n
    full = t_sel + w.steps * per_step
    return {"value": w.B * w.steps / full, "unit": "tokens/s", "cores": orc.num_threads(), "kind": "oracle",
            "sample": (f"1 selection ({t_sel:.3f} s) + {n} of {w.steps} decode steps "
                       f"({per_step * 1e3:.2f} ms/step), extrapolated to one full pass")}


def _counter_values(d, counter, kernel):
    import csv
    import glob
    vals = []
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            if r["Counter_Name"] == counter and r["Kernel_Name"].startswith(kernel):
                vals.append(float(r["Counter_Value"]))
    if not vals:
        raise SystemExit(f"no {counter} samples for {kernel} under {d}")
    return sorted(vals)[len(vals) // 2], len(vals)


def pmc_summary(args):
    """Per-launch HBM traffic of the decode kernel from FETCH_SIZE and
    WRITE_SIZE (KiB per dispatch), each scaled by what the same counter reads
    for a plain device copy of known size."""
    from paper_2609_25537_amd import workloads as wl
    w = wl.get(args.workload)
    fd, wd, cfd, cwd = args.pmc_summary
    known_kib = args.copy_probe_mib * 1024.0
    copy_fetch, _ = _counter_values(cfd, "FETCH_SIZE", "__amd_rocclr_copyBuffer")
    copy_write, _ = _counter_values(cwd, "WRITE_SIZE", "__amd_rocclr_copyBuffer")
    fetch, nf = _counter_values(fd, "FETCH_SIZE", "decode_kernel")
    write, nw = _counter_values(wd, "WRITE_SIZE", "decode_kernel")
    fs, ws = known_kib / copy_fetch, known_kib / copy_write
    fetch_b, write_b = fetch * fs * 1024, write * ws * 1024
    rec = {"kernel_hash": decode_kernel_hash(), "bytes_per_launch": round(fetch_b + write_b),
           "fetch_bytes": round(fetch_b), "write_bytes": round(write_b),
           "fetch_kib_raw": fetch, "write_kib_raw": write, "fetch_scale": round(fs, 4), "write_scale": round(ws, 4),
           "dispatches": [nf, nw], "algorithmic_bytes": decode_bytes(w)}
    data = {}
    if os.path.exists(TRAFFIC_FILE):
        with open(TRAFFIC_FILE) as f:
            data = json.load(f)
    data[w.name] = rec
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(data, f, indent=1, sort_keys=True)
        f.write("\n")
    print(json.dumps({w.name: rec}))


def main():
    args = parse()
    if args.pmc_summary:
        pmc_summary(args)
        return
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU only; --gpus {args.gpus} is not supported "
              "(each sequence shards independently across GPUs, see the design notes).", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2609_25537_amd import cmc
    from paper_2609_25537_amd import workloads as wl

    if args.copy_probe:
        n = args.copy_probe << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda:0")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(2):
            dst.copy_(src)
        e1.record()
        torch.cuda.synchronize()
        sec = e0.elapsed_time(e1) * 1e-3 / 2
        print(json.dumps({"copy_probe_bytes": n, "launches": 3, "copy_s": sec,
                          "copy_read_plus_write_GBs": round(2 * n / sec / 1e9, 1)}), flush=True)
        return

    cmc.lib()  # fail loudly before any work if the HIP library is missing
    dev = torch.device("cuda:0")
    w = wl.get(args.workload)
    if w.layers != 1:
        raise SystemExit(f"workload {w.name} has {w.layers} layers; use bench_stack mode (not in this build yet)")
    steps = args.decode_steps or w.steps
    pool = args.step_pool or (steps if w.B * w.Hq * w.Dh * 4 <= (1 << 20) else 64)
    inp = Inputs(w, steps, pool, dev)
    torch.cuda.synchronize()

    graph = None if args.eager else capture(lambda: run_pass(inp, steps))

    def one():
        if graph is not None:
            graph.replay()
        else:
            run_pass(inp, steps)

    for _ in range(args.warmup):
        one()
    torch.cuda.synchronize()
    s = torch.cuda.current_stream()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(s)
    for _ in range(args.steps):
        one()
    e1.record(s)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    ms_per_step = ms / args.steps
    tokens = w.B * steps * args.steps
    value = tokens / (ms * 1e-3)

    t_launch = time_decode_launch(inp, args.launch_reps)
    nbytes = decode_bytes(w)
    achieved = nbytes / t_launch / 1e9
    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        with open(TRAFFIC_FILE) as f:
            tr = json.load(f)
        entry = tr.get(w.name)
        if entry and entry.get("kernel_hash") == decode_kernel_hash():
            traffic = entry.get("bytes_per_launch")
    roofline = {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                "kernel": "decode_kernel (cmc_decode_step)", "bytes_per_launch": nbytes,
                "launch_us": round(t_launch * 1e6, 3)}

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, args.cpu_seconds)

    line = {
        "metric": "two-tier decode tokens/s and achieved HBM GB/s (% of MI355X peak)",
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.kv_dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "Hq": w.Hq, "Hkv": w.Hkv, "Dh": w.Dh, "N": w.N,
                   "D": w.D, "k": w.k, "W": w.W, "decode_steps": steps, "layers": w.layers,
                   "kv_dtype": w.kv_dtype, "step_input_sets": inp.P, "graph": bool(graph)},
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    txt = json.dumps(line)
    print(txt, flush=True)
    if args.out:
        with open(args.out, "a") as f:
            f.write(txt + "\n")


if __name__ == "__main__":
    main()
