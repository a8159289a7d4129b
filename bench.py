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
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
LLC_BYTES = 256 << 20  # MI355X last-level (Infinity) cache
DECODE_SOURCES = ["paper_2609_25537_amd/csrc/decode.hip", "paper_2609_25537_amd/csrc/device_common.hpp"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "decode_traffic.json")


def _strip_comments(src: str) -> str:
    """C++ source without comments or blank-line differences (the decode
    kernel's code, so that a comment edit keeps its measured counters)."""
    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
    src = re.sub(r"//[^\n]*", "", src)
    return "\n".join(line.rstrip() for line in src.splitlines() if line.strip())


def decode_kernel_hash() -> str:
    h = hashlib.sha256()
    for f in DECODE_SOURCES:
        with open(os.path.join(ROOT, f)) as fh:
            h.update(_strip_comments(fh.read()).encode())
    return h.hexdigest()[:16]


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5, help="timed passes (each = select + decode_steps)")
    ap.add_argument("--warmup", type=int, default=1)
    from paper_2609_25537_amd import workloads as _wl
    names = [*_wl.WORKLOADS, *_wl.DENOISE_WORKLOADS, *_wl.BRIDGE_WORKLOADS]
    ap.add_argument("--workload", default="llama3_8b_layer", metavar="NAME",
                    help="one of: " + ", ".join(names))
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
    ap.add_argument("--vendor-gemm-probe", action="store_true",
                    help="with a MemoryBridge workload: time torch's bf16 addmm (the vendor BLAS) on the "
                         "projection's two GEMM shapes instead of the library, for comparison")
    ap.add_argument("--launch-reps", type=int, default=500,
                    help="back-to-back decode launches timed for the roofline figure")
    ap.add_argument("--batched", choices=["auto", "on", "off"], default="auto",
                    help="add the batched legs (the 32-layer stack's decode launches and the Mistral-shaped batch "
                         "over 8 layer copies, launches rotating so that nothing is served from the last-level "
                         "cache) to the JSON line; auto: with the default workload")
    ap.add_argument("--baseline-steps", type=int, default=4,
                    help="stack workloads: timed decode steps of the uncompressed-cache baseline (0: skip it)")
    ap.add_argument("--selection-only", action="store_true",
                    help="time only the Tier-1 selection (score pass + top-k) of a uniform decode workload, with "
                         "fp32 keys and with the same keys as bf16, --steps calls each; prints its JSON object")
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
        self.idx = torch.empty((w.B, w.idx_stride), dtype=torch.int32, device=dev)
        self.out = torch.empty((w.B, w.Hq, w.Dh), dtype=torch.float32, device=dev)
        if w.ragged:
            rs = wl.ragged_sizes(w)
            self.n_rows, self.q_rows = to_dev(rs["n_rows"], dev), to_dev(rs["q_rows"], dev)
            self.k_out = torch.empty((w.B,), dtype=torch.int32, device=dev)
        from paper_2609_25537_amd import cmc
        self.sel_ws = torch.empty(max(1, cmc.cmc_select_workspace_bytes(w.B, w.N)), dtype=torch.uint8, device=dev)
        self.dec_ws = cmc.decode_workspace(w.B, w.Hq, w.Hkv, w.Dh, w.idx_stride, w.W, dev)
        # Tier-1 rows gathered once per question into contiguous blocks.
        self.gk = torch.empty((w.B, w.Hkv, w.idx_stride, w.Dh), dtype=self.pk.dtype, device=dev)
        self.gv = torch.empty_like(self.gk)

    def select(self):
        from paper_2609_25537_amd import cmc
        w = self.w
        if w.ragged:
            cmc.cmc_select_cmes_ragged(self.keys, self.qv, self.n_rows, w.k, q_rows=self.q_rows,
                                       idx_stride=w.idx_stride, idx_out=self.idx, k_out=self.k_out,
                                       workspace=self.sel_ws)
        else:
            cmc.cmc_select_cmes(self.keys, self.qv, w.k, idx_out=self.idx, workspace=self.sel_ws)
        cmc.cmc_gather_tier1(self.pk, self.pv, self.idx, w.idx_stride, k_len=self.k_out if w.ragged else None,
                             out_k=self.gk, out_v=self.gv)

    def decode_step(self, j):
        from paper_2609_25537_amd import cmc
        w = self.w
        if w.ragged:
            cmc.cmc_decode_step_ragged(self.q[j], self.gk, self.gv, None, self.k_out, w.idx_stride, self.wk,
                                       self.wv, self.wc, self.nk[j], self.nv[j], w.scale, out=self.out,
                                       workspace=self.dec_ws)
        else:
            cmc.cmc_decode_step(self.q[j], self.gk, self.gv, None, w.k, self.wk, self.wv, self.wc, self.nk[j],
                                self.nv[j], w.scale, out=self.out, workspace=self.dec_ws)


def run_pass(inp: Inputs, steps: int):
    """One pass of the hot path: select (and gather the selected rows) once,
    then `steps` decode iterations."""
    inp.select()
    for t in range(steps):
        inp.decode_step(t % inp.P)


def decode_bytes(w, counts=None) -> float:
    """Algorithmic bytes of one decode-step launch: K and V of each
    sequence's pool rows (k, or a ragged sequence's own k_b + q_b, read from
    the gathered Tier-1 block) and of its ring rows -- min(count_b + 1, W)
    with count_b the tokens in the ring before the launch (its filled slots,
    one of which the appended row replaces once the ring is full, plus that
    row read from the input) -- the appended row written into the ring, q
    and out.  counts None: every ring full.  counts may be [B] or [L][B] (L
    launches: the mean over them)."""
    from paper_2609_25537_amd import workloads as wl
    if w.ragged:
        rs = wl.ragged_sizes(w)
        pool = int(np.minimum(rs["n_rows"], w.k).sum() + rs["q_rows"].sum())
    else:
        pool = w.B * w.k
    if counts is None:
        ring = w.B * w.W
    else:
        c = np.asarray(counts, np.int64).reshape(-1, w.B)
        ring = float(np.minimum(c + 1, w.W).sum(axis=1).mean())
    row = w.Dh * w.kv_bytes * 2
    kv = w.Hkv * (pool + ring) * row
    ring_write = w.B * w.Hkv * row
    total = kv + ring_write + w.B * w.Hq * w.Dh * 4 * 2
    return int(total) if counts is None else float(total)


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
            inp.decode_step(r % inp.P)

    g = capture(launches)
    s = torch.cuda.current_stream()
    g.replay()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    s.synchronize()
    c0 = inp.wc.cpu().numpy().astype(np.int64)  # ring fills before the timed launches
    a.record(s)
    g.replay()
    b.record(s)
    b.synchronize()
    counts = c0[None, :] + np.arange(reps, dtype=np.int64)[:, None]
    return a.elapsed_time(b) / reps * 1e-3, counts  # seconds, [reps][B] counts before each launch


def cpu_baseline(w, budget_s: float):
    """Time the fp64 CPU oracle on a bounded sample: one selection and as
    many decode iterations as fit in the budget; report tokens/s for a full
    pass (selection amortised over the workload's decode steps)."""
    import oracle
    from paper_2609_25537_amd import workloads as wl
    orc = oracle.default()
    keys, qv = wl.sel_keys(w), wl.q_vecs(w)
    rs = wl.ragged_sizes(w)
    t0 = time.perf_counter()
    if w.ragged:
        idx, k_out = orc.select_ragged(keys, qv, rs["n_rows"], w.k, rs["q_rows"], w.idx_stride)
    else:
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
        if w.ragged:
            orc.two_tier_decode_ragged(q, pk, pv, idx, k_out, w.idx_stride, wk, wv, cnt, w.W, w.scale)
        else:
            orc.two_tier_decode(q, pk, pv, idx, w.k, wk, wv, cnt, w.W, w.scale)
        t_dec += time.perf_counter() - t0
        n += 1
    per_step = t_dec / n
    full = t_sel + w.steps * per_step
    # The same oracle on one thread: a few more steps from where the sample
    # stopped (bounded to about a tenth of the budget).
    threads = orc.num_threads()
    orc.set_num_threads(1)
    n1, t1 = 0, 0.0
    try:
        while n1 < 2 or (t1 < budget_s / 10 and n1 < 64):
            nk, nv = wl.step_new_kv(w, (n + n1) % w.steps)
            q = wl.step_q(w, (n + n1) % w.steps)
            t0 = time.perf_counter()
            orc.window_append(wk, wv, cnt, nk, nv)
            if w.ragged:
                orc.two_tier_decode_ragged(q, pk, pv, idx, k_out, w.idx_stride, wk, wv, cnt, w.W, w.scale)
            else:
                orc.two_tier_decode(q, pk, pv, idx, w.k, wk, wv, cnt, w.W, w.scale)
            t1 += time.perf_counter() - t0
            n1 += 1
    finally:
        orc.set_num_threads(threads)
    per_step1 = t1 / n1
    return {"value": w.B * w.steps / full, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "cpu_model": cpu_model(),
            "value_1thread": w.B * w.steps / (t_sel * threads + w.steps * per_step1),
            "sample": (f"1 selection ({t_sel:.3f} s) + {n} of {w.steps} decode steps "
                       f"({per_step * 1e3:.2f} ms/step), extrapolated to one full pass; 1 thread: "
                       f"{n1} steps ({per_step1 * 1e3:.2f} ms/step), selection scaled by the thread count")}


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
    # The counted run starts from the workload's initial ring fills and
    # appends one row per dispatch: the median dispatch (the median counter
    # value, the fetch growing with the fill) saw fill + n // 2 tokens.
    alg = decode_bytes(w)
    if w.layers == 1:
        _, _, cnt0 = wl.window_kv(w)
        alg = round(decode_bytes(w, cnt0.astype(np.int64) + nf // 2))
    rec = {"kernel_hash": decode_kernel_hash(), "bytes_per_launch": round(fetch_b + write_b),
           "fetch_bytes": round(fetch_b), "write_bytes": round(write_b),
           "fetch_kib_raw": fetch, "write_kib_raw": write, "fetch_scale": round(fs, 4), "write_scale": round(ws, 4),
           "dispatches": [nf, nw], "algorithmic_bytes": alg, "algorithmic_bytes_rings_full": decode_bytes(w)}
    data = {}
    if os.path.exists(TRAFFIC_FILE):
        with open(TRAFFIC_FILE) as f:
            data = json.load(f)
    data[w.name] = rec
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(data, f, indent=1, sort_keys=True)
        f.write("\n")
    print(json.dumps({w.name: rec}))


class StackLayer:
    """Device-resident inputs of one decoder layer of a stack workload."""

    def __init__(self, w, layer, P, dev):
        import torch
        from paper_2609_25537_amd import workloads as wl
        bf = torch.bfloat16 if w.kv_dtype == "bf16" else torch.float32
        dn = lambda role, ids, shape, dt=bf: wl.device_normal(w.seed, role, ids, shape, w.kv_std, dev, dt)
        self.pk = dn("cme_k", (layer,), (w.B, w.Hkv, w.N, w.Dh))
        self.pv = dn("cme_v", (layer,), (w.B, w.Hkv, w.N, w.Dh))
        self.wk = dn("win_k", (layer,), (w.B, w.Hkv, w.W, w.Dh))
        self.wv = dn("win_v", (layer,), (w.B, w.Hkv, w.W, w.Dh))
        self.wc = torch.full((w.B,), w.W, dtype=torch.int32, device=dev)
        self.q = [dn("q", (layer, t), (w.B, w.Hq, w.Dh), torch.float32) for t in range(P)]
        self.nk = [dn("new_k", (layer, t), (w.B, w.Hkv, 1, w.Dh)) for t in range(P)]
        self.nv = [dn("new_v", (layer, t), (w.B, w.Hkv, 1, w.Dh)) for t in range(P)]
        self.gk = torch.empty((w.B, w.Hkv, w.k, w.Dh), dtype=bf, device=dev)  # gathered Tier-1 rows
        self.gv = torch.empty_like(self.gk)


def batched_leg(name: str, dev, reps: int = 512, P: int = 4):
    """Launch-level HBM figure of a batched workload, for the same JSON line
    as the headline: its decode launches (cmc_decode_step, rings full)
    rotating over the workload's layers (the 32-layer stack; the Mistral-
    shaped batch over 8 layer copies), replayed from a graph and timed with
    HIP events on the replay stream.  The Tier-1 blocks are drawn directly
    as the gathered rows the decode reads (the selection does not change
    the launch).  Throughput is attention-only tokens/s for all layers."""
    import torch
    from paper_2609_25537_amd import cmc
    from paper_2609_25537_amd import workloads as wl
    w = wl.get(name)
    bf = torch.bfloat16 if w.kv_dtype == "bf16" else torch.float32
    dn = lambda role, ids, shape, dt=bf: wl.device_normal(w.seed, role, ids, shape, w.kv_std, dev, dt)
    layers = []
    for l in range(w.layers):
        layers.append(dict(gk=dn("cme_k", (l, 1), (w.B, w.Hkv, w.k, w.Dh)),
                           gv=dn("cme_v", (l, 1), (w.B, w.Hkv, w.k, w.Dh)),
                           wk=dn("win_k", (l,), (w.B, w.Hkv, w.W, w.Dh)),
                           wv=dn("win_v", (l,), (w.B, w.Hkv, w.W, w.Dh)),
                           wc=torch.full((w.B,), w.W, dtype=torch.int32, device=dev),
                           q=[dn("q", (l, t), (w.B, w.Hq, w.Dh), torch.float32) for t in range(P)],
                           nk=[dn("new_k", (l, t), (w.B, w.Hkv, 1, w.Dh)) for t in range(P)],
                           nv=[dn("new_v", (l, t), (w.B, w.Hkv, 1, w.Dh)) for t in range(P)]))
    out = torch.empty((w.B, w.Hq, w.Dh), dtype=torch.float32, device=dev)
    ws = cmc.decode_workspace(w.B, w.Hq, w.Hkv, w.Dh, w.k, w.W, dev)
    L = len(layers)

    def launches():
        for r in range(reps):
            Ly, j = layers[r % L], (r // L) % P
            cmc.cmc_decode_step(Ly["q"][j], Ly["gk"], Ly["gv"], None, w.k, Ly["wk"], Ly["wv"], Ly["wc"],
                                Ly["nk"][j], Ly["nv"][j], w.scale, out=out, workspace=ws)

    g = capture(launches)
    st = torch.cuda.current_stream()
    g.replay()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    st.synchronize()
    a.record(st)
    g.replay()
    b.record(st)
    b.synchronize()
    t = a.elapsed_time(b) / reps * 1e-3
    nbytes = decode_bytes(w)
    achieved = nbytes / t / 1e9
    del g, layers, ws
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return {"workload": w.name, "B": w.B, "Hq": w.Hq, "Hkv": w.Hkv, "Dh": w.Dh, "k": w.k, "W": w.W,
            "layers_rotated": L, "launches_timed": reps,
            "kernel": "decode_kernel (cmc_decode_step), rings full",
            "launch_us": round(t * 1e6, 3), "bytes_per_launch": nbytes,
            "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                         "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": recorded_traffic(w),
                         "cache_resident": False},
            "tokens_per_s_all_layers": round(w.B / (L * t), 1)}


def selection_leg(name: str, dev, reps: int = 5):
    """Tier-1 selection (score pass + top-k, once per question) of a batched
    workload with fp32 keys and with the same keys rounded to bf16
    (key_dtype CMC_BF16): ms per call and the score pass's key bytes per ms.
    Keys and questions are drawn on the device."""
    import torch
    from paper_2609_25537_amd import cmc
    from paper_2609_25537_amd import workloads as wl
    w = wl.get(name)
    keys = wl.device_normal(w.seed, "sel_keys", (0,), (w.B, w.N, w.D), 1.0, dev, torch.float32)
    qv = wl.device_normal(w.seed, "q_vec", (0,), (w.B, w.D), 1.0, dev, torch.float32)
    idx = torch.empty((w.B, w.k), dtype=torch.int32, device=dev)
    ws = torch.empty(max(1, cmc.cmc_select_workspace_bytes(w.B, w.N)), dtype=torch.uint8, device=dev)
    res = {"workload": w.name, "B": w.B, "N": w.N, "D": w.D, "k": w.k}
    for tag, kt in (("fp32_keys", keys), ("bf16_keys", None)):
        if kt is None:
            kt = keys.to(torch.bfloat16)
            del keys
        cmc.cmc_select_cmes(kt, qv, w.k, idx_out=idx, workspace=ws)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            cmc.cmc_select_cmes(kt, qv, w.k, idx_out=idx, workspace=ws)
        b.record()
        b.synchronize()
        ms = a.elapsed_time(b) / reps
        nbytes = kt.numel() * kt.element_size()
        res[tag] = {"ms": round(ms, 4), "key_bytes": nbytes, "GBs": round(nbytes / ms / 1e6, 1),
                    "frac_of_hbm_peak": round(nbytes / ms / 1e6 / HBM_PEAK_GBS, 4)}
        del kt
    del qv, idx, ws
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return res


def run_stack(args, w, dev):
    """A decoder stack of w.layers layers sharing one index list: one pass is
    the selection plus w.steps decode steps, each running the two-tier decode
    of every layer.  Then the same kernel over an uncompressed cache of
    w.full_ctx prefilled tokens (k = 0, a ring that never wraps), timed for
    a few steps.  Inputs are drawn on the device (see workloads)."""
    import torch
    from paper_2609_25537_amd import cmc
    from paper_2609_25537_amd import workloads as wl
    steps = args.decode_steps or w.steps
    P = min(steps, args.step_pool or 16)
    gb = 1e9
    torch.cuda.reset_peak_memory_stats()
    keys = wl.device_normal(w.seed, "sel_keys", (0,), (w.B, w.N, w.D), 1.0, dev, torch.float32)
    qv = wl.device_normal(w.seed, "q_vec", (0,), (w.B, w.D), 1.0, dev, torch.float32)
    idx = torch.empty((w.B, w.k), dtype=torch.int32, device=dev)
    sel_ws = torch.empty(max(1, cmc.cmc_select_workspace_bytes(w.B, w.N)), dtype=torch.uint8, device=dev)
    layers = [StackLayer(w, l, P, dev) for l in range(w.layers)]
    out = torch.empty((w.B, w.Hq, w.Dh), dtype=torch.float32, device=dev)
    ws = cmc.decode_workspace(w.B, w.Hq, w.Hkv, w.Dh, w.k, w.W, dev)
    torch.cuda.synchronize()

    def step_fn(j):
        def f():
            for Ly in layers:
                cmc.cmc_decode_step(Ly.q[j], Ly.gk, Ly.gv, None, w.k, Ly.wk, Ly.wv, Ly.wc, Ly.nk[j], Ly.nv[j],
                                    w.scale, out=out, workspace=ws)
        return f

    def select_and_gather():
        cmc.cmc_select_cmes(keys, qv, w.k, idx_out=idx, workspace=sel_ws)
        for Ly in layers:
            cmc.cmc_gather_tier1(Ly.pk, Ly.pv, idx, w.k, out_k=Ly.gk, out_v=Ly.gv)

    select_and_gather()
    graphs = [capture(step_fn(j)) for j in range(P)]

    def one_pass():
        select_and_gather()
        for t in range(steps):
            graphs[t % P].replay()

    for _ in range(args.warmup):
        one_pass()
    st = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(st)
    for _ in range(args.steps):
        one_pass()
    e1.record(st)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    peak_two_tier = torch.cuda.max_memory_allocated() / gb

    # Average duration of one layer's decode launch (graph replay).  The
    # launches rotate over the layers, as a decode step does: one layer's
    # K/V (about 200 MB) fits in the 256 MB last-level cache, so repeating a
    # single layer would time cache hits rather than HBM.
    def launches():
        for r in range(args.launch_reps):
            Ly, j = layers[r % len(layers)], (r // len(layers)) % P
            cmc.cmc_decode_step(Ly.q[j], Ly.gk, Ly.gv, None, w.k, Ly.wk, Ly.wv, Ly.wc, Ly.nk[j], Ly.nv[j],
                                w.scale, out=out, workspace=ws)
    g = capture(launches)
    g.replay()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    st.synchronize()
    a.record(st)
    g.replay()
    b.record(st)
    b.synchronize()
    t_launch = a.elapsed_time(b) / args.launch_reps * 1e-3

    del graphs, g, layers, keys, qv, sel_ws, ws
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    torch.cuda.reset_peak_memory_stats()
    res = {"ms": ms, "steps": steps, "P": P, "t_launch": t_launch, "baseline": None,
           "footprint_GB": {"two_tier_peak_allocated": round(peak_two_tier, 2)}}
    if args.baseline_steps <= 0 or w.full_ctx <= 0:
        return res

    # Uncompressed baseline: the same decode kernel over every cached token.
    Wb = w.full_ctx + steps
    bf = torch.bfloat16 if w.kv_dtype == "bf16" else torch.float32
    base = []
    for l in range(w.layers):
        bk = torch.empty((w.B, w.Hkv, Wb, w.Dh), dtype=bf, device=dev)
        bv = torch.empty_like(bk)
        bk[:, :, :w.full_ctx] = wl.device_normal(w.seed, "full_k", (l,), (w.B, w.Hkv, w.full_ctx, w.Dh),
                                                 w.kv_std, dev, bf)
        bv[:, :, :w.full_ctx] = wl.device_normal(w.seed, "full_v", (l,), (w.B, w.Hkv, w.full_ctx, w.Dh),
                                                 w.kv_std, dev, bf)
        q = wl.device_normal(w.seed, "q", (l, 0), (w.B, w.Hq, w.Dh), w.kv_std, dev, torch.float32)
        nk = wl.device_normal(w.seed, "new_k", (l, 0), (w.B, w.Hkv, 1, w.Dh), w.kv_std, dev, bf)
        nv = wl.device_normal(w.seed, "new_v", (l, 0), (w.B, w.Hkv, 1, w.Dh), w.kv_std, dev, bf)
        base.append((bk, bv, torch.full((w.B,), w.full_ctx, dtype=torch.int32, device=dev), q, nk, nv))
    pool0 = torch.zeros((w.B, w.Hkv, 1, w.Dh), dtype=bf, device=dev)
    bws = cmc.decode_workspace(w.B, w.Hq, w.Hkv, w.Dh, 0, Wb, dev)
    torch.cuda.synchronize()

    def base_step():
        for bk, bv, bc, q, nk, nv in base:
            cmc.cmc_decode_step(q, pool0, pool0, None, 0, bk, bv, bc, nk, nv, w.scale, out=out, workspace=bws)

    base_step()
    torch.cuda.synchronize()
    e0.record(st)
    for _ in range(args.baseline_steps):
        base_step()
    e1.record(st)
    torch.cuda.synchronize()
    base_ms = e0.elapsed_time(e1) / args.baseline_steps
    peak_base = torch.cuda.max_memory_allocated() / gb
    # After the warm-up step the timed steps attend full_ctx + 2 ... keys; the
    # key count grows by one per step, so scale the measured per-step time by
    # the mean key count of a whole pass (full_ctx + 1 ... full_ctx + steps).
    keys_t = w.full_ctx + 2 + (args.baseline_steps - 1) / 2
    base_pass_ms = base_ms * steps * ((w.full_ctx + (steps + 1) / 2) / keys_t)
    del base, pool0, bws
    torch.cuda.empty_cache()

    kv_row = w.Dh * w.kv_bytes * 2
    analytic = {
        "two_tier_compact": w.layers * w.B * w.Hkv * (w.k + w.W) * kv_row / gb,
        "two_tier_resident_pool": w.layers * w.B * w.Hkv * (w.N + w.W) * kv_row / gb,
        "baseline_first_step": w.layers * w.B * w.Hkv * (w.full_ctx + 1) * kv_row / gb,
        "baseline_last_step": w.layers * w.B * w.Hkv * (w.full_ctx + steps) * kv_row / gb,
    }
    return {
        "ms": ms, "steps": steps, "P": P, "t_launch": t_launch,
        "baseline": {"ms_per_step": round(base_ms, 3), "steps_timed": args.baseline_steps,
                     "mean_keys_per_sequence_timed": keys_t,
                     "extrapolated_pass_ms": round(base_pass_ms, 1),
                     "tokens_per_s": round(w.B * steps / (base_pass_ms * 1e-3), 1)},
        "footprint_GB": {"two_tier_peak_allocated": round(peak_two_tier, 2),
                         "baseline_peak_allocated": round(peak_base, 2),
                         **{k: round(v, 2) for k, v in analytic.items()}},
    }


def main():
    args = parse()
    if args.pmc_summary:
        pmc_summary(args)
        return
    if args.gpus != 1:
        print(f"bench.py: the library runs on one GPU; --gpus {args.gpus} is not supported "
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
    if args.selection_only:
        w = wl.get(args.workload)
        if w.ragged or w.layers != 1:
            print("bench.py: --selection-only takes a uniform single-layer decode workload", file=sys.stderr)
            sys.exit(2)
        print(json.dumps(selection_leg(w.name, dev, reps=max(1, args.steps))), flush=True)
        return
    if args.workload in wl.DENOISE_WORKLOADS:
        return main_denoise(args, wl.DENOISE_WORKLOADS[args.workload], dev)
    if args.workload in wl.BRIDGE_WORKLOADS:
        if args.vendor_gemm_probe:
            return vendor_gemm_probe(wl.BRIDGE_WORKLOADS[args.workload], dev)
        return main_bridge(args, wl.BRIDGE_WORKLOADS[args.workload], dev)
    w = wl.get(args.workload)
    if w.layers != 1:
        return main_stack(args, w, dev)
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

    P_inputs = inp.P
    t_launch, counts = time_decode_launch(inp, args.launch_reps)
    nbytes = decode_bytes(w, counts)
    achieved = nbytes / t_launch / 1e9
    sel_ms = time_select(inp)
    stream = stream_read_probe(dev)
    traffic = recorded_traffic(w)
    roofline = {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                "kernel": "decode_kernel (cmc_decode_step)", "bytes_per_launch": round(nbytes),
                "rings_full": bool((counts >= w.W).all()),
                "launch_us": round(t_launch * 1e6, 3),
                "stream_read_GBs": stream, "frac_of_stream_read": round(achieved / stream, 4),
                # bytes touched between reuses below the 256 MB last-level cache: the figure is
                # cache-resident latency, not an HBM bandwidth claim
                "cache_resident": nbytes * w.layers < LLC_BYTES}

    batched = selection = None
    if args.batched == "on" or (args.batched == "auto" and w.name == "llama3_8b_layer"):
        del inp, graph
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        batched = [batched_leg("llama_stack32", dev), batched_leg("mistral7b_batch64_x8", dev)]
        selection = selection_leg("mistral7b_batch64", dev)

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
                   "kv_dtype": w.kv_dtype, "step_input_sets": P_inputs, "graph": not args.eager,
                   **({"ragged": {"ctx_tokens": [w.ctx_min, w.ctx_max], "ratio": w.ratio,
                                  "question_rows": [w.q_min, w.q_max]}} if w.ragged else {})},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "select_ms": round(sel_ms, 4),
        "attention_only": True,
    }
    if batched is not None:
        # the >= 70% HBM figures at the Llama/Mistral head geometry (Hq 32, Hkv 8, Dh 128): batched
        # launches whose bytes between reuses exceed the last-level cache
        line["batched"] = batched
        # the once-per-question selection of the Mistral-shaped batch (4.29 GB of fp32 keys), and the
        # same keys in bf16
        line["batched_selection"] = selection
    txt = json.dumps(line)
    print(txt, flush=True)
    if args.out:
        with open(args.out, "a") as f:
            f.write(txt + "\n")


def recorded_traffic(w):
    """HBM bytes per decode launch from the counter record, if it was taken
    on the current decode kernel code; else None."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    with open(TRAFFIC_FILE) as f:
        entry = json.load(f).get(w.name)
    if entry and entry.get("kernel_hash") == decode_kernel_hash():
        return entry.get("bytes_per_launch")
    return None


def time_select(inp, reps: int = 5) -> float:
    """Milliseconds of one selection + Tier-1 gather (once per question),
    reported apart from the decode steps it is amortised over."""
    import torch
    inp.select()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        inp.select()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def stream_read_probe(dev, mib: int = 2048, reps: int = 5) -> float:
    """A STREAM-like read measured in the same run: GB/s of torch's row sums
    over a 2 GiB fp32 tensor viewed as 4096-wide rows (of the torch reductions
    tried, the fastest reader; a reference point for the decode rate, not the
    product)."""
    import torch
    x = torch.ones(mib << 18, dtype=torch.float32, device=dev).view(-1, 4096)
    x.sum(1)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        x.sum(1)
    e1.record()
    torch.cuda.synchronize()
    gbs = x.numel() * 4 * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del x
    return round(gbs, 1)


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def denoise_bytes(w, n_tokens) -> int:
    """Algorithmic bytes of one cmc_denoise call: every embedding row of
    every sequence read once, the Eq. 3 byte written and read back, the kept
    positions written (4 bytes per position of the [B][n] list)."""
    tok = int(np.sum(n_tokens))
    return tok * w.H * w.elem_bytes + 2 * w.B * w.n + 4 * w.B * w.n


def denoise_cpu_baseline(w, n_tokens, budget_s: float):
    """The oracle on whole sequences until the budget is spent; tokens/s."""
    import oracle
    from paper_2609_25537_amd import workloads as wl
    orc = oracle.default()
    done_tok, t = 0, 0.0
    b = 0
    while b < w.B and (b < 1 or t < budget_s):
        e = wl.denoise_emb(w, b)[None]
        nt = n_tokens[b:b + 1]
        t0 = time.perf_counter()
        mc = orc.denoise_scores(e, w.g, nt)
        orc.denoise_select(mc, w.tau, w.keep_min_every, nt, w.chunk_tokens)
        t += time.perf_counter() - t0
        done_tok += int(nt[0])
        b += 1
    return {"value": done_tok / t, "unit": "tokens/s", "cores": orc.num_threads(), "kind": "oracle",
            "sample": f"{b} of {w.B} contexts ({done_tok} tokens, {t:.2f} s)"}


def main_denoise(args, w, dev):
    """Graph-based context denoising of a batch of contexts: one step is one
    cmc_denoise call (statistic + Eq. 3 + floor + compaction + chunk
    offsets) over all B contexts, inputs resident in HBM."""
    import torch
    from paper_2609_25537_amd import cmc
    from paper_2609_25537_amd import workloads as wl
    n_tokens = wl.denoise_tokens(w)
    emb = to_dev(wl.denoise_emb(w), dev)
    nt = to_dev(n_tokens, dev)
    kept_idx = torch.empty((w.B, w.n), dtype=torch.int32, device=dev)
    kept_count = torch.empty((w.B,), dtype=torch.int32, device=dev)
    nch = -(-w.n // w.chunk_tokens)
    chunk_offset = torch.empty((w.B, nch), dtype=torch.int32, device=dev)
    n_chunks = torch.empty((w.B,), dtype=torch.int32, device=dev)
    ws = torch.empty(max(1, cmc.cmc_denoise_workspace_bytes(w.B, w.n)), dtype=torch.uint8, device=dev)

    def call():
        cmc.cmc_denoise(emb, g=w.g, tau=w.tau, keep_min_every=w.keep_min_every, n_tokens=nt,
                        chunk_tokens=w.chunk_tokens, kept_idx=kept_idx, kept_count=kept_count,
                        chunk_offset=chunk_offset, n_chunks_out=n_chunks, workspace=ws)

    reps = max(1, args.launch_reps // 10)
    g = capture(lambda: [call() for _ in range(reps)])
    for _ in range(args.warmup):
        g.replay()
    st = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(st)
    for _ in range(args.steps):
        g.replay()
    e1.record(st)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    calls = args.steps * reps
    t_call = ms * 1e-3 / calls
    tok = int(n_tokens.sum())
    nbytes = denoise_bytes(w, n_tokens)
    achieved = nbytes / t_call / 1e9
    kept = int(kept_count.sum().item())
    cpu = None if args.no_cpu_baseline else denoise_cpu_baseline(w, n_tokens, args.cpu_seconds)
    line = {
        "metric": "denoised context tokens/s and achieved HBM GB/s (% of MI355X peak)",
        "value": round(tok * calls / (ms * 1e-3), 1), "unit": "tokens/s", "n_gpus": 1, "steps": calls,
        "warmup": args.warmup, "ms_per_step": round(ms / calls, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "n_max": w.n, "tokens": tok, "H": w.H, "g": w.g, "tau": w.tau,
                   "keep_min_every": w.keep_min_every, "chunk_tokens": w.chunk_tokens, "graph": True,
                   "retention": round(kept / tok, 4)},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                     "kernel": "denoise_gram_wg_kernel (bf16 embeddings; denoise_score_kernel for fp32) "
                               "+ denoise_select_kernel (one cmc_denoise call)",
                     "bytes_per_launch": nbytes, "launch_us": round(t_call * 1e6, 3)},
        "cpu_baseline": cpu,
    }
    txt = json.dumps(line)
    print(txt, flush=True)
    if args.out:
        with open(args.out, "a") as f:
            f.write(txt + "\n")


MFMA_BF16_PEAK_TFLOPS = 2500.0


def bridge_cpu_baseline(w, budget_s: float):
    """The fp64 oracle on rows of the workload until the budget is spent."""
    import oracle
    from paper_2609_25537_amd import workloads as wl
    orc = oracle.default()
    p = wl.bridge_params(w)
    done, t, r0 = 0, 0.0, 0
    while done < 16 or t < budget_s:
        rows = list(range(r0, min(r0 + 16, w.M)))
        h = wl.bridge_h(w, rows)
        t0 = time.perf_counter()
        orc.memory_bridge(h, p["w1"], p["b1"], p["w2"], p["b2"], p["gamma"], p["beta"], w.nu, w.eps)
        t += time.perf_counter() - t0
        done += len(rows)
        r0 = (r0 + 16) % w.M
        if done >= w.M:
            break
    return {"value": done / t, "unit": "CME rows/s", "cores": orc.num_threads(), "kind": "oracle",
            "sample": f"{done} of {w.M} rows ({t:.2f} s)"}


def vendor_gemm_probe(w, dev, reps: int = 20):
    """Reference point, not the product path: torch's bf16 addmm (bias added,
    no activation) on the MemoryBridge's two GEMM shapes, random operands,
    timed with HIP events over `reps` back-to-back calls."""
    import torch
    lines = []
    for (K, N) in [(w.Hc, w.F), (w.F, w.Hd)]:
        a = torch.randn(w.M, K, device=dev, dtype=torch.bfloat16)
        bt = torch.randn(N, K, device=dev, dtype=torch.bfloat16)
        bias = torch.randn(N, device=dev, dtype=torch.bfloat16)
        for _ in range(3):
            torch.addmm(bias, a, bt.t())
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            torch.addmm(bias, a, bt.t())
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        lines.append({"vendor_gemm": "torch.addmm bf16", "M": w.M, "K": K, "N": N, "ms": round(ms, 4),
                      "tflops": round(2.0 * w.M * K * N / (ms * 1e-3) / 1e12, 1)})
        del a, bt, bias
    for ln in lines:
        print(json.dumps(ln), flush=True)


def main_bridge(args, w, dev):
    """MemoryBridge projection of a batch of CME vectors: one step is one
    cmc_memory_bridge call (two MFMA GEMMs, LayerNorm, tanh, cap), inputs
    resident in HBM."""
    import torch
    from paper_2609_25537_amd import cmc
    from paper_2609_25537_amd import workloads as wl
    p = wl.bridge_params(w)
    h = to_dev(wl.bridge_h(w), dev)
    d = {k: to_dev(v, dev) for k, v in p.items()}
    out = torch.empty((w.M, w.Hd), dtype=torch.float32, device=dev)
    h_norms = torch.empty((w.M,), dtype=torch.float32, device=dev)  # the CME norms localization ranks
    ws = torch.empty(cmc.cmc_bridge_workspace_bytes(w.M, w.F), dtype=torch.uint8, device=dev)

    def call():
        cmc.cmc_memory_bridge(h, d["w1"], d["b1"], d["w2"], d["b2"], d["gamma"], d["beta"], w.nu, w.eps, out=out,
                              h_norms_out=h_norms, workspace=ws)

    reps = max(1, args.launch_reps // 50)
    g = capture(lambda: [call() for _ in range(reps)])
    for _ in range(args.warmup):
        g.replay()
    st = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(st)
    for _ in range(args.steps):
        g.replay()
    e1.record(st)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    calls = args.steps * reps
    t_call = ms * 1e-3 / calls
    flops = 2.0 * w.M * (w.Hc * w.F + w.F * w.Hd)
    achieved = flops / t_call / 1e12
    cpu = None if args.no_cpu_baseline else bridge_cpu_baseline(w, args.cpu_seconds)
    line = {
        "metric": "MemoryBridge CME rows/s and achieved TFLOP/s (% of MI355X dense bf16 MFMA peak)",
        "value": round(w.M * calls / (ms * 1e-3), 1), "unit": "CME rows/s", "n_gpus": 1, "steps": calls,
        "warmup": args.warmup, "ms_per_step": round(ms / calls, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.name, "M": w.M, "Hc": w.Hc, "F": w.F, "Hd": w.Hd, "nu": w.nu, "graph": True},
        "roofline": {"bound": "mfma", "achieved": round(achieved, 2), "peak": MFMA_BF16_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / MFMA_BF16_PEAK_TFLOPS, 4), "traffic": None,
                     "kernel": "cme_norm_kernel + gemm_nt_kernel x2 + bridge_norm_kernel (one cmc_memory_bridge "
                               "call, CME norms included)",
                     "flops_per_launch": flops, "launch_us": round(t_call * 1e6, 3)},
        "cpu_baseline": cpu,
    }
    txt = json.dumps(line)
    print(txt, flush=True)
    if args.out:
        with open(args.out, "a") as f:
            f.write(txt + "\n")


def main_stack(args, w, dev):
    r = run_stack(args, w, dev)
    steps = r["steps"]
    ms_per_pass = r["ms"] / args.steps
    value = w.B * steps * args.steps / (r["ms"] * 1e-3)
    nbytes = decode_bytes(w)
    achieved = nbytes / r["t_launch"] / 1e9
    stream = stream_read_probe(dev)
    line = {
        "metric": "two-tier decode tokens/s and achieved HBM GB/s (% of MI355X peak)",
        "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_pass, 3), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": w.kv_dtype, "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "Hq": w.Hq, "Hkv": w.Hkv, "Dh": w.Dh, "N": w.N, "D": w.D,
                   "k": w.k, "W": w.W, "decode_steps": steps, "layers": w.layers, "kv_dtype": w.kv_dtype,
                   "step_input_sets": r["P"], "graph": True, "full_ctx": w.full_ctx},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": recorded_traffic(w),
                     "kernel": "decode_kernel (cmc_decode_step), one layer, layers rotating", "bytes_per_launch": nbytes,
                     "launch_us": round(r["t_launch"] * 1e6, 3),
                     "stream_read_GBs": stream, "frac_of_stream_read": round(achieved / stream, 4),
                     "cache_resident": False},
        "uncompressed_baseline": r["baseline"],
        "speedup_vs_uncompressed": (round(r["baseline"]["extrapolated_pass_ms"] / ms_per_pass, 2)
                                    if r["baseline"] else None),
        "footprint_GB": r["footprint_GB"],
        "cpu_baseline": None,
    }
    txt = json.dumps(line)
    print(txt, flush=True)
    if args.out:
        with open(args.out, "a") as f:
            f.write(txt + "\n")


if __name__ == "__main__":
    main()
