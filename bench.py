#!/usr/bin/env python3
"""Benchmark: fused outlier-aware W4A16 decode matmul on one MI355X.

Workload (one "step"): the four Llama-3-8B decode linears (qkv 4096x6144,
o 4096x4096, gate+up 4096x28672, down 14336x4096), each at M = 1, 4, 8, 16,
INT4 group 128, 1 % uniform bf16 outliers, synthetic seeded inputs -- 16
fused matmuls per step.  Weights are held in R rotated copies per shape
(about 1 GiB in all) so no launch finds its weights in the 256 MB MALL.
Every launch is captured in a HIP graph and replayed, as a decode loop
would run them.

value = algorithmic bytes of the step / step time, in GB/s, where the bytes
of one matmul are INT4 codes + fp16 scales + INT4 zero-points + stored
Tile-COO bytes (padding included) + X + Y.

Prints ONE JSON line (the contract) and, with --details, a per-matmul table
to stderr.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "effective HBM GB/s (% of MI355X peak) and µs/matmul, M=1–16, 1% outliers"
HBM_PEAK_GBS = 8000.0
SHAPES = [("qkv", 4096, 6144), ("o", 4096, 4096), ("gate_up", 4096, 28672),
          ("down", 14336, 4096)]
MS = [1, 4, 8, 16]
FRAC = 0.01
COPY_CAL_BYTES = 256 << 20  # plain device copy used to calibrate FETCH_SIZE / WRITE_SIZE
# The headline step uses the library's default Tile-COO packing (by-bucket
# groups, one bucket per tile: the fewest padding slots).  The format of the
# paper's decoding kernel (by-column groups, 16 buckets per tile) is timed
# beside it.
PAPER_TILECOO = {"group_mode": 0, "buckets_per_tile": 16}
# streaming-read probe launch shapes (workgroups, waves per workgroup, 16-byte
# loads in flight per lane); the fastest one at each byte count is the ceiling
PROBE_CONFIGS = [(256, 8, 4), (512, 4, 4), (512, 8, 2), (1024, 4, 2), (1024, 4, 4),
                 (2048, 4, 2)]
TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "fused_llama3_8b_decode_traffic.md")
# bf16 GEMM comparator: candidates per weight layout and workspace limit
GEMM_CANDIDATES = 16
GEMM_WORKSPACE = 64 << 20


def kernel_name(fq, M, K, N, packing=None, flags=0):
    """Template instance of the fused kernel the library launches for (M, K, N),
    a Tile-COO packed with `packing` (default: the library default) and the
    switches `flags`."""
    packing = packing or {}
    c = fq.fq_launch_config(M, K, N, buckets_per_tile=packing.get("buckets_per_tile"),
                            group_mode=packing.get("group_mode"), flags=flags)
    mb = 1 if min(M, 32) <= 16 else 2
    mode = 0 if c["mapping"] == "gather" else 1
    sk = "true" if c["stream_k"] else "false"
    xs = c["x_stage_loads"]
    bk = "true" if c["bulk_scales"] else "false"
    dv = "true" if flags & fq.FQ_DENSE_VALU else "false"
    return (f"matmul_kernel<{mb}, {mode}, {c['strip_cols'] // 16}, true, true, "
            f"{c['dense_waves']}, {sk}, {c['outlier_waves']}, {xs}, {bk}, {dv}>")


def dominant_kernel(fq, cases):
    """The kernel instance that takes most of the step, and its cases."""
    groups = {}
    for c in cases:
        groups.setdefault(kernel_name(fq, c.M, c.K, c.N), []).append(c)
    # weigh each instance by the bytes it moves (the step is bandwidth-bound)
    name = max(groups, key=lambda k: sum(c.bytes for c in groups[k]))
    return name, groups[name]


def algorithmic_bytes(M, K, N, tilecoo_bytes):
    return (K * N // 2 + (K // 128) * N * 2 + (K // 128) * N // 2 + tilecoo_bytes
            + 2 * M * K + 2 * M * N)


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def warm_replays(torch, g, min_ms: float = 20.0, max_replays: int = 400):
    """Replays graph g until the GPU has been busy for at least min_ms: after
    host-side preparation (packing, captures) the first replays run slower
    until the clocks ramp up, and one replay is not enough to absorb that."""
    t0 = time.perf_counter()
    for i in range(max_replays):
        g.replay()
        if i % 2 == 1:
            torch.cuda.synchronize()
            if (time.perf_counter() - t0) * 1e3 >= min_ms:
                break
    torch.cuda.synchronize()


def capture_graph(torch, fn):
    """A HIP graph of fn's launches (captured on a side stream after one
    eager warm-up call)."""
    g = torch.cuda.CUDAGraph()
    st = torch.cuda.Stream()
    st.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(st):
        fn()
    torch.cuda.current_stream().wait_stream(st)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


def graph_us(torch, g, launches, reps):
    """Average duration per launch of a graph of `launches` launches, HIP
    events around `reps` warmed replays on the replay stream."""
    warm_replays(torch, g)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e3 / (reps * launches)


class StreamProbe:
    """The streaming-read ceiling at a byte count: libfqprobe's plain 16-byte
    read of the same number of bytes, over R rotated buffers (the rotation the
    matmul's own measurement uses), graph-replayed like the matmuls; the
    fastest of PROBE_CONFIGS."""

    def __init__(self, torch, dev, R):
        from paper_2608_15531_amd import probe
        self.torch, self.dev, self.R, self.probe = torch, dev, R, probe
        self.sink = torch.zeros(max(c[0] for c in PROBE_CONFIGS), dtype=torch.int32, device=dev)
        self.cache = {}

    def us(self, nbytes):
        nbytes = -(-nbytes // 16) * 16
        if nbytes in self.cache:
            return self.cache[nbytes]
        torch = self.torch
        bufs = [torch.empty(nbytes // 4, dtype=torch.int32, device=self.dev)
                for _ in range(self.R)]
        L = 4 * self.R
        best = None
        for wgs, waves, d in PROBE_CONFIGS:
            g = capture_graph(torch, lambda: [self.probe.fq_probe_stream_read(
                bufs[i % self.R], nbytes, wgs, waves, d, self.sink) for i in range(L)])
            t = graph_us(torch, g, L, max(2, 160 // L))
            if best is None or t < best[0]:
                best = (t, {"workgroups": wgs, "waves": waves, "loads_in_flight": d})
            del g
        del bufs
        self.cache[nbytes] = best
        return best


def bf16_dequant_weight(torch, Wq, scales, zeros, k, n, v, K, N, group=128):
    """bf16(dequant(W_Q) + W_O) [K][N] on the device: the dense bf16 weight the
    bf16 GEMM comparator reads in place of the INT4 codes and the outliers
    (codes: nibble k % 8 of word [k / 8][n]; zero-points: nibble n % 8 of word
    [g][n / 8]; outliers: int32 positions, bf16 bits)."""
    dev = Wq.device
    sh = torch.arange(0, 32, 4, device=dev, dtype=torch.int32)
    q = ((Wq.view(K // 8, 1, N) >> sh.view(1, 8, 1)) & 15).view(K // group, group, N)
    z = ((zeros.view(K // group, N // 8, 1) >> sh.view(1, 1, 8)) & 15).view(K // group, 1, N)
    w = ((q - z).float() * scales.float().view(K // group, 1, N)).view(K, N)
    vals = torch.from_numpy(v.view(np.int16).copy()).view(torch.bfloat16).to(dev).float()
    w.index_put_((torch.from_numpy(k.astype(np.int64)).to(dev),
                  torch.from_numpy(n.astype(np.int64)).to(dev)), vals, accumulate=True)
    return w.to(torch.bfloat16)


class GemmComparator:
    """The bf16 GEMM comparator (libfqgemm, include/fq_gemm_ref.h): hipBLASLt
    on a dense bf16 weight of the same K x N, fp32 accumulation, bf16 Y.  For
    each (M, K, N) every candidate hipBLASLt's heuristic offers (up to
    GEMM_CANDIDATES, in both weight layouts: [K][N] and the linear-layer
    [N][K]) is timed over rotated weight copies in the graph-replay harness,
    and the fastest is kept, after a check of its output against
    torch.matmul in fp32."""

    LAYOUTS = ("kn", "nk")

    def __init__(self, torch, dev, source=None, max_candidates=None):
        from paper_2608_15531_amd import gemm_ref
        self.torch, self.dev, self.g = torch, dev, gemm_ref
        self.source = gemm_ref.HEURISTIC if source is None else source
        self.max_c = max_candidates or GEMM_CANDIDATES
        self.ws = torch.empty(GEMM_WORKSPACE, dtype=torch.uint8, device=dev)

    def weights(self, K, N, copies, base=None):
        """Rotated weight copies per layout, {"kn": [...], "nk": [...]}, as
        flat bf16 tensors.  base: the [K][N] bf16 weight to copy (its
        transpose for [N][K]); without it, random values, one set of buffers
        read in either layout (a GEMM's time does not depend on the values)."""
        torch = self.torch
        if base is None:
            Ws = [torch.randn(K * N, device=self.dev, dtype=torch.bfloat16)
                  for _ in range(copies)]
            return {"kn": Ws, "nk": Ws}
        nk = base.t().contiguous().view(-1)
        return {"kn": [base.reshape(-1).clone() for _ in range(copies)],
                "nk": [nk.clone() for _ in range(copies)]}

    def _launches(self, x, Ws, y, layout, i):
        K, N = x.shape[1], y.shape[1]
        shape = (K, N) if layout == "kn" else (N, K)
        return lambda: [self.g.gemm(x, W.view(shape), y, layout, i, self.ws)
                        for W in Ws[layout]]

    def search(self, M, K, N, Ws, reps, x=None):
        """Times every candidate; returns a dict with the fastest one's
        per-launch us, layout, kernel name and check, the number timed and
        the us of hipBLASLt's own first choice in the [K][N] layout.
        x: the bf16 activations [M][K] (default: random)."""
        torch, g = self.torch, self.g
        if x is None:
            x = torch.randn(M, K, device=self.dev, dtype=torch.bfloat16)
        y = torch.empty(M, N, device=self.dev, dtype=torch.bfloat16)
        timed = []
        for layout in self.LAYOUTS:
            n = g.prepare(M, K, N, layout, self.source, self.max_c, GEMM_WORKSPACE)
            for i in range(n):
                _, name = g.candidate(M, K, N, layout, i)
                gr = capture_graph(torch, self._launches(x, Ws, y, layout, i))
                for _ in range(2):
                    gr.replay()
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record()
                for _ in range(4):
                    gr.replay()
                e1.record()
                torch.cuda.synchronize()
                timed.append((e0.elapsed_time(e1) * 1e3 / (4 * len(Ws[layout])), layout, i, name))
                del gr
        first = next(t for t in timed if t[1] == "kn" and t[2] == 0)
        _, layout, i, name = min(timed)
        gr = capture_graph(torch, self._launches(x, Ws, y, layout, i))
        us = graph_us(torch, gr, len(Ws[layout]), reps)
        del gr
        # the kept candidate computes the product: Y against fp32 torch.matmul
        W0 = Ws[layout][0].view((K, N) if layout == "kn" else (N, K))
        g.gemm(x, W0, y, layout, i, self.ws)
        ref = x.float() @ (W0.float() if layout == "kn" else W0.float().t())
        # bf16 rounding of Y plus fp32 accumulation in any order
        mag = x.float().abs() @ (W0.float().abs() if layout == "kn" else W0.float().abs().t())
        err = (y.float() - ref).abs() - (2.0 ** -8 * ref.abs() + 2.0 ** -14 * mag)
        if bool((err > 0).any()) or not bool(torch.isfinite(y).all()):
            raise RuntimeError(f"bf16 GEMM comparator {name} ({layout}) differs from torch.matmul")
        return {"us": us, "layout": layout, "index": i, "kernel": name, "candidates": len(timed),
                "heuristic_first_us": first[0], "heuristic_first_kernel": first[3]}


def cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def kernel_source_digest():
    """sha256 over the device sources; counter figures are tied to it."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2608_15531_amd", "csrc")
    for f in ("kernels.hip", "device.hpp", "internal.hpp"):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(kernel):
    """HBM bytes per dominant-kernel launch from the committed counter summary
    (FETCH_SIZE + WRITE_SIZE, each scaled by the copy-kernel calibration), or
    None when the summary is missing, covers another kernel instance or was
    taken on other kernel sources."""
    try:
        with open(TRAFFIC_PROFILE) as fh:
            for line in fh:
                if line.startswith("traffic_json:"):
                    rec = json.loads(line.split(":", 1)[1])
                    if (rec.get("kernel_sources_sha256") == kernel_source_digest()
                            and rec.get("kernel") == kernel):
                        return rec
    except OSError:
        pass
    return None


def pmc_summary(fetch_csv, write_csv, sq_csv, log_path):
    """Turn the rocprofv3 --pmc CSVs of a --pmc-pass run into the traffic
    summary (markdown on stdout, ending in the traffic_json line bench.py
    reads).  No GPU needed."""
    import csv
    meta = None
    with open(log_path) as fh:
        for line in fh:
            if line.startswith('{"pmc_pass"'):
                meta = json.loads(line)
    if meta is None:
        raise SystemExit(f"no pmc_pass line in {log_path}")
    kernel = meta["kernel"]
    narrow = meta.get("role") == "narrow"
    flag = "--pmc-pass-narrow" if narrow else "--pmc-pass"
    sfx = "_narrow" if narrow else ""
    dest = ("profiles/fused_llama3_8b_decode_narrow_traffic.md" if narrow
            else "profiles/fused_llama3_8b_decode_traffic.md")

    def read(path):
        rows = {}
        for r in csv.DictReader(open(path)):
            d = rows.setdefault(int(r["Dispatch_Id"]), {"name": r["Kernel_Name"]})
            d[r["Counter_Name"]] = d.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
        return [rows[k] for k in sorted(rows)]

    def is_dom(d):
        return d["name"].replace("void fqk::", "").split("(")[0].strip() == kernel

    def is_copy(d):
        return "copyBuffer" in d["name"]

    f, w = read(fetch_csv), read(write_csv)
    fd = [d["FETCH_SIZE"] for d in f if is_dom(d)]
    wd = [d["WRITE_SIZE"] for d in w if is_dom(d)]
    fc = [d["FETCH_SIZE"] for d in f if is_copy(d)]
    wc = [d["WRITE_SIZE"] for d in w if is_copy(d)]
    if not fd or not fc or len(fd) != len(wd):
        raise SystemExit("dominant kernel or copy kernel missing from the counter CSVs")
    cal = meta["copy_bytes"]
    ff, wf = cal / (fc[-1] * 1024), cal / (wc[-1] * 1024)
    fetch = sum(fd) / len(fd) * 1024 * ff
    write = sum(wd) / len(wd) * 1024 * wf
    alg = meta["algorithmic_bytes_per_launch"]
    cases = meta["pmc_pass"]
    title = ("narrow-strip kernel (qkv and o)" if narrow else "dominant kernel")
    out = [f"# Fused W4A16 outlier matmul, {title}: HBM traffic and SQ counters", "",
           "Commands (repo root, MI355X, ROCm 7.2; `export TMPDIR=/tmp` first), one counter "
           "pass each, then this summary (no GPU):", "",
           "    timeout -s KILL 150 rocprofv3 --pmc FETCH_SIZE --output-format csv -d "
           f"gpurun_out/pmc_fetch{sfx} -o run -- python3 -u bench.py {flag} "
           f"> gpurun_out/pmc_fetch{sfx}.log",
           "    timeout -s KILL 150 rocprofv3 --pmc WRITE_SIZE --output-format csv -d "
           f"gpurun_out/pmc_write{sfx} -o run -- python3 -u bench.py {flag}",
           "    timeout -s KILL 150 rocprofv3 --pmc SQ_WAVE_CYCLES SQ_BUSY_CYCLES "
           "SQ_ACTIVE_INST_VALU SQ_VALU_MFMA_BUSY_CYCLES SQ_LDS_BANK_CONFLICT SQ_ACTIVE_INST_LDS "
           f"SQ_INSTS_VALU SQ_WAVES GRBM_GUI_ACTIVE --output-format csv -d gpurun_out/pmc_sq{sfx} "
           f"-o run -- python3 -u bench.py {flag}",
           "    python bench.py --pmc-summary "
           f"gpurun_out/pmc_fetch{sfx}/run_counter_collection.csv "
           f"gpurun_out/pmc_write{sfx}/run_counter_collection.csv "
           f"gpurun_out/pmc_sq{sfx}/run_counter_collection.csv gpurun_out/pmc_fetch{sfx}.log "
           f"> {dest}", "",
           "(the .log file is the stdout of the first pass, which names the launches)", "",
           f"Kernel `{kernel}`: launches {', '.join(cases)} of the Llama-3-8B decode step, "
           f"each once per rotated weight copy ({meta['copies']} copies), then one plain device "
           f"copy of {cal} bytes that calibrates the counters.", "",
           "## Calibration", "",
           f"The copy kernel moves {cal} bytes each way: FETCH_SIZE read {fc[-1]:.2f} KiB, "
           f"WRITE_SIZE {wc[-1]:.2f} KiB, so the factors are fetch {ff:.4f} and write {wf:.4f}.",
           "", "## Traffic per launch (calibrated)", "", "| case | FETCH MB | WRITE MB |",
           "|---|---|---|"]
    n = len(cases)
    for i, c in enumerate(cases):
        fs = [fd[j] for j in range(i, len(fd), n)]
        ws_ = [wd[j] for j in range(i, len(wd), n)]
        out.append(f"| {c} | {sum(fs) / len(fs) * 1024 * ff / 1e6:.2f} | "
                   f"{sum(ws_) / len(ws_) * 1024 * wf / 1e6:.3f} |")
    out += ["", f"Mean over the {len(fd)} launches: fetch {fetch / 1e6:.2f} MB + write "
                f"{write / 1e6:.3f} MB = {(fetch + write) / 1e6:.2f} MB per launch, against "
                f"{alg / 1e6:.2f} MB of algorithmic bytes per launch ({(fetch + write) / alg:.3f}x)."]
    if sq_csv:
        q = [d for d in read(sq_csv) if is_dom(d)]
        tot = {}
        for d in q:
            for k, v in d.items():
                if k != "name":
                    tot[k] = tot.get(k, 0.0) + v
        out += ["", "## SQ counters (sums over the same launches)", "", "| counter | value |",
                "|---|---|"]
        out += [f"| {k} | {v:.4g} |" for k, v in sorted(tot.items())]
        wc_ = tot.get("SQ_WAVE_CYCLES", 0.0)
        if wc_:
            ratios = []
            for k, lab in [("SQ_ACTIVE_INST_VALU", "VALU-active"), ("SQ_ACTIVE_INST_LDS", "LDS-active")]:
                if k in tot:
                    ratios.append(f"{lab} / wave cycles: {tot[k] / wc_:.3f}")
            if "SQ_LDS_BANK_CONFLICT" in tot and tot.get("SQ_ACTIVE_INST_LDS"):
                ratios.append("LDS bank-conflict cycles / LDS-active cycles: "
                              f"{tot['SQ_LDS_BANK_CONFLICT'] / tot['SQ_ACTIVE_INST_LDS']:.3f}")
            if "SQ_INSTS_VALU" in tot and tot.get("SQ_WAVES"):
                ratios.append(f"VALU instructions per wave: {tot['SQ_INSTS_VALU'] / tot['SQ_WAVES']:.0f}")
            out += ["", "; ".join(ratios) + "."]
    rec = {"kernel": kernel, "kernel_sources_sha256": kernel_source_digest(),
           "hbm_bytes_per_launch": round(fetch + write), "fetch_bytes_per_launch": round(fetch),
           "write_bytes_per_launch": round(write), "algorithmic_bytes_per_launch": round(alg),
           "fetch_factor": round(ff, 5), "write_factor": round(wf, 5), "launches": len(fd)}
    if narrow:
        out += ["", "The same figures as a record (bench.py takes roofline.traffic from the "
                    "dominant kernel's summary only).", "", "traffic_json: " + json.dumps(rec)]
    else:
        out += ["", "bench.py reads the line below and reports `hbm_bytes_per_launch` as "
                    "roofline.traffic only while the kernel sources still hash to "
                    "`kernel_sources_sha256` and the dominant kernel is the same instance.", "",
                "traffic_json: " + json.dumps(rec)]
    print("\n".join(out))


def cpu_baseline(fq, col_fraction: float = 0.25, runs: int = 3):
    """The fp64 NumPy oracle as it stands, timed on the host cores this
    process may use (BLAS threads pinned to that count), wall-clock median of
    `runs` runs per case, on a bounded sample of the workloads: the small
    single matmul (4096 x 4096) at M = 1, 4, 8, 16, and the four Llama-3-8B
    decode linears at M = 1, each on its first `col_fraction` of the columns
    (a contiguous block; bytes counted for that block).  Also the oracle's
    own Tile-COO pack against the library's fq_pack_tile_coo on the 4096 x
    4096 outliers, same packing.  Tile-COO bytes are the library default
    packing's, as in the step."""
    import oracle
    from synth import make_problem, seed_for
    cores = len(os.sched_getaffinity(0))
    try:
        from threadpoolctl import threadpool_limits
        limiter = threadpool_limits(limits=cores)
    except Exception:  # pragma: no cover
        limiter = None

    def median_s(fn):
        ts = []
        for _ in range(runs):
            t0 = time.perf_counter()
            fn()
            ts.append(time.perf_counter() - t0)
        return float(np.median(ts))

    rows, t_total, b_total = [], 0.0, 0
    # the small single matmul at every row count of the decode sweep
    for mi, M in enumerate(MS):
        p = make_problem(M, 4096, 4096, frac=FRAC, seed=seed_for(0, 0, mi))
        host = fq.fq_pack_tile_coo(4096, 4096, p.k, p.n, p.v)
        nb = algorithmic_bytes(M, 4096, 4096, int(host.sizes.bytes))
        oracle.matmul(p.X, p.Wq, p.scales, p.zeros, 4096, 4096, 128, p.k, p.n, p.v)   # warm
        t = median_s(lambda: oracle.matmul(p.X, p.Wq, p.scales, p.zeros, 4096, 4096, 128,
                                           p.k, p.n, p.v))
        rows.append({"case": f"4096x4096 M={M}", "s": round(t, 3), "bytes": nb})
        t_total += t
        b_total += nb
    # the decode linears at M = 1, a contiguous block of columns each
    for si, (name, K, N) in enumerate(SHAPES):
        p = make_problem(1, K, N, frac=FRAC, seed=seed_for(1, si, 0))
        host = fq.fq_pack_tile_coo(K, N, p.k, p.n, p.v)
        ncols = max(64, int(N * col_fraction) // 64 * 64)
        cols = np.arange(ncols)
        nb = int(round(algorithmic_bytes(1, K, N, int(host.sizes.bytes)) * ncols / N))
        t = median_s(lambda: oracle.matmul(p.X, p.Wq, p.scales, p.zeros, K, N, 128, p.k, p.n,
                                           p.v, cols))
        rows.append({"case": f"{name} {K}x{N} M=1 columns [0,{ncols})", "s": round(t, 3),
                     "bytes": nb})
        t_total += t
        b_total += nb
    # Tile-COO pack: the oracle's against the library's, same outliers and packing
    p = make_problem(1, 4096, 4096, frac=FRAC, seed=seed_for(0, 0, 0))
    d = fq.fq_default_tilecoo_params()
    op = oracle.Params(buckets=d.buckets_per_tile, group_mode=d.group_mode, reorder=d.reorder)
    pack_oracle = median_s(lambda: oracle.pack_tile_coo(4096, 4096, p.k, p.n, p.v, op))
    pack_lib = median_s(lambda: fq.fq_pack_tile_coo(4096, 4096, p.k, p.n, p.v))
    if limiter is not None:
        limiter.restore_original_limits()
    return {"value": round(b_total / t_total / 1e9, 4), "unit": "GB/s", "cores": cores,
            "kind": "oracle", "cpu_model": cpu_model(),
            "sample": f"fp64 NumPy oracle, median of {runs} wall-clock runs each, BLAS threads "
                      f"pinned to the {cores} cores of os.sched_getaffinity: 4096x4096 at "
                      f"M=1,4,8,16 and the Llama-3-8B decode linears at M=1 on their first "
                      f"{col_fraction:.0%} of columns; {t_total:.1f} s of medians over "
                      f"{b_total / 1e6:.1f} MB of algorithmic bytes",
            "per_case": rows,
            "pack_4096x4096_s": {"oracle_pack_tile_coo": round(pack_oracle, 3),
                                 "library_fq_pack_tile_coo": round(pack_lib, 4)}}


def ablation(fq, torch, cases, order, ws, R, dev, capture_fn=None):
    """Per-matmul graph-replay times of the paper's ablation steps (Sec. 5.4)
    as this library implements them: the unfused two-kernel baseline; SD, the
    fused kernel on an unreordered Tile-COO; SD+RE, with the column and element
    reordering of Sec. 3.2.2 (the default configuration); SD+EW and SD+EW+RE,
    the same with extra outlier waves beside the dense waves of each
    workgroup (warp specialisation, FQ_SPARSE_WAVES); and the default with
    the Stream-K schedule.  Prints one JSON line."""
    from synth import make_problem, seed_for
    # The paper's format (by-column groups, 16 buckets per tile), where the
    # reordering has buckets to balance: without reordering, one per shape,
    # R copies; the reordered one is each case's tcs_paper.
    plain = {}
    for si, (name, K, N) in enumerate(SHAPES):
        p = make_problem(1, K, N, frac=FRAC, seed=seed_for(1, si, 0))
        prm = dict(PAPER_TILECOO, reorder=0)
        host = fq.fq_pack_tile_coo(K, N, p.k, p.n, p.v, prm)
        plain[name] = [fq.TileCOODevice(host, dev) for _ in range(R)]
    need_sk = max(fq.fq_workspace_bytes(c.M, c.K, c.N, flags=fq.FQ_SCHED_STREAM_K) for c in cases)
    need_ew = max(fq.fq_workspace_bytes(c.M, c.K, c.N, flags=fq.FQ_SPARSE_WAVES) for c in cases)
    ws_big = torch.zeros(max(need_sk, need_ew, ws.numel()), dtype=torch.uint8, device=dev)
    EW = fq.FQ_SPARSE_WAVES
    variants = {
        "unfused": lambda c, r: fq.fq_w4a16_outlier_matmul_unfused(
            c.X, *c.weights[r], c.tcs_paper[r], Y=c.Y, ws=ws),
        "SD": lambda c, r: fq.fq_w4a16_outlier_matmul(
            c.X, *c.weights[r], plain[c.name][r], Y=c.Y, ws=ws),
        "SD+RE": lambda c, r: fq.fq_w4a16_outlier_matmul(
            c.X, *c.weights[r], c.tcs_paper[r], Y=c.Y, ws=ws),
        "SD+EW": lambda c, r: fq.fq_w4a16_outlier_matmul(
            c.X, *c.weights[r], plain[c.name][r], Y=c.Y, ws=ws_big, flags=EW),
        "SD+EW+RE": lambda c, r: fq.fq_w4a16_outlier_matmul(
            c.X, *c.weights[r], c.tcs_paper[r], Y=c.Y, ws=ws_big, flags=EW),
        "SD+RE+StreamK": lambda c, r: fq.fq_w4a16_outlier_matmul(
            c.X, *c.weights[r], c.tcs_paper[r], Y=c.Y, ws=ws_big, flags=fq.FQ_SCHED_STREAM_K),
        "default": lambda c, r: fq.fq_w4a16_outlier_matmul(
            c.X, *c.weights[r], c.tcs[r], Y=c.Y, ws=ws),
    }

    def capture(fn):
        g = torch.cuda.CUDAGraph()
        st = torch.cuda.Stream()
        st.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(st):
            fn()
        torch.cuda.current_stream().wait_stream(st)
        torch.cuda.synchronize()
        with torch.cuda.graph(g):
            fn()
        torch.cuda.synchronize()
        return g

    L, reps = 4 * R, 5
    table = []
    for c in order:
        row = {"shape": c.name, "M": c.M}
        for vname, fn in variants.items():
            g = capture(lambda: [fn(c, i % R) for i in range(L)])
            warm_replays(torch, g)
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                g.replay()
            e1.record()
            torch.cuda.synchronize()
            row[vname] = round(e0.elapsed_time(e1) * 1e3 / (reps * L), 3)
        table.append(row)
        log(json.dumps(row))
    geo = {}
    for vname in variants:
        if vname == "unfused":
            continue
        r = np.array([t["unfused"] / t[vname] for t in table])
        geo[vname] = round(float(np.exp(np.log(r).mean())), 4)
    print(json.dumps({"ablation": "geometric-mean speedup over the unfused two-kernel baseline",
                      "workload": "Llama-3-8B decode linears at M=1,4,8,16, 1% uniform outliers; "
                                  "Tile-COO in the paper's format (by-column groups, 16 buckets "
                                  "per tile) except 'default' (the library default packing: "
                                  "by-bucket groups, one bucket per tile)",
                      "speedup": geo, "per_matmul_us": table}), flush=True)


MFMA_PEAK_TFLOPS = 2500.0   # MI355X dense bf16


def unfused_workspace_bytes(fq, M, K, N):
    """Workspace that serves the fused, unfused and dense-only entry points."""
    pr = fq._problem(M, K, N, 0, 0)
    need = fq.C.c_size_t(0)
    fq.load().fq_workspace_bytes_unfused(fq.C.byref(pr), fq.C.byref(need))
    return max(need.value, fq.fq_workspace_bytes(M, K, N))


def mfma_flops(fq, M, K, N):
    """FLOPs the matrix cores execute in one fused launch: per 16-row block and
    128 x (strip width) tile, 4 x NCB dense MFMAs, 4 row-sum MFMAs and, with
    the MFMA outlier mapping, 4 x NCB image MFMAs of 16 x 16 x 32."""
    c = fq.fq_launch_config(M, K, N)
    ncb = c["strip_cols"] // 16
    slabs = (M + 31) // 32
    mb = 1 if min(M, 32) <= 16 else 2
    per_tile = 4 * ncb + 4 + (4 * ncb if c["mapping"] == "mfma" else 0)
    return slabs * mb * (N // c["strip_cols"]) * (K // 128) * per_tile * 16 * 16 * 32 * 2


LARGE_M_CASES = [(4096, 14336, M) for M in (32, 64, 128)] + [(14336, 4096, M) for M in (32, 64, 128)]


def pmc_pass_large_m(fq, torch, dev, launches=4):
    """Eager fused launches of the larger-M cases, in a fixed order, for a
    rocprofv3 --pmc run of the MFMA counters (one JSON line names them)."""
    from synth import make_activations, make_problem, seed_for
    order = []
    for si, (K, N, M) in enumerate(LARGE_M_CASES):
        p = make_problem(1, K, N, frac=FRAC, seed=seed_for(4, si, 0))
        host = fq.fq_pack_tile_coo(K, N, p.k, p.n, p.v)
        Wq, s, z = fq.to_device(p, dev)[1:]
        tc = fq.TileCOODevice(host, dev)
        x = torch.from_numpy(make_activations(M, K, seed_for(4, si, 1)).view(np.int16).copy())
        x = x.view(torch.bfloat16).to(dev)
        for _ in range(launches):
            fq.fq_w4a16_outlier_matmul(x, Wq, s, z, tc)
        torch.cuda.synchronize()
        order.append({"K": K, "N": N, "M": M, "launches": launches,
                      "kernel": kernel_name(fq, M, K, N), "flops": mfma_flops(fq, M, K, N)})
    print(json.dumps({"pmc_large_m": order}), flush=True)


def pmc_summary_mfma(csv_path, log_path):
    """MFMA counters of a --pmc-pass-large-m run (MfmaUtil, MfmaFlopsBF16) as a
    markdown table.  No GPU needed."""
    import csv
    meta = None
    with open(log_path) as fh:
        for line in fh:
            if line.startswith('{"pmc_large_m"'):
                meta = json.loads(line)["pmc_large_m"]
    if meta is None:
        raise SystemExit(f"no pmc_large_m line in {log_path}")
    rows = {}
    for r in csv.DictReader(open(csv_path)):
        if "matmul_kernel" not in r["Kernel_Name"]:
            continue
        d = rows.setdefault(int(r["Dispatch_Id"]), {})
        d[r["Counter_Name"]] = d.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    disp = [rows[k] for k in sorted(rows)]
    if len(disp) != sum(c["launches"] for c in meta):
        raise SystemExit(f"{len(disp)} matmul dispatches in the CSV, expected "
                         f"{sum(c['launches'] for c in meta)}")
    out = ["| K x N | M | kernel | MfmaUtil % (counter) | MFMA bf16 FLOPs per launch (counter) | "
           "MFMA FLOPs per launch (model) |", "|---|---|---|---|---|---|"]
    i = 0
    for c in meta:
        ds = disp[i:i + c["launches"]]
        i += c["launches"]
        util = sum(d["MfmaUtil"] for d in ds) / len(ds)
        fl = sum(d["MfmaFlopsBF16"] for d in ds) / len(ds)
        out.append(f"| {c['K']}x{c['N']} | {c['M']} | `{c['kernel']}` | {util:.1f} | {fl:.4g} | "
                   f"{c['flops']:.4g} |")
    return out


def _json_lines(path, prefix):
    with open(path) as fh:
        return [json.loads(line) for line in fh if line.startswith(prefix)]


def trace_summary(stats_csv, traced_log, plain_log):
    """Markdown summary of the rocprofv3 kernel trace of the default step
    (stdout).  traced_log: stdout of the bench run under the profiler;
    plain_log: stdout of a default bench run of the same tree.  No GPU."""
    import csv
    import paper_2608_15531_amd as fq
    rows = list(csv.DictReader(open(stats_csv)))
    traced = _json_lines(traced_log, '{"metric"')[0]
    plain = _json_lines(plain_log, '{"metric"')[0]
    inst = {}
    for name, K, N in SHAPES:
        for M in MS:
            inst.setdefault(kernel_name(fq, M, K, N), []).append(f"{name}/M{M}")

    def short(n):
        return n.replace("void fqk::", "").split("(")[0].strip()

    dom_name = traced["roofline"]["kernel"]
    out = ["# Fused W4A16 outlier matmul, Llama-3-8B decode linears (M=1,4,8,16), "
           "kernel-trace summary", "",
           "Commands (repo root, MI355X, ROCm 7.2; `export TMPDIR=/tmp` first): the traced run, "
           "a default run, then this summary (no GPU):", "",
           "    rocprofv3 --kernel-trace --stats --output-format csv -d gpurun_out/prof_bench "
           "-o bench -- python3 -u bench.py --steps 200 --warmup 20 --no-cpu-baseline "
           "--no-compare > gpurun_out/prof_bench.log",
           "    python3 -u bench.py > gpurun_out/bench_full.log",
           "    python bench.py --trace-summary gpurun_out/prof_bench/bench_kernel_stats.csv "
           "gpurun_out/prof_bench.log gpurun_out/bench_full.log "
           "> profiles/fused_llama3_8b_decode_kernel_trace.md", "",
           "Workload: qkv 4096x6144, o 4096x4096, gate_up 4096x28672, down 14336x4096 at "
           "M=1,4,8,16; 1% uniform bf16 outliers, Tile-COO 128x64, the library default packing "
           "(by-bucket groups, one bucket per tile; the paper-format step of the same run, "
           "by-column groups with 16 buckets, is included in the counts); 8 rotated weight "
           "copies per shape (graph replay).", "",
           "`matmul_kernel<MB, MODE, NCB, DENSE, SPARSE, NW, SK, NWS, XR, BK, DV>`: MB 16-row "
           "blocks; MODE 0 = LDS-gather outlier mapping, 1 = MFMA image mapping; NCB 16-column "
           "MFMA blocks per strip (2: 32-column strips, 4: 64-column strips); NW waves per "
           "workgroup; SK Stream-K; NWS extra outlier-only waves; XR row-wise X loads per tile "
           "reordered through LDS (ceil(M/4); 0 = loads in operand order); BK scales and "
           "zero-points loaded once per wave; DV dense products by VALU dot products "
           "(ablation).", "",
           f"Kernel sources sha256 (kernels.hip, device.hpp, internal.hpp): "
           f"`{kernel_source_digest()}`", "",
           "| kernel | launches (shapes, default packing) | calls | total ns | average ns | min ns "
           "| max ns |", "|---|---|---|---|---|---|---|"]
    tc = tn = 0
    for r in rows:
        k = short(r["Name"])
        if "matmul_kernel" in k:
            tc += int(r["Calls"])
            tn += int(r["TotalDurationNs"])
        out.append(f"| `{k}` | {', '.join(inst.get(k, []))} | {r['Calls']} | "
                   f"{r['TotalDurationNs']} | {float(r['AverageNs']):.0f} | {r['MinNs']} | "
                   f"{r['MaxNs']} |")
    dom = [r for r in rows if short(r["Name"]) == dom_name][0]
    rt, rp = traced["roofline"], plain["roofline"]
    if rp["traffic"]:
        tail = f", traffic {rp['traffic']}."
    else:
        rec = measured_traffic(dom_name)
        tail = (" (its roofline.traffic is null when the counter summary for these sources "
                "was not yet committed")
        if rec:
            tail += (f"; with it committed, bench.py reports roofline.traffic "
                     f"{rec['hbm_bytes_per_launch']} bytes per launch).")
        else:
            tail += ")."
    out += ["", f"Dominant kernel `{dom_name}` ({', '.join(rt['launches'])}: the instance that "
                f"moves most of the step's bytes): average {float(dom['AverageNs']) / 1e3:.2f} us "
                f"per launch (kernel execution only).",
            f"bench.py, same run: value {traced['value']} GB/s, ms_per_step "
            f"{traced['ms_per_step']}; roofline.us_per_launch {rt['us_per_launch']} us (HIP events "
            f"over warmed graph replays of each dominant matmul alone, 32 launches per graph, so "
            f"it also holds the dispatch gap between consecutive kernels, about 1.3 us), achieved "
            f"{rt['achieved']} GB/s, frac {rt['frac']}.",
            f"The default bench run without the profiler (same tree): value {plain['value']} GB/s, "
            f"ms_per_step {plain['ms_per_step']}, roofline.us_per_launch {rp['us_per_launch']} us, "
            f"frac {rp['frac']}" + tail,
            f"Every fused matmul launch of the run (warm-up replays included): {tc} calls, "
            f"{tn / tc / 1e3:.2f} us on average."]
    print("\n".join(out))


def ablation_summary(log_path):
    """Markdown summary of a --ablation run (stdout).  No GPU."""
    rec = _json_lines(log_path, '{"ablation"')[0]
    table = rec["per_matmul_us"]
    names = [k for k in table[0] if k not in ("shape", "M")]
    out = ["# Ablation of the fused kernel (Sec. 5.4 steps as this library implements them)", "",
           "Commands (repo root, MI355X, ROCm 7.2), the run, then this summary (no GPU):", "",
           "    python3 -u bench.py --ablation > gpurun_out/ablation.log",
           "    python bench.py --ablation-summary gpurun_out/ablation.log "
           "> profiles/ablation_llama3_8b_decode.md", "",
           f"Workload: {rec['workload']}; Tile-COO 128x64; "
           "graph replays over rotated weight copies, warmed for 20 ms, HIP events per launch.  "
           "unfused = dense W4A16 kernel then the Tile-COO SpMM kernel; SD = the fused kernel on "
           "a Tile-COO packed without reordering; RE = with the column and element reordering "
           "(the default packing); EW = extra outlier-only waves beside the dense waves "
           "(`FQ_SPARSE_WAVES`); StreamK = the Stream-K schedule (`FQ_SCHED_STREAM_K`).", "",
           "Geometric-mean speedup over the unfused baseline: " +
           ", ".join(f"{k} {v:.3f}x" for k, v in rec["speedup"].items()) + ".", "",
           "| shape | M | " + " | ".join(f"{n} us" for n in names) + " |",
           "|---|---|" + "---|" * len(names)]
    for t in table:
        out.append(f"| {t['shape']} | {t['M']} | " + " | ".join(f"{t[n]:.2f}" for n in names) + " |")
    print("\n".join(out))


def _gemm_cols(r):
    """The bf16 GEMM comparator's two table cells of a sweep record."""
    if "bf16_gemm_us" not in r:
        return "- | -"
    return f"{r['bf16_gemm_us']:.2f} ({r['bf16_gemm_layout']}) | {r['speedup_vs_bf16_gemm']:.2f}x"


def sweep_summary(density_log, b70_log, large_m_log, mfma_csv, mfma_log):
    """Markdown summary of the three sweeps and the MFMA counter pass
    (stdout).  No GPU."""
    sw = {k: _json_lines(p, '{"sweep"') for k, p in
          (("density", density_log), ("70b", b70_log), ("large-m", large_m_log))}
    out = ["# Sweeps beyond the decode step: density and structure, Llama-3-70B decode "
           "linears, larger M", "",
           "Commands (repo root, MI355X, ROCm 7.2): one run per table (every launch is "
           "graph-replayed over rotated weight copies, at least 4 and at least 1 GiB, warmed "
           "for 20 ms, HIP events per launch), the MFMA counter pass "
           "(`export TMPDIR=/tmp` first), then this summary (no GPU):", "",
           "    python bench.py --sweep density > gpurun_out/sweep_density.log",
           "    python bench.py --sweep 70b > gpurun_out/sweep_70b.log",
           "    python bench.py --sweep large-m > gpurun_out/sweep_large-m.log",
           "    timeout -s KILL 200 rocprofv3 --pmc MfmaUtil MfmaFlopsBF16 --output-format csv "
           "-d gpurun_out/pmc_mfma -o run -- python3 -u bench.py --pmc-pass-large-m "
           "> gpurun_out/pmc_mfma.log",
           "    python bench.py --sweep-summary gpurun_out/sweep_density.log "
           "gpurun_out/sweep_70b.log gpurun_out/sweep_large-m.log "
           "gpurun_out/pmc_mfma/run_counter_collection.csv gpurun_out/pmc_mfma.log "
           "> profiles/sweeps_density_70b_large_m.md", "",
           "Bytes are the algorithmic bytes of the operator (INT4 codes, fp16 scales, INT4 "
           "zeros, stored Tile-COO bytes, X, Y); `% peak` is against 8 TB/s.  MFMA columns "
           "(larger M): `alg TF` = (2MKN + 2M nnz) / t, `MFMA TF` = FLOPs the matrix cores "
           "execute (dense, row-sum and outlier-image MFMAs, padded rows included) / t, against "
           "the 2500 TFLOP/s dense bf16 peak.  Tile-COO: the library default packing (by-bucket "
           "groups, one bucket per tile).  `bf16 GEMM us` (70B and larger M): the bf16 GEMM "
           "comparator on bf16(dequant(W_Q) + W_O) and the same X (hipBLASLt through "
           "libfqgemm, fastest of its heuristic candidates in both weight layouts, over rotated "
           "bf16 copies); `fused vs bf16 GEMM` = its time / the fused time.", "",
           "## Density and structure (M=8, 4096x14336)", "",
           "| outliers | clustered share | Tile-COO MB | fused us | GB/s | % peak | unfused us | "
           "fused vs unfused | dense-only us | kernel |", "|---|---|---|---|---|---|---|---|---|---|"]
    for r in sw["density"]:
        out.append(f"| {100 * r['frac']:.1f}% {r['dist']} | {r.get('clustered_share', '-')} | "
                   f"{r['tilecoo_bytes'] / 1e6:.2f} | {r['fused_us']:.2f} | {r['fused_GBs']:.0f} | "
                   f"{r['pct_hbm_peak']} | {r['unfused_us']:.2f} | {r['fused_vs_unfused']:.2f}x | "
                   f"{r['dense_only_us']:.2f} | `{r['kernel']}` |")
    out += ["", "## Llama-3-70B decode linears (1% uniform)", "",
            "| K x N | M | fused us | GB/s | % peak | unfused us | fused vs unfused | "
            "dense-only us | bf16 GEMM us | fused vs bf16 GEMM | kernel |",
            "|---|---|---|---|---|---|---|---|---|---|---|"]
    for r in sw["70b"]:
        out.append(f"| {r['K']}x{r['N']} | {r['M']} | {r['fused_us']:.2f} | {r['fused_GBs']:.0f} | "
                   f"{r['pct_hbm_peak']} | {r['unfused_us']:.2f} | {r['fused_vs_unfused']:.2f}x | "
                   f"{r['dense_only_us']:.2f} | {_gemm_cols(r)} | `{r['kernel']}` |")
    out += ["", "Layer aggregate (the four Llama-3-70B linears of one decode layer: total "
                "algorithmic bytes / total fused time):", "",
            "| M | bytes | fused us | GB/s | % peak | unfused us | fused vs unfused |",
            "|---|---|---|---|---|---|---|"]
    for M in sorted({r["M"] for r in sw["70b"]}):
        rs = [r for r in sw["70b"] if r["M"] == M]
        b = sum(r["bytes"] for r in rs)
        t = sum(r["fused_us"] for r in rs)
        tu = sum(r["unfused_us"] for r in rs)
        out.append(f"| {M} | {b} | {t:.2f} | {b / t / 1e3:.0f} | "
                   f"{100 * b / t / 1e3 / HBM_PEAK_GBS:.1f} | {tu:.2f} | {tu / t:.2f}x |")
    out += ["", "## Larger M (1% uniform)", "",
            "| K x N | M | fused us | GB/s | % peak | alg TF | MFMA TF | MFMA % peak | unfused us "
            "| fused vs unfused | dense-only us | bf16 GEMM us | fused vs bf16 GEMM | kernel |",
            "|---|---|---|---|---|---|---|---|---|---|---|---|---|---|"]
    for r in sw["large-m"]:
        out.append(f"| {r['K']}x{r['N']} | {r['M']} | {r['fused_us']:.2f} | {r['fused_GBs']:.0f} | "
                   f"{r['pct_hbm_peak']} | {r['alg_TFLOPs']} | {r['mfma_TFLOPs']} | "
                   f"{r['mfma_util_pct']} | {r['unfused_us']:.2f} | {r['fused_vs_unfused']:.2f}x | "
                   f"{r['dense_only_us']:.2f} | {_gemm_cols(r)} | `{r['kernel']}` |")
    out += ["", "## MFMA counters (larger M)", "",
            "Four eager launches per case.  `MfmaUtil` is rocprofv3's derived metric (MFMA busy "
            "cycles summed over SIMDs / (GPU-active cycles x SIMDs)); `MfmaFlopsBF16` counts 512 "
            "x the bf16 MFMA math-op instructions.  The counted FLOPs equal the model that "
            "`bench.py --sweep large-m` divides by time for its `MFMA TF` column.", ""]
    out += pmc_summary_mfma(mfma_csv, mfma_log)
    out += ["", "At 5 % clustered the requested outliers do not fit into the 2 % of columns (they "
                "fill completely), so the realised clustered share is 40 %."]
    print("\n".join(out))


def sweep(fq, torch, which, dev, copies_min=4):
    """Per-matmul timings of the other workloads (not the step): the density
    and structure sweep, the Llama-3-70B decode layer, and the larger-M
    crossover with MFMA utilisation.  One JSON line per matmul."""
    from synth import make_activations, make_problem, seed_for
    if which == "density":
        cases = [(2, 0, 8, 4096, 14336, f, d) for d in ("uniform", "clustered")
                 for f in (0.0, 0.005, 0.01, 0.02, 0.05)]
    elif which == "70b":
        shapes = [("qkv70", 8192, 10240), ("o70", 8192, 8192), ("gate_up70", 8192, 57344),
                  ("down70", 28672, 8192)]
        cases = [(3, si, M, K, N, 0.01, "uniform") for si, (_, K, N) in enumerate(shapes)
                 for M in (1, 8, 16, 32)]
    else:
        cases = [(4, si, M, K, N, 0.01, "uniform")
                 for si, (K, N) in enumerate([(4096, 14336), (14336, 4096)])
                 for M in (32, 64, 128)]

    def capture(fn):
        g = torch.cuda.CUDAGraph()
        st = torch.cuda.Stream()
        st.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(st):
            fn()
        torch.cuda.current_stream().wait_stream(st)
        torch.cuda.synchronize()
        with torch.cuda.graph(g):
            fn()
        torch.cuda.synchronize()
        return g

    def per_launch_us(fn, L, reps=4):
        g = capture(lambda: [fn(i) for i in range(L)])
        warm_replays(torch, g)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / (reps * L)

    # the bf16 GEMM comparator beside the 70B and larger-M matmuls (the
    # paper's batch-size comparison with a vendor bf16 GEMM)
    comp = GemmComparator(torch, dev) if which in ("70b", "large-m") else None

    # weights per (shape, density, structure): enough rotated copies to pass 1 GiB
    weights = {}
    for cfg, si, M, K, N, frac, dist in cases:
        key = (K, N, frac, dist)
        if key in weights:
            continue
        weights.clear()
        torch.cuda.empty_cache()
        p = make_problem(1, K, N, frac=frac, dist=dist, seed=seed_for(cfg, si, 0) + int(frac * 1000))
        host = fq.fq_pack_tile_coo(K, N, p.k, p.n, p.v)
        R = max(copies_min, -(-(1 << 30) // (K * N // 2 + host.sizes.bytes)))
        weights[key] = ([fq.to_device(p, dev)[1:] for _ in range(R)],
                        [fq.TileCOODevice(host, dev) for _ in range(R)], host, p.meta)
        W, T, host, meta = weights[key]
        Wb = comp.weights(K, N, max(2, min(8, int(2.2e9 // (2 * K * N)))),
                          base=bf16_dequant_weight(torch, *W[0], p.k, p.n, p.v, K, N)) \
            if comp else None
        mis = {1: 0, 8: 1, 16: 2, 32: 3, 64: 1, 128: 2}
        for c2 in [c for c in cases if (c[3], c[4], c[5], c[6]) == key]:
            M2 = c2[2]
            xb = make_activations(M2, K, seed_for(cfg, si, mis.get(M2, 0)))
            x = torch.from_numpy(xb.view(np.int16).copy()).view(torch.bfloat16).to(dev)
            Y = torch.empty((M2, N), dtype=torch.bfloat16, device=dev)
            ws = torch.zeros(unfused_workspace_bytes(fq, M2, K, N), dtype=torch.uint8, device=dev)
            L = 4 * len(W)
            us = per_launch_us(lambda i: fq.fq_w4a16_outlier_matmul(
                x, *W[i % len(W)], T[i % len(W)], Y=Y, ws=ws), L)
            us_unf = per_launch_us(lambda i: fq.fq_w4a16_outlier_matmul_unfused(
                x, *W[i % len(W)], T[i % len(W)], Y=Y, ws=ws), L)
            us_dense = per_launch_us(lambda i: fq.fq_w4a16_matmul(
                x, *W[i % len(W)], Y=Y, ws=ws), L)
            nbytes = algorithmic_bytes(M2, K, N, int(host.sizes.bytes))
            nnz = int(host.sizes.nnz)
            rec = {"sweep": which, "K": K, "N": N, "M": M2, "frac": frac, "dist": dist,
                   "nnz": nnz, "tilecoo_bytes": int(host.sizes.bytes), "bytes": nbytes,
                   "kernel": kernel_name(fq, M2, K, N), "copies": len(W),
                   "fused_us": round(us, 3), "fused_GBs": round(nbytes / us / 1e3, 1),
                   "pct_hbm_peak": round(100 * nbytes / us / 1e3 / HBM_PEAK_GBS, 1),
                   "unfused_us": round(us_unf, 3), "dense_only_us": round(us_dense, 3),
                   "fused_vs_unfused": round(us_unf / us, 3)}
            if "realised_share" in meta:
                rec["clustered_share"] = round(meta["realised_share"], 3)
            if comp is not None:
                best = comp.search(M2, K, N, Wb, max(2, 160 // len(Wb["kn"])), x=x)
                rec.update(bf16_gemm_us=round(best["us"], 3), bf16_gemm_layout=best["layout"],
                           bf16_gemm_kernel=best["kernel"],
                           speedup_vs_bf16_gemm=round(best["us"] / us, 3))
            if which == "large-m":
                alg = 2 * M2 * K * N + 2 * M2 * nnz
                mf = mfma_flops(fq, M2, K, N)
                rec.update(alg_TFLOPs=round(alg / us / 1e6, 1),
                           mfma_TFLOPs=round(mf / us / 1e6, 1),
                           mfma_util_pct=round(100 * mf / us / 1e6 / MFMA_PEAK_TFLOPS, 2))
            print(json.dumps(rec), flush=True)
        del Wb


# Tile-COO packings compared for the element-reordering study (Sec. 3.2.2):
# (name, params) over the same outliers
PACKINGS = [
    ("bucket1_none", {"group_mode": 1, "buckets_per_tile": 1, "reorder": 0}),
    ("bucket1_columns", {"group_mode": 1, "buckets_per_tile": 1, "reorder": 1}),
    ("bucket1_re_k2_4", {"group_mode": 1, "buckets_per_tile": 1, "reorder": 3,
                         "elems_per_bank": 2, "n_bank_groups": 4}),
    ("bucket1_re_k1_4", {"group_mode": 1, "buckets_per_tile": 1, "reorder": 3,
                         "elems_per_bank": 1, "n_bank_groups": 4}),
    ("bucket1_re_k1_8", {"group_mode": 1, "buckets_per_tile": 1, "reorder": 3,
                         "elems_per_bank": 1, "n_bank_groups": 8}),
    ("bucket16_re_k2_4", {"group_mode": 1, "buckets_per_tile": 16, "reorder": 3,
                          "elems_per_bank": 2, "n_bank_groups": 4}),
    ("column16_none", {"group_mode": 0, "buckets_per_tile": 16, "reorder": 0}),
    ("column16_re_k2_4", {"group_mode": 0, "buckets_per_tile": 16, "reorder": 3,
                          "elems_per_bank": 2, "n_bank_groups": 4}),
]
PACKING_CASES = [("gate_up", 4096, 28672, 1), ("gate_up", 4096, 28672, 16), ("o", 4096, 4096, 1)]


def packing_pass(fq, torch, dev, timing: bool, R: int = 8):
    """The fused kernel on each Tile-COO packing of PACKINGS over the same
    outliers (PACKING_CASES).  timing: graph-replayed us per launch (JSON line
    per case); else eager launches, one per rotated copy, for a rocprofv3
    --pmc pass of the LDS counters (one JSON line names the sequence)."""
    from synth import make_activations, make_problem, seed_for
    si_of = {n: i for i, (n, _, _) in enumerate(SHAPES)}
    seq, rows = [], []
    for name, K, N, M in PACKING_CASES:
        p = make_problem(1, K, N, frac=FRAC, seed=seed_for(1, si_of[name], 0))
        W = [fq.to_device(p, dev)[1:] for _ in range(R)]
        x = torch.from_numpy(make_activations(M, K, seed_for(1, si_of[name], MS.index(M)))
                             .view(np.int16).copy()).view(torch.bfloat16).to(dev)
        Y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
        ws = torch.zeros(fq.fq_workspace_bytes(M, K, N), dtype=torch.uint8, device=dev)
        row = {"case": f"{name}/M{M}"}
        for pname, prm in PACKINGS:
            host = fq.fq_pack_tile_coo(K, N, p.k, p.n, p.v, prm)
            T = [fq.TileCOODevice(host, dev) for _ in range(R)]
            fn = lambda i: fq.fq_w4a16_outlier_matmul(x, *W[i % R], T[i % R], Y=Y, ws=ws)
            if timing:
                g = capture_graph(torch, lambda: [fn(i) for i in range(4 * R)])
                row[pname] = round(graph_us(torch, g, 4 * R, max(2, 160 // (4 * R))), 3)
                row[pname + "_groups"] = int(host.sizes.n_groups)
                del g
            else:
                for i in range(R):
                    fn(i)
                torch.cuda.synchronize()
                seq.append({"case": row["case"], "packing": pname, "launches": R,
                            "groups": int(host.sizes.n_groups)})
            del T
        if timing:
            print(json.dumps(row), flush=True)
            rows.append(row)
        del W
        torch.cuda.empty_cache()
    if not timing:
        print(json.dumps({"packing_pass": seq}), flush=True)


def packing_summary(csv_path, pass_log, timing_log):
    """Markdown on stdout: LDS bank-conflict counters and times of the fused
    kernel per Tile-COO packing (--packing-pass under rocprofv3 --pmc, and
    --packing-sweep).  No GPU."""
    import csv
    seq = _json_lines(pass_log, '{"packing_pass"')[0]["packing_pass"]
    times = {r["case"]: r for r in _json_lines(timing_log, '{"case"')}
    disp = {}
    for r in csv.DictReader(open(csv_path)):
        if "matmul_kernel" not in r["Kernel_Name"]:
            continue
        d = disp.setdefault(int(r["Dispatch_Id"]), {})
        d[r["Counter_Name"]] = d.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    ds = [disp[k] for k in sorted(disp)]
    need = sum(c["launches"] for c in seq)
    if len(ds) < need:
        raise SystemExit(f"{len(ds)} fused dispatches, expected {need}")
    ds = ds[len(ds) - need:]   # the warm-up launches of bench's main() come first
    out = ["# LDS bank conflicts of the outlier scatter against the Tile-COO packing "
           "(element reordering, Sec. 3.2.2)", "",
           "Commands (repo root, MI355X, ROCm 7.2; `export TMPDIR=/tmp` first), then this "
           "summary (no GPU):", "",
           "    timeout -s KILL 200 rocprofv3 --pmc SQ_LDS_BANK_CONFLICT SQ_ACTIVE_INST_LDS "
           "SQ_INSTS_LDS GRBM_GUI_ACTIVE --output-format csv -d gpurun_out/pmc_pack -o run -- "
           "python3 -u bench.py --packing-pass > gpurun_out/pmc_pack.log",
           "    python3 -u bench.py --packing-sweep > gpurun_out/packing_sweep.log",
           "    python bench.py --packing-summary gpurun_out/pmc_pack/run_counter_collection.csv "
           "gpurun_out/pmc_pack.log gpurun_out/packing_sweep.log "
           "> profiles/lds_bank_conflicts_packing.md", "",
           "The same 1 % uniform outliers packed eight ways; the fused kernel in its default "
           "launch plan (the MFMA outlier mapping: each lane writes the four values of one "
           "16-byte group into an LDS image of the tile's B operand, 2-byte stores, so the 64 "
           "lanes of one store hold the same slot of 64 different groups).  Counters per "
           "launch (mean of 8, one per rotated weight copy); time per launch from graph "
           "replays.  `re_kE_G`: element reordering with bank group (k / E) % G, rotated per "
           "bucket.", "",
           "| case | packing | groups | LDS instructions | LDS-active cycles | bank-conflict "
           "cycles | conflict / active | us per launch |",
           "|---|---|---|---|---|---|---|---|"]
    i = 0
    for c in seq:
        d = ds[i:i + c["launches"]]
        i += c["launches"]
        n = len(d)
        ins = sum(x.get("SQ_INSTS_LDS", 0) for x in d) / n
        act = sum(x.get("SQ_ACTIVE_INST_LDS", 0) for x in d) / n
        con = sum(x.get("SQ_LDS_BANK_CONFLICT", 0) for x in d) / n
        us = times.get(c["case"], {}).get(c["packing"])
        out.append(f"| {c['case']} | {c['packing']} | {c['groups']} | {ins:.4g} | {act:.4g} | "
                   f"{con:.4g} | {con / max(act, 1):.3f} | {us if us is not None else '-'} |")
    print("\n".join(out))


DENSE_PATH_COUNTERS = ("SQ_WAVE_CYCLES SQ_BUSY_CYCLES SQ_ACTIVE_INST_VALU SQ_VALU_MFMA_BUSY_CYCLES "
                       "SQ_INSTS_VALU SQ_WAVES GRBM_GUI_ACTIVE")


def dense_path_pass(fq, torch, dev, timing: bool, R: int = 8):
    """The dense path on MFMA (the default at every M) against the same kernel
    with FQ_DENSE_VALU (VALU bf16 dot products, a GEMV), at one row on the
    Llama-3-8B decode shapes: fused and dense-only.  timing: graph-replayed us
    per launch (JSON line per shape); else eager launches, one per rotated
    copy, for a rocprofv3 --pmc pass (one JSON line names the sequence)."""
    from synth import make_activations, make_problem, seed_for
    M = 1
    seq = []
    for si, (name, K, N) in enumerate(SHAPES):
        p = make_problem(1, K, N, frac=FRAC, seed=seed_for(1, si, 0))
        host = fq.fq_pack_tile_coo(K, N, p.k, p.n, p.v)
        W = [fq.to_device(p, dev)[1:] for _ in range(R)]
        T = [fq.TileCOODevice(host, dev) for _ in range(R)]
        x = torch.from_numpy(make_activations(M, K, seed_for(1, si, 0)).view(np.int16).copy())
        x = x.view(torch.bfloat16).to(dev)
        Y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
        ws = torch.zeros(fq.fq_workspace_bytes(M, K, N), dtype=torch.uint8, device=dev)
        row = {"case": f"{name}/M{M}", "bytes": algorithmic_bytes(M, K, N, host.sizes.bytes)}
        for variant, dense_only, flags in (("fused_mfma", False, 0),
                                           ("fused_valu", False, fq.FQ_DENSE_VALU),
                                           ("dense_mfma", True, 0),
                                           ("dense_valu", True, fq.FQ_DENSE_VALU)):
            if dense_only:
                fn = lambda i, f=flags: fq.fq_w4a16_matmul(x, *W[i % R], Y=Y, ws=ws, flags=f)
            else:
                fn = lambda i, f=flags: fq.fq_w4a16_outlier_matmul(x, *W[i % R], T[i % R], Y=Y,
                                                                    ws=ws, flags=f)
            if timing:
                g = capture_graph(torch, lambda: [fn(i) for i in range(4 * R)])
                row[variant] = round(graph_us(torch, g, 4 * R, max(2, 160 // (4 * R))), 3)
                del g
            else:
                for i in range(R):
                    fn(i)
                torch.cuda.synchronize()
                seq.append({"case": row["case"], "variant": variant, "launches": R})
        if timing:
            row["kernel_mfma"] = kernel_name(fq, M, K, N)
            row["kernel_valu"] = kernel_name(fq, M, K, N, flags=fq.FQ_DENSE_VALU)
            print(json.dumps(row), flush=True)
        del W, T
        torch.cuda.empty_cache()
    if not timing:
        print(json.dumps({"dense_path_pass": seq}), flush=True)


def dense_path_summary(csv_path, pass_log, timing_log):
    """Markdown on stdout: time and SQ counters of the dense path on MFMA
    against VALU dot products at one row (--dense-path-pass under rocprofv3
    --pmc, and --dense-path-sweep).  No GPU."""
    import csv
    seq = _json_lines(pass_log, '{"dense_path_pass"')[0]["dense_path_pass"]
    times = {r["case"]: r for r in _json_lines(timing_log, '{"case"')}
    disp = {}
    for r in csv.DictReader(open(csv_path)):
        if "matmul_kernel" not in r["Kernel_Name"]:
            continue
        d = disp.setdefault(int(r["Dispatch_Id"]), {})
        d[r["Counter_Name"]] = d.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    ds = [disp[k] for k in sorted(disp)]
    need = sum(c["launches"] for c in seq)
    if len(ds) < need:
        raise SystemExit(f"{len(ds)} matmul dispatches, expected {need}")
    ds = ds[len(ds) - need:]   # the warm-up launches of bench's main() come first
    out = ["# Dense path at one row: MFMA (the default) against VALU dot products (a GEMV)", "",
           "Commands (repo root, MI355X, ROCm 7.2; `export TMPDIR=/tmp` first), then this "
           "summary (no GPU):", "",
           f"    timeout -s KILL 200 rocprofv3 --pmc {DENSE_PATH_COUNTERS} --output-format csv "
           "-d gpurun_out/pmc_dense -o run -- python3 -u bench.py --dense-path-pass "
           "> gpurun_out/pmc_dense.log",
           "    python3 -u bench.py --dense-path-sweep > gpurun_out/dense_path_sweep.log",
           "    python bench.py --dense-path-summary gpurun_out/pmc_dense/run_counter_collection.csv "
           "gpurun_out/pmc_dense.log gpurun_out/dense_path_sweep.log "
           "> profiles/dense_path_mfma_vs_valu_m1.md", "",
           "The same kernel, loads, tiles and outlier path; only the dense products differ.  "
           "`mfma`: each lane's dequantised codes are the B operand of "
           "v_mfma_f32_16x16x32_bf16 (one MFMA per 16 columns and 32 k, plus one per 32 k for "
           "the row sums that remove the zero-points).  `valu` (FQ_DENSE_VALU): the same codes "
           "multiplied with the lane's X values by v_dot2_f32_bf16 (four per packed word), "
           "the lane's k-chunk sums added across lanes after the last tile.  One row (M = 1, "
           "where a GEMV does the least extra work), 1 % outliers in the default packing, "
           "rotated weight copies; time per launch from graph replays, counters per launch "
           "(mean of the 8 launches, one per copy).  VALU-active is a fraction of the summed "
           "wave cycles; MFMA-busy cycles are the counter's sum over the chip per launch "
           "(compare across rows, not against a peak).", "",
           "| case | variant | us per launch | GB/s | VALU instructions per wave | VALU-active / "
           "wave cycles | MFMA-busy cycles per launch | waves |",
           "|---|---|---|---|---|---|---|---|"]
    i = 0
    for c in seq:
        d = ds[i:i + c["launches"]]
        i += c["launches"]
        n = len(d)
        get = lambda k: sum(x.get(k, 0.0) for x in d) / n
        waves = get("SQ_WAVES")
        t = times.get(c["case"], {})
        us = t.get(c["variant"])
        gbs = f"{t['bytes'] / us / 1e3:.0f}" if us else "-"
        out.append(f"| {c['case']} | {c['variant']} | {us if us is not None else '-'} | {gbs} | "
                   f"{get('SQ_INSTS_VALU') / max(waves, 1):.0f} | "
                   f"{get('SQ_ACTIVE_INST_VALU') / max(get('SQ_WAVE_CYCLES'), 1):.3f} | "
                   f"{get('SQ_VALU_MFMA_BUSY_CYCLES'):.4g} | "
                   f"{waves:.0f} |")
    kern = {r["case"]: (r.get("kernel_mfma"), r.get("kernel_valu")) for r in times.values()}
    out += ["", "Kernel instances: " + "; ".join(f"{k}: `{a}` / `{b}`" for k, (a, b) in kern.items())]
    print("\n".join(out))


TILE_PROBE_SHAPES = [(4096, 28672), (14336, 4096)]
TILE_PROBE_GPT = 21   # groups per tile: the default packing's mean at 1 % outliers


def tile_load_probe(torch, dev, R: int = 4):
    """Markdown on stdout: the per-tile loads of the fused kernel without its
    compute (fq_probe_tile_loads), one kind of load added at a time, graph
    replays over R rotated buffers."""
    from paper_2608_15531_amd import probe
    P = probe
    variants = [("codes only", 0), ("+ scales, zero-points", P.FQ_PROBE_SCALES | P.FQ_PROBE_ZEROS),
                ("+ X", P.FQ_PROBE_X), ("+ groups", P.FQ_PROBE_GROUPS),
                ("+ X, groups", P.FQ_PROBE_X | P.FQ_PROBE_GROUPS),
                ("+ all four", P.FQ_PROBE_SCALES | P.FQ_PROBE_ZEROS | P.FQ_PROBE_X | P.FQ_PROBE_GROUPS),
                ("+ X, masked to 16 lanes", P.FQ_PROBE_X | P.FQ_PROBE_MASKED),
                ("+ groups, masked to 21 lanes", P.FQ_PROBE_GROUPS | P.FQ_PROBE_MASKED)]
    out = ["# Per-tile load cost: the fused kernel's loads without its compute", "",
           "Command (repo root, MI355X, ROCm 7.2):", "",
           "    python3 -u bench.py --tile-load-probe > profiles/tile_load_probe.md", "",
           "`fq_probe_tile_loads` (include/fq_probe.h) issues the loads of the fused kernel's "
           "tile loop on 64-column strips (four waves per strip, two 128-row tiles in flight per "
           "wave, four 16-byte code loads per lane and tile) and nothing else; each row adds one "
           "kind of per-tile load (scales 8 B, zero-point word 4 B, one 16-byte X load, one "
           f"16-byte Tile-COO group load with {TILE_PROBE_GPT} groups per tile).  Graph replays "
           f"over {R} rotated buffers; us per launch.  The added bytes are 3-10 % of the codes', "
           "so a plain bandwidth bound predicts almost no change.", "",
           "| K x N | loads per tile and lane | us per launch | vs codes only | code MB |",
           "|---|---|---|---|---|"]
    for K, N in TILE_PROBE_SHAPES:
        T = K // 128
        bufs = []
        for _ in range(R):
            bufs.append((torch.zeros(K * N // 8, dtype=torch.int32, device=dev),
                         torch.zeros(T * N, dtype=torch.int16, device=dev),
                         torch.zeros(T * N // 8, dtype=torch.int32, device=dev),
                         torch.zeros(K, dtype=torch.int16, device=dev),
                         torch.zeros(T * (N // 64) * TILE_PROBE_GPT * 4, dtype=torch.int32,
                                     device=dev)))
        sink = torch.zeros(N // 64, dtype=torch.int32, device=dev)
        base = None
        for label, extra in variants:
            L = 8 * R
            g = capture_graph(torch, lambda: [probe.fq_probe_tile_loads(
                *bufs[i % R], K, N, TILE_PROBE_GPT, extra, sink) for i in range(L)])
            us = min(graph_us(torch, g, L, 6), graph_us(torch, g, L, 6))
            del g
            base = us if base is None else base
            out.append(f"| {K}x{N} | {label} | {us:.2f} | {us - base:+.2f} | "
                       f"{K * N / 2 / 1e6:.1f} |")
        del bufs
        torch.cuda.empty_cache()
    print("\n".join(out))


STRIP_PROBE_CONFIGS = {   # (strip columns, waves, split) per shape; the plan's own is added
    "qkv": [(64, 4, 1), (64, 8, 2), (32, 8, 1), (32, 4, 2), (16, 8, 1), (16, 4, 1)],
    "o": [(64, 4, 4), (64, 8, 2), (32, 8, 1), (32, 4, 2), (16, 8, 1), (16, 4, 1)],
    "gate_up": [(64, 4, 1), (64, 8, 1), (32, 8, 1), (32, 4, 1), (16, 8, 1)],
    "down": [(64, 4, 8), (64, 8, 4), (32, 8, 2), (32, 4, 4), (16, 8, 1), (16, 4, 2)],
}


def strip_load_probe(fq, torch, dev, R: int = 8):
    """Markdown on stdout: the fused kernel's per-tile loads without its
    compute (fq_probe_strip_loads) for several strip widths, splits and wave
    counts on each decode shape, graph replays over R rotated buffers; the
    launch shape the library plans at M = 1 is marked."""
    from paper_2608_15531_amd import probe
    out = ["# Launch shapes by their loads alone: strip width, split and waves", "",
           "Command (repo root, MI355X, ROCm 7.2):", "",
           "    python3 -u bench.py --strip-load-probe > profiles/strip_load_probe.md", "",
           "`fq_probe_strip_loads` (include/fq_probe.h) issues the fused kernel's per-tile loads "
           "(four code loads of strip/4 bytes, one 16-byte X load and one 16-byte Tile-COO group "
           f"load per lane and tile, {TILE_PROBE_GPT} groups per tile; two tiles in flight per "
           "wave) and nothing else, for one (strip width, waves, split) launch shape at a time.  "
           f"Graph replays over {R} rotated buffers; us per launch.  `plan` marks the shape the "
           "library launches at M = 1 (its cross-workgroup reduction, when split > 1, is not "
           "part of the probe).", "",
           "| matmul | strip columns | waves | split | workgroups | us per launch | plan |",
           "|---|---|---|---|---|---|---|"]
    for name, K, N in SHAPES:
        T = K // 128
        cfg = fq.fq_launch_config(1, K, N)
        plan = (cfg["strip_cols"], cfg["dense_waves"], cfg["split_k"])
        shapes = list(STRIP_PROBE_CONFIGS[name])
        if plan not in shapes:
            shapes.insert(0, plan)
        codes = [torch.zeros(K * N // 8, dtype=torch.int32, device=dev) for _ in range(R)]
        groups = [torch.zeros(T * (N // 64) * TILE_PROBE_GPT * 4, dtype=torch.int32, device=dev)
                  for _ in range(R)]
        x = torch.zeros(K, dtype=torch.int16, device=dev)
        sink = torch.zeros(N, dtype=torch.int32, device=dev)
        for sc, nw, S in shapes:
            if T // S < nw or N // sc * S > N:
                continue
            L = 4 * R
            g = capture_graph(torch, lambda: [probe.fq_probe_strip_loads(
                codes[i % R], x, groups[i % R], K, N, sc, nw, S, TILE_PROBE_GPT, sink)
                for i in range(L)])
            us = min(graph_us(torch, g, L, 10), graph_us(torch, g, L, 10))
            del g
            out.append(f"| {name} | {sc} | {nw} | {S} | {N // sc * S} | {us:.2f} | "
                       f"{'yes' if (sc, nw, S) == plan else ''} |")
            log(out[-1])
        del codes, groups
        torch.cuda.empty_cache()
    print("\n".join(out))


def launch_timeline(torch, dev, R: int = 8):
    """Markdown on stdout: where a fused launch's time goes, per wave, from the
    instrumented build (libfq_stamps.so): each Llama-3-8B decode matmul in a
    graph of 4 R launches over R rotated weight copies, the last launch's
    stamps after replays, median of 5."""
    import paper_2608_15531_amd as fq
    from synth import make_activations, make_problem, seed_for
    fq.use_instrumented_build()
    out = ["# Launch timeline of the fused kernel (per-wave timestamps)", "",
           "Command (repo root, MI355X, ROCm 7.2):", "",
           "    python3 -u bench.py --launch-timeline > profiles/launch_timeline.md", "",
           "The instrumented build `libfq_stamps.so` (include/fq_debug.h: the same kernels with "
           "four `s_memrealtime` stamps per wave) runs each Llama-3-8B decode matmul (default "
           "packing, 1 % outliers) in a graph of 32 launches over 8 rotated weight copies; after "
           "warm replays the last launch's stamps are read.  Times in us from the first wave's "
           "start: `start` = when a wave began (median / max over waves), `first data` = from "
           "its start until its first tile's loads had arrived, `loop` = its tile loop, "
           "`epilogue` = from the loop's end to its exit (the workgroup barrier, the reduction "
           "across waves and, under split-K, across workgroups), `end` = its exit (median / max: "
           "the max is the kernel's span).  `launch` = HIP-event time per launch of the graph "
           "(the span plus the dispatch gap).  Medians over 5 replays.", "",
           "| matmul | waves | launch us | start med / max | first data | loop | epilogue "
           "(med / p90) | end med / max |", "|---|---|---|---|---|---|---|---|"]
    ws = torch.zeros(64 << 20, dtype=torch.uint8, device=dev)
    for si, (name, K, N) in enumerate(SHAPES):
        p = make_problem(1, K, N, frac=FRAC, seed=seed_for(1, si, 0))
        host = fq.fq_pack_tile_coo(K, N, p.k, p.n, p.v)
        W = [fq.to_device(p, dev)[1:] for _ in range(R)]
        T = [fq.TileCOODevice(host, dev) for _ in range(R)]
        for mi, M in enumerate(MS):
            x = torch.from_numpy(make_activations(M, K, seed_for(1, si, mi)).view(np.int16)
                                 .copy()).view(torch.bfloat16).to(dev)
            Y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
            c = fq.fq_launch_config(M, K, N)
            nw = c["workgroups"] * (c["dense_waves"] + c["outlier_waves"])
            L = 4 * R
            g = capture_graph(torch, lambda: [fq.fq_w4a16_outlier_matmul(
                x, *W[i % R], T[i % R], Y=Y, ws=ws) for i in range(L)])
            rows = []
            for _ in range(5):
                us = graph_us(torch, g, L, 2)
                st = fq.fq_debug_wave_stamps(nw).astype(np.int64)
                t0 = st[:, 0].min()
                start = (st[:, 0] - t0) / 100.0
                first = (st[:, 1] - st[:, 0]) / 100.0
                loop = (st[:, 2] - st[:, 1]) / 100.0
                epi = (st[:, 3] - st[:, 2]) / 100.0
                end = (st[:, 3] - t0) / 100.0
                rows.append([us, np.median(start), start.max(), np.median(first), np.median(loop),
                             np.median(epi), np.percentile(epi, 90), np.median(end), end.max()])
            del g
            m = np.median(np.array(rows), axis=0)
            out.append(f"| {name}/M{M} | {nw} | {m[0]:.2f} | {m[1]:.2f} / {m[2]:.2f} | "
                       f"{m[3]:.2f} | {m[4]:.2f} | {m[5]:.2f} / {m[6]:.2f} | "
                       f"{m[7]:.2f} / {m[8]:.2f} |")
        del W, T
        torch.cuda.empty_cache()
    print("\n".join(out))


def gemm_search_check(torch, dev, R: int = 8):
    """Markdown on stdout: for each decode shape at M = 1 and 16, the bf16
    GEMM comparator's fastest candidate from hipBLASLt's heuristic (the
    search bench.py uses) against the fastest of every algorithm the library
    holds that accepts the problem (both weight layouts each time)."""
    from paper_2608_15531_amd import gemm_ref
    out = ["# bf16 GEMM comparator: heuristic search against exhaustive search", "",
           "Command (repo root, MI355X, ROCm 7.2):", "",
           "    python3 -u bench.py --gemm-search-check", "",
           f"Each candidate: a graph of calls cycling over rotated bf16 weight copies (as in "
           f"bench.py's comparison), the fastest re-timed; heuristic: up to {GEMM_CANDIDATES} "
           "candidates per layout.  `first` is hipBLASLt's own first heuristic choice in the "
           "[K][N] layout.", "",
           "| matmul | search | candidates | best us | layout | best kernel (tile) | first us |",
           "|---|---|---|---|---|---|---|"]
    for name, K, N in SHAPES:
        copies = max(2, min(R, int(2.2e9 // (2 * K * N))))
        for M in (1, 16):
            for label, src, mc in (("heuristic", gemm_ref.HEURISTIC, GEMM_CANDIDATES),
                                   ("exhaustive", gemm_ref.EXHAUSTIVE, 4096)):
                comp = GemmComparator(torch, dev, source=src, max_candidates=mc)
                Ws = comp.weights(K, N, copies)
                b = comp.search(M, K, N, Ws, 40)
                tile = b["kernel"].split("_MT")[1].split("_")[0] if "_MT" in b["kernel"] else "?"
                first = f"{b['heuristic_first_us']:.3f}" if src == gemm_ref.HEURISTIC else "-"
                out.append(f"| {name}/M{M} | {label} | {b['candidates']} | {b['us']:.3f} | "
                           f"{b['layout']} | MT{tile} | {first} |")
                log(out[-1])
                del Ws, comp
                torch.cuda.empty_cache()
    print("\n".join(out))


def xcd_probe(torch, dev):
    """Markdown on stdout: the XCD each workgroup runs on, against workgroup
    index mod 8 (the placement the matmul kernels' workgroup dealing assumes
    for L2 sharing), over the grid sizes and workgroup sizes the kernels
    launch with; three launches each."""
    from paper_2608_15531_amd import probe
    out_lines = ["# Workgroup placement on the XCDs", "",
                 "Command (repo root, MI355X, ROCm 7.2):", "",
                 "    python3 -u bench.py --xcd-probe > profiles/xcd_placement.md", "",
                 "`fq_probe_workgroup_xcd` (include/fq_probe.h): each workgroup writes the XCC_ID "
                 "hardware register.  `round robin` = every workgroup w ran on XCD w mod 8.", "",
                 "| workgroups | threads | launch | round robin | workgroups per XCD |",
                 "|---|---|---|---|---|"]
    for n, th in ((128, 512), (192, 512), (256, 512), (384, 256), (448, 256), (512, 256),
                  (1024, 256), (4096, 64)):
        out = torch.full((n,), -1, dtype=torch.int32, device=dev)
        for rep in range(3):
            probe.fq_probe_workgroup_xcd(out, n, th)
            torch.cuda.synchronize()
            ids = out.cpu().numpy()
            rr = bool((ids == (np.arange(n) % 8)).all())
            hist = np.bincount(ids, minlength=8).tolist()
            out_lines.append(f"| {n} | {th} | {rep} | {'yes' if rr else 'no'} | {hist} |")
    print("\n".join(out_lines))


TRACE_WARM, TRACE_REPS = 2, 7   # replays per case in the kernel-trace pass
GEMM_TRACE_CALLS = 8            # eager comparator calls per case in that pass


def trace_pass(fq, torch, order, launch, R, dev):
    """For a rocprofv3 --kernel-trace run: each (shape, M) fused matmul alone,
    a graph of 4R launches over the rotated copies replayed a fixed number of
    times, in step order; then the bf16 GEMM comparator (hipBLASLt through
    libfqgemm, the candidate its search keeps; the search runs before the
    fused cases) of each shape at M = 1 and 16, GEMM_TRACE_CALLS eager calls
    each with a synchronisation between cases.  One JSON line names the
    sequence, so the trace splits per matmul (--trace-per-matmul)."""
    comp = GemmComparator(torch, dev)
    gemm, operands = [], []
    for name, K, N in SHAPES:
        # rotated weight copies as in the timed comparison, so that no call
        # finds its weight in the last-level cache; made now, so that only
        # the comparator's kernels run after the fused cases
        Ws = comp.weights(K, N, max(2, min(R, int(2.2e9 // (2 * K * N)))))
        for M in (1, 16):
            best = comp.search(M, K, N, Ws, 2)
            gemm.append({"case": f"{name}/M{M}", "M": M, "K": K, "N": N, "layout": best["layout"],
                         "kernel": best["kernel"], "index": best["index"],
                         "copies": len(Ws[best["layout"]]),
                         "bytes": 2 * K * N + 2 * M * K + 2 * M * N})
            shape = (K, N) if best["layout"] == "kn" else (N, K)
            operands.append(([W.view(shape) for W in Ws[best["layout"]]],
                             torch.randn(M, K, device=dev, dtype=torch.bfloat16),
                             torch.empty(M, N, device=dev, dtype=torch.bfloat16)))
        del Ws
    torch.cuda.synchronize()
    L = 4 * R
    seq = []
    for c in order:
        g = capture_graph(torch, lambda c=c: [launch(c, i % R, "fused") for i in range(L)])
        for _ in range(TRACE_WARM + TRACE_REPS):
            g.replay()
        torch.cuda.synchronize()
        seq.append({"case": f"{c.name}/M{c.M}", "kernel": kernel_name(fq, c.M, c.K, c.N),
                    "bytes": c.bytes, "launches": L * (1 + TRACE_WARM + TRACE_REPS),
                    "untimed": L * (1 + TRACE_WARM)})
        del g
    for e, (Ws, x, y) in zip(gemm, operands):
        # each (M, K, N) was prepared once, by its search: the index still holds
        for i in range(GEMM_TRACE_CALLS):
            comp.g.gemm(x, Ws[i % len(Ws)], y, e["layout"], e["index"], comp.ws)
        torch.cuda.synchronize()
    del operands
    # prelude: main() launches every case once eagerly before this pass
    print(json.dumps({"trace_pass": seq, "gemm": gemm, "gemm_calls": GEMM_TRACE_CALLS,
                      "prelude": len(order)}), flush=True)


def trace_pass_unfused(fq, torch, order, launch, R):
    """For a rocprofv3 --kernel-trace run: each (shape, M) case's fused graph
    and then its unfused graph (4R launches each, TRACE_WARM + TRACE_REPS
    replays), in step order.  One JSON line names the sequence, so the trace
    splits per case and variant (--trace-unfused-summary)."""
    L = 4 * R
    seq = []
    for c in order:
        for variant, per in (("fused", 1), ("unfused", 2)):
            g = capture_graph(torch, lambda c=c, v=variant: [launch(c, i % R, v) for i in range(L)])
            for _ in range(TRACE_WARM + TRACE_REPS):
                g.replay()
            torch.cuda.synchronize()
            seq.append({"case": f"{c.name}/M{c.M}", "variant": variant, "per_launch": per,
                        "dispatches": per * L * (1 + TRACE_WARM + TRACE_REPS),
                        "untimed": per * L * (1 + TRACE_WARM)})
            del g
    print(json.dumps({"trace_pass_unfused": seq, "prelude": len(order)}), flush=True)


def trace_unfused_summary(trace_csv, log_path):
    """Markdown on stdout: kernel-only durations of the unfused variant (its
    dense kernel and its Tile-COO SpMM kernel, and their sum per launch)
    beside the fused kernel's, from a --trace-pass-unfused run.  No GPU."""
    import csv
    meta = _json_lines(log_path, '{"trace_pass_unfused"')[0]
    rows = list(csv.DictReader(open(trace_csv)))
    ks = sorted((r for r in rows if "matmul_kernel" in r["Kernel_Name"]),
                key=lambda r: int(r["Start_Timestamp"]))[meta["prelude"]:]
    need = sum(c["dispatches"] for c in meta["trace_pass_unfused"])
    if len(ks) != need:
        raise SystemExit(f"{len(ks)} matmul dispatches in the trace, expected {need}")

    def dur(r):
        return (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3

    def short(n):
        return n.replace("void fqk::", "").split("(")[0].strip()
    res, i = {}, 0
    for c in meta["trace_pass_unfused"]:
        chunk = ks[i:i + c["dispatches"]][c["untimed"]:]
        i += c["dispatches"]
        if c["per_launch"] == 1:
            res.setdefault(c["case"], {})["fused"] = (float(np.median([dur(r) for r in chunk])),
                                                     short(chunk[0]["Kernel_Name"]))
        else:
            dense, spmm = chunk[0::2], chunk[1::2]
            names = ({short(r["Kernel_Name"]) for r in dense}, {short(r["Kernel_Name"]) for r in spmm})
            if len(names[0]) != 1 or len(names[1]) != 1:
                raise SystemExit(f"{c['case']}: unfused dispatches do not alternate: {names}")
            sums = [dur(a) + dur(b) for a, b in zip(dense, spmm)]
            res[c["case"]]["unfused"] = (float(np.median([dur(r) for r in dense])),
                                         float(np.median([dur(r) for r in spmm])),
                                         float(np.median(sums)), names[0].pop(), names[1].pop())
    L = meta["trace_pass_unfused"][0]["dispatches"] // (1 + TRACE_WARM + TRACE_REPS)
    out = ["# Unfused variant against the fused kernel: kernel-only durations per matmul "
           "(rocprofv3 kernel trace), Llama-3-8B decode linears", "",
           "Commands (repo root, MI355X, ROCm 7.2; `export TMPDIR=/tmp` first), then this "
           "summary (no GPU):", "",
           "    rocprofv3 --kernel-trace --output-format csv -d gpurun_out/trace_unf -o run -- "
           "python3 -u bench.py --trace-pass-unfused > gpurun_out/trace_unf.log",
           "    python bench.py --trace-unfused-summary gpurun_out/trace_unf/run_kernel_trace.csv "
           "gpurun_out/trace_unf.log > profiles/unfused_llama3_8b_decode_per_matmul.md", "",
           f"Each case: a graph of {L} launches of the fused kernel, then one of the unfused "
           f"variant (its dense kernel writes fp32 partial sums, its SpMM kernel re-reads X and "
           f"them and adds the outliers), each replayed {TRACE_REPS} times after {TRACE_WARM} "
           "warm-up replays and the capture's warm-up call (not counted), over the rotated "
           "weight copies.  `unfused sum` = median over launches of the two kernels' durations "
           "added; the benchmark's `unfused_us` is the event-timed pair (dispatch gaps "
           "included).  Kernel sources sha256 (kernels.hip, device.hpp, internal.hpp): "
           f"`{kernel_source_digest()}`", "",
           "| matmul | fused us | unfused dense us | unfused SpMM us | unfused sum us | "
           "unfused sum / fused |", "|---|---|---|---|---|---|"]
    for case, d in res.items():
        f = d["fused"][0]
        ud, us_, usum = d["unfused"][:3]
        out.append(f"| {case} | {f:.3f} | {ud:.3f} | {us_:.3f} | {usum:.3f} | {usum / f:.2f}x |")
    kinds = {}
    for d in res.values():
        kinds.setdefault("fused", set()).add(d["fused"][1])
        kinds.setdefault("unfused dense", set()).add(d["unfused"][3])
        kinds.setdefault("unfused SpMM", set()).add(d["unfused"][4])
    out += ["", "Kernel instances:", ""]
    for k, v in kinds.items():
        out.append(f"- {k}: " + ", ".join(f"`{n}`" for n in sorted(v)))
    print("\n".join(out))


def trace_per_matmul(trace_csv, log_path):
    """Markdown on stdout: rocprofv3 kernel-only durations of a --trace-pass
    run split per (shape, M), and the bf16 GEMM comparator's kernel names.
    The pass launches each case's graph (1 capture warm-up call plus
    TRACE_WARM + TRACE_REPS replays of 4R launches) in order, so the fused
    dispatches, sorted by start time, split into consecutive runs.  No GPU."""
    import csv
    meta = _json_lines(log_path, '{"trace_pass"')[0]
    rows = list(csv.DictReader(open(trace_csv)))
    fused = sorted((r for r in rows if "matmul_kernel" in r["Kernel_Name"]),
                   key=lambda r: int(r["Start_Timestamp"]))
    need = sum(c["launches"] for c in meta["trace_pass"])
    fused = fused[meta.get("prelude", 0):]
    if len(fused) != need:
        raise SystemExit(f"{len(fused)} fused dispatches in the trace, expected {need}")

    def short(n):
        return n.replace("void fqk::", "").split("(")[0].strip()
    out_rows, inst = [], {}
    i = 0
    for c in meta["trace_pass"]:
        chunk = fused[i:i + c["launches"]]
        i += c["launches"]
        names = {short(r["Kernel_Name"]) for r in chunk}
        if names != {c["kernel"]}:
            raise SystemExit(f"{c['case']}: kernels {names}, expected {c['kernel']}")
        ns = np.array([int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
                       for r in chunk[c["untimed"]:]], dtype=np.float64)
        med, mean = float(np.median(ns)) / 1e3, float(ns.mean()) / 1e3
        out_rows.append((c, med, mean, ns.size))
        inst.setdefault(c["kernel"], []).append((c, mean, ns.size))
    out = ["# Fused W4A16 outlier matmul, per-matmul kernel-only durations (rocprofv3 kernel "
           "trace), Llama-3-8B decode linears", "",
           "Commands (repo root, MI355X, ROCm 7.2; `export TMPDIR=/tmp` first), then this "
           "summary (no GPU):", "",
           "    rocprofv3 --kernel-trace --output-format csv -d gpurun_out/trace_pm -o run -- "
           "python3 -u bench.py --trace-pass > gpurun_out/trace_pm.log",
           "    python bench.py --trace-per-matmul gpurun_out/trace_pm/run_kernel_trace.csv "
           "gpurun_out/trace_pm.log > profiles/fused_llama3_8b_decode_per_matmul.md", "",
           f"Each case: a graph of {meta['trace_pass'][0]['launches'] // (1 + TRACE_WARM + TRACE_REPS)}"
           f" launches cycling over the rotated weight copies, {TRACE_REPS} timed replays after "
           f"{TRACE_WARM} warm-up replays and the capture's warm-up call (not counted).  "
           "Tile-COO: the library default packing (by-bucket groups, one bucket per tile).  "
           "`frac` = algorithmic bytes / median kernel duration / 8 TB/s.", "",
           f"Kernel sources sha256 (kernels.hip, device.hpp, internal.hpp): "
           f"`{kernel_source_digest()}`", "",
           "| matmul | kernel | launches | median us | mean us | bytes | GB/s (median) | frac |",
           "|---|---|---|---|---|---|---|---|"]
    for c, med, mean, n in out_rows:
        out.append(f"| {c['case']} | `{c['kernel']}` | {n} | {med:.3f} | {mean:.3f} | "
                   f"{c['bytes']} | {c['bytes'] / med / 1e3:.0f} | "
                   f"{c['bytes'] / med / 1e3 / HBM_PEAK_GBS:.3f} |")
    out += ["", "Per kernel instance (launch-weighted averages over its matmuls):", "",
            "| kernel | matmuls | mean us per launch | mean bytes per launch | frac |",
            "|---|---|---|---|---|"]
    for k, lst in inst.items():
        n = sum(x[2] for x in lst)
        t = sum(x[1] * x[2] for x in lst) / n
        b = sum(x[0]["bytes"] * x[2] for x in lst) / n
        out.append(f"| `{k}` | {', '.join(x[0]['case'] for x in lst)} | {t:.3f} | {b:.0f} | "
                   f"{b / t / 1e3 / HBM_PEAK_GBS:.3f} |")
    # the comparator's dispatches after the last fused one, in start order:
    # each case runs gemm_calls calls of its kept kernel; any other dispatch
    # (a library call may add a helper kernel) is counted with the case whose
    # calls it precedes or falls between
    last_fused = int(fused[-1]["End_Timestamp"])
    rest = sorted((r for r in rows if int(r["Start_Timestamp"]) > last_fused),
                  key=lambda r: int(r["Start_Timestamp"]))
    calls = meta["gemm_calls"]
    out += ["", "bf16 GEMM comparator: hipBLASLt through libfqgemm (include/fq_gemm_ref.h), the "
                "candidate its search kept (fastest of the heuristic candidates in the [K][N] and "
                f"[N][K] weight layouts), {calls} eager calls per case after the fused matmuls, "
                "cycling over rotated copies of a random bf16 weight of the same shape (a GEMM's "
                "time does not depend on the values) like the fused cases; kernel-only durations "
                "from the same trace.  Bytes: bf16 W, X and Y.", "",
            "| matmul | layout | kernel | calls | weight copies | median us | other dispatches | "
            "bytes | GB/s (median) |", "|---|---|---|---|---|---|---|---|---|"]
    j = 0
    for e in meta["gemm"]:
        own, others = [], 0
        while len(own) < calls and j < len(rest):
            r = rest[j]
            j += 1
            if r["Kernel_Name"].split("(")[0].strip() == e["kernel"]:
                own.append(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
            else:
                others += 1
        if len(own) < calls:
            raise SystemExit(f"{e['case']}: {len(own)} dispatches of {e['kernel']} in the trace, "
                             f"expected {calls}")
        med = float(np.median(own)) / 1e3
        out.append(f"| {e['case']} | {e['layout']} | `{e['kernel'][:110]}` | {calls} | "
                   f"{e['copies']} | {med:.3f} | {others} | {e['bytes']} | {e['bytes'] / med / 1e3:.0f} |")
    print("\n".join(out))


class Case:
    """One (shape, M) matmul with R rotated weight copies on the device."""

    def __init__(self, fq, torch, name, K, N, M, weights, tcs, x, dev, tcs_paper=None):
        self.name, self.K, self.N, self.M = name, K, N, M
        self.weights = weights            # list of (Wq, scales, zeros)
        self.tcs = tcs                    # list of TileCOODevice (library default packing)
        self.tcs_paper = tcs_paper        # the same outliers in the paper's format
        self.X = x
        self.Y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
        self.bytes = algorithmic_bytes(M, K, N, tcs[0].nbytes)
        self.bytes_paper = algorithmic_bytes(M, K, N, tcs_paper[0].nbytes) if tcs_paper else None


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--copies", type=int, default=8, help="rotated weight copies per shape")
    ap.add_argument("--variant", choices=["fused", "unfused", "dense"], default="fused",
                    help="what the timed step runs (fused is the reported number)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-compare", action="store_true",
                    help="skip the unfused / dense-only / hipBLASLt comparison table")
    ap.add_argument("--details", action="store_true", help="per-matmul table on stderr")
    ap.add_argument("--ablation", action="store_true",
                    help="no step timing: per-matmul times of the unfused baseline and of the "
                         "fused kernel with its techniques added one by one (SD: fused; EW: "
                         "outlier waves beside the dense waves; RE: Tile-COO reordering) and "
                         "with Stream-K; prints one JSON line of geometric-mean speedups")
    ap.add_argument("--pmc-pass", action="store_true",
                    help="no timing: eager launches of the dominant kernel's matmuls over the "
                         "rotated copies, then a plain copy of COPY_CAL_BYTES, for rocprofv3 "
                         "--pmc FETCH_SIZE / WRITE_SIZE collection")
    ap.add_argument("--tile-load-probe", action="store_true",
                    help="markdown: cost of each kind of per-tile load (fq_probe_tile_loads)")
    ap.add_argument("--launch-timeline", action="store_true",
                    help="markdown: per-wave launch timeline from the instrumented build")
    ap.add_argument("--strip-load-probe", action="store_true",
                    help="markdown: launch shapes (strip width, waves, split) compared by "
                         "the fused kernel's per-tile loads alone")
    ap.add_argument("--gemm-search-check", action="store_true",
                    help="markdown: the bf16 GEMM comparator's heuristic search against an "
                         "exhaustive one over every supported hipBLASLt algorithm")
    ap.add_argument("--xcd-probe", action="store_true",
                    help="markdown: the XCD each workgroup runs on, for the grid sizes the "
                         "kernels use")
    ap.add_argument("--pmc-pass-narrow", action="store_true",
                    help="as --pmc-pass, for the 32-column-strip instance of qkv and o at one row")
    ap.add_argument("--dense-path-pass", action="store_true",
                    help="eager launches of the dense path on MFMA and on VALU dot products "
                         "(FQ_DENSE_VALU) at one row, for a rocprofv3 --pmc pass")
    ap.add_argument("--dense-path-sweep", action="store_true",
                    help="graph-replayed times of the same comparison")
    ap.add_argument("--dense-path-summary", nargs=3, metavar=("CSV", "PASS_LOG", "SWEEP_LOG"),
                    help="no GPU: summarise --dense-path-pass counters and --dense-path-sweep times")
    ap.add_argument("--sweep", choices=["density", "70b", "large-m"],
                    help="no step timing: per-matmul timings of the density / structure "
                         "sweep (M=8, 4096x14336), the Llama-3-70B decode linears (M=1..32) "
                         "or the larger-M crossover (M=32..128, with MFMA utilisation)")
    ap.add_argument("--pmc-pass-large-m", action="store_true",
                    help="eager fused launches of the larger-M cases for a rocprofv3 --pmc "
                         "run of MfmaUtil / MfmaFlopsBF16")
    ap.add_argument("--pmc-summary-mfma", nargs=2, metavar=("CSV", "LOG"),
                    help="no GPU: summarise a --pmc-pass-large-m counter CSV")
    ap.add_argument("--pmc-summary", nargs=4, metavar=("FETCH_CSV", "WRITE_CSV", "SQ_CSV", "LOG"),
                    help="no GPU: summarise the rocprofv3 counter CSVs of --pmc-pass runs "
                         "(SQ_CSV may be '-') into the traffic profile text")
    ap.add_argument("--trace-summary", nargs=3, metavar=("STATS_CSV", "TRACED_LOG", "PLAIN_LOG"),
                    help="no GPU: the kernel-trace profile text from rocprofv3's kernel stats "
                         "and the bench output of the traced and of a plain run")
    ap.add_argument("--ablation-summary", metavar="LOG",
                    help="no GPU: the ablation profile text from the output of --ablation")
    ap.add_argument("--trace-pass", action="store_true",
                    help="no timing: each matmul's fused graph replayed a fixed number of "
                         "times, then the bf16 GEMM comparator, for a rocprofv3 --kernel-trace "
                         "run split per matmul by --trace-per-matmul")
    ap.add_argument("--trace-pass-unfused", action="store_true",
                    help="no timing: each matmul's fused and unfused graphs replayed a fixed "
                         "number of times, for a rocprofv3 --kernel-trace run summarised by "
                         "--trace-unfused-summary")
    ap.add_argument("--trace-unfused-summary", nargs=2, metavar=("KERNEL_TRACE_CSV", "LOG"),
                    help="no GPU: kernel-only durations of the unfused variant's two kernels "
                         "beside the fused kernel's, from a --trace-pass-unfused run")
    ap.add_argument("--trace-per-matmul", nargs=2, metavar=("KERNEL_TRACE_CSV", "LOG"),
                    help="no GPU: per-matmul kernel-only durations from a --trace-pass run's "
                         "kernel trace")
    ap.add_argument("--packing-pass", action="store_true",
                    help="eager fused launches per Tile-COO packing (element reordering "
                         "study) for a rocprofv3 --pmc pass of the LDS counters")
    ap.add_argument("--packing-sweep", action="store_true",
                    help="graph-replayed us per launch of the fused kernel per Tile-COO packing")
    ap.add_argument("--packing-summary", nargs=3, metavar=("CSV", "PASS_LOG", "SWEEP_LOG"),
                    help="no GPU: the LDS bank-conflict profile from --packing-pass and "
                         "--packing-sweep")
    ap.add_argument("--sweep-summary", nargs=5,
                    metavar=("DENSITY_LOG", "70B_LOG", "LARGE_M_LOG", "MFMA_CSV", "MFMA_LOG"),
                    help="no GPU: the sweeps profile text from the three --sweep outputs and "
                         "the --pmc-pass-large-m counter run")
    args = ap.parse_args()
    if args.trace_per_matmul:
        trace_per_matmul(*args.trace_per_matmul)
        return
    if args.trace_unfused_summary:
        trace_unfused_summary(*args.trace_unfused_summary)
        return
    if args.packing_summary:
        packing_summary(*args.packing_summary)
        return
    if args.dense_path_summary:
        dense_path_summary(*args.dense_path_summary)
        return
    if args.trace_summary:
        trace_summary(*args.trace_summary)
        return
    if args.sweep_summary:
        sweep_summary(*args.sweep_summary)
        return
    if args.ablation_summary:
        ablation_summary(args.ablation_summary)
        return
    if args.pmc_summary:
        fcsv, wcsv, sqcsv, logp = args.pmc_summary
        pmc_summary(fcsv, wcsv, None if sqcsv == "-" else sqcsv, logp)
        return
    if args.pmc_summary_mfma:
        print("\n".join(pmc_summary_mfma(*args.pmc_summary_mfma)))
        return

    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the operator shards along N without communication; see the design notes)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2608_15531_amd as fq
    from synth import make_activations, make_problem, seed_for

    if args.launch_timeline:
        launch_timeline(torch, torch.device("cuda:0"))
        return
    fq.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    R = args.copies
    if args.sweep:
        sweep(fq, torch, args.sweep, dev)
        return
    if args.pmc_pass_large_m:
        pmc_pass_large_m(fq, torch, dev)
        return
    if args.xcd_probe:
        xcd_probe(torch, dev)
        return
    if args.gemm_search_check:
        gemm_search_check(torch, dev)
        return
    if args.strip_load_probe:
        strip_load_probe(fq, torch, dev)
        return
    if args.tile_load_probe:
        tile_load_probe(torch, dev)
        return
    if args.dense_path_pass or args.dense_path_sweep:
        dense_path_pass(fq, torch, dev, timing=args.dense_path_sweep)
        return
    if args.packing_pass or args.packing_sweep:
        packing_pass(fq, torch, dev, timing=args.packing_sweep)
        return

    # ---------------------------------------------------------- inputs
    # torch.matmul, the bf16 GEMM comparator, on hipBLASLt (torch's "cublaslt"
    # backend on ROCm); the backend torch reports is recorded with the results
    torch.backends.cuda.preferred_blas_library("cublaslt")
    blas = str(torch.backends.cuda.preferred_blas_library())
    cases = []
    pack_s = {}
    bf16_w = {}   # the bf16 GEMM comparator's weight per shape
    for si, (name, K, N) in enumerate(SHAPES):
        t0 = time.perf_counter()
        p = make_problem(1, K, N, frac=FRAC, seed=seed_for(1, si, 0))
        t1 = time.perf_counter()
        host = fq.fq_pack_tile_coo(K, N, p.k, p.n, p.v)
        pack_s[name] = time.perf_counter() - t1
        host_p = fq.fq_pack_tile_coo(K, N, p.k, p.n, p.v, PAPER_TILECOO)
        weights, tcs, tcs_p = [], [], []
        for _ in range(R):
            weights.append(fq.to_device(p, dev)[1:])
            tcs.append(fq.TileCOODevice(host, dev))
            tcs_p.append(fq.TileCOODevice(host_p, dev))
        if not args.no_compare:
            bf16_w[name] = bf16_dequant_weight(torch, *weights[0], p.k, p.n, p.v, K, N)
        log(f"[setup] {name} K={K} N={N}: generate {t1 - t0:.1f}s, pack {pack_s[name]:.2f}s, "
            f"tilecoo {host.sizes.bytes / 1e6:.2f} MB (paper format "
            f"{host_p.sizes.bytes / 1e6:.2f} MB), {R} copies")
        for mi, M in enumerate(MS):
            xb = make_activations(M, K, seed_for(1, si, mi))
            x = torch.from_numpy(xb.view(np.int16).copy()).view(torch.bfloat16).to(dev)
            cases.append(Case(fq, torch, name, K, N, M, weights, tcs, x, dev, tcs_p))
        del p
    order = sorted(cases, key=lambda c: (c.M, [s[0] for s in SHAPES].index(c.name)))
    step_bytes = sum(c.bytes for c in order)

    max_ws = max(fq.fq_workspace_bytes(c.M, c.K, c.N) for c in cases)
    max_ws_unf = max(unfused_workspace_bytes(fq, c.M, c.K, c.N) for c in cases)
    ws = torch.zeros(max(max_ws, max_ws_unf), dtype=torch.uint8, device=dev)

    def launch(c, r, variant):
        Wq, s, z = c.weights[r]
        if variant == "fused":
            fq.fq_w4a16_outlier_matmul(c.X, Wq, s, z, c.tcs[r], Y=c.Y, ws=ws)
        elif variant == "fused_paper":
            fq.fq_w4a16_outlier_matmul(c.X, Wq, s, z, c.tcs_paper[r], Y=c.Y, ws=ws)
        elif variant == "unfused":
            fq.fq_w4a16_outlier_matmul_unfused(c.X, Wq, s, z, c.tcs[r], Y=c.Y, ws=ws)
        else:
            fq.fq_w4a16_matmul(c.X, Wq, s, z, Y=c.Y, ws=ws)

    # warm the code paths eagerly once (LDS attributes, allocator)
    for c in order:
        launch(c, 0, args.variant)
    torch.cuda.synchronize()

    if args.ablation:
        ablation(fq, torch, cases, order, ws, R, dev, capture_fn=None)
        return

    if args.pmc_pass or args.pmc_pass_narrow:
        # Each matmul of the dominant instance (or of the narrow-strip instance
        # of qkv and o at one row) once per weight copy, then the copy kernel
        # whose byte count calibrates the counters.
        if args.pmc_pass_narrow:
            qkv = next(c for c in order if c.name == "qkv" and c.M == 1)
            dom_name = kernel_name(fq, 1, qkv.K, qkv.N)
            dom = [c for c in order if kernel_name(fq, c.M, c.K, c.N) == dom_name]
        else:
            dom_name, dom = dominant_kernel(fq, order)
        for r in range(R):
            for c in dom:
                launch(c, r, "fused")
        torch.cuda.synchronize()
        src = torch.ones(COPY_CAL_BYTES, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"pmc_pass": [f"{c.name}/M{c.M}" for c in dom], "kernel": dom_name,
                          "role": "narrow" if args.pmc_pass_narrow else "dominant",
                          "copies": R,
                          "algorithmic_bytes_per_launch": sum(c.bytes for c in dom) / len(dom),
                          "copy_bytes": COPY_CAL_BYTES}), flush=True)
        return

    if args.trace_pass:
        trace_pass(fq, torch, order, launch, R, dev)
        return
    if args.trace_pass_unfused:
        trace_pass_unfused(fq, torch, order, launch, R)
        return

    def capture(fn):
        return capture_graph(torch, fn)

    # One graph per rotation slot: a whole step on weight copy r.
    graphs = [capture(lambda r=r: [launch(c, r, args.variant) for c in order])
              for r in range(R)]

    for i in range(args.warmup):
        graphs[i % R].replay()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record()
    for i in range(args.steps):
        graphs[i % R].replay()
    end.record()
    torch.cuda.synchronize()
    ms_step = start.elapsed_time(end) / args.steps
    value = step_bytes / (ms_step * 1e-3) / 1e9

    # The same step on the paper's Tile-COO format (by-column groups, 16
    # buckets per tile), reported beside the headline.
    paper_step = None
    if args.variant == "fused":
        graphs_p = [capture(lambda r=r: [launch(c, r, "fused_paper") for c in order])
                    for r in range(R)]
        for i in range(args.warmup):
            graphs_p[i % R].replay()
        torch.cuda.synchronize()
        start.record()
        for i in range(args.steps):
            graphs_p[i % R].replay()
        end.record()
        torch.cuda.synchronize()
        ms_p = start.elapsed_time(end) / args.steps
        bytes_p = sum(c.bytes_paper for c in order)
        paper_step = {"tilecoo": "by-column groups, 16 buckets per tile (the format of the "
                                 "paper's decoding kernel)",
                      "ms_per_step": round(ms_p, 5),
                      "value": round(bytes_p / (ms_p * 1e-3) / 1e9, 2),
                      "unit": "GB/s", "step_bytes": bytes_p,
                      "us_per_matmul": round(ms_p * 1e3 / len(order), 3),
                      "default_speedup": round(ms_p / ms_step, 3)}
        del graphs_p

    # --------------------------------------------- per-matmul durations
    # Each (shape, M) matmul alone: a graph of LPG launches cycling over the
    # copies, replayed; HIP events on the replay stream give the average
    # duration (the gap between two replays is spread over LPG launches).
    LPG = 4 * R

    def per_launch_us(c, variant, reps):
        g = capture(lambda: [launch(c, i % R, variant) for i in range(LPG)])
        return graph_us(torch, g, LPG, reps)

    reps = max(2, 160 // LPG)
    probe = StreamProbe(torch, dev, R)
    details = []
    for c in order:
        us = per_launch_us(c, "fused", reps)
        p_us, p_cfg = probe.us(c.bytes)
        d = {"shape": c.name, "M": c.M, "K": c.K, "N": c.N, "bytes": c.bytes,
             "tilecoo_bytes": c.tcs[0].nbytes, "tilecoo_min_bytes": 4 * int(c.tcs[0].sizes.nnz),
             "tilecoo_paper_format_bytes": c.tcs_paper[0].nbytes,
             "kernel": kernel_name(fq, c.M, c.K, c.N),
             "fused_us": round(us, 3), "fused_GBs": round(c.bytes / us / 1e3, 1),
             "pct_peak": round(100 * c.bytes / us / 1e3 / HBM_PEAK_GBS, 1),
             "probe_us": round(p_us, 3), "probe_GBs": round(c.bytes / p_us / 1e3, 1),
             "pct_of_probe": round(100 * p_us / us, 1), "probe_config": p_cfg}
        if not args.no_compare:
            d["unfused_us"] = round(per_launch_us(c, "unfused", reps), 3)
            d["dense_only_us"] = round(per_launch_us(c, "dense", reps), 3)
            d["fused_vs_unfused"] = round(d["unfused_us"] / us, 3)
            d["fused_vs_dense_only"] = round(us / d["dense_only_us"], 3)
        details.append(d)
    del probe

    if not args.no_compare:
        # bf16 GEMM comparator: hipBLASLt called directly (libfqgemm) on
        # bf16(dequant(W_Q) + W_O) and the same X, the fastest of its
        # heuristic candidates in both weight layouts; and torch.matmul on the
        # same operands for reference.
        comp = GemmComparator(torch, dev)
        for si, (name, K, N) in enumerate(SHAPES):
            copies = max(2, min(R, int(2.2e9 // (2 * K * N))))
            Ws = comp.weights(K, N, copies, base=bf16_w.pop(name))
            for d in details:
                if d["shape"] != name:
                    continue
                M = d["M"]
                x = next(c for c in order if c.name == name and c.M == M).X
                best = comp.search(M, K, N, Ws, reps, x=x)
                gemm_bytes = 2 * K * N + 2 * M * K + 2 * M * N   # bf16 W, X and Y
                d["bf16_gemm_us"] = round(best["us"], 3)
                d["bf16_gemm_GBs"] = round(gemm_bytes / best["us"] / 1e3, 1)
                d["bf16_gemm_kernel"] = best["kernel"]
                d["bf16_gemm_layout"] = best["layout"]
                d["bf16_gemm_candidates"] = best["candidates"]
                d["bf16_gemm_heuristic_first_us"] = round(best["heuristic_first_us"], 3)
                d["speedup_vs_bf16_gemm"] = round(best["us"] / d["fused_us"], 3)
                out = torch.empty(M, N, device=dev, dtype=torch.bfloat16)
                g = capture(lambda: [torch.matmul(x, W.view(K, N), out=out) for W in Ws["kn"]])
                d["torch_matmul_us"] = round(graph_us(torch, g, copies, reps), 3)
                del g
            del Ws
            torch.cuda.empty_cache()
        del comp

    # Dominant kernel: the fused kernel instance that moves most of the
    # step's bytes; the other launches are reported beside it.
    dom_name, dom_cases = dominant_kernel(fq, order)
    dom_keys = {(c.name, c.M) for c in dom_cases}

    def agg(sel):
        b = sum(d["bytes"] for d in details if sel(d))
        t = sum(d["fused_us"] for d in details if sel(d))
        n = sum(1 for d in details if sel(d))
        return b, t, n
    dom_b, dom_t, dom_n = agg(lambda d: (d["shape"], d["M"]) in dom_keys)
    oth_b, oth_t, _ = agg(lambda d: (d["shape"], d["M"]) not in dom_keys)
    traffic_rec = measured_traffic(dom_name)
    achieved = dom_b / (dom_t * 1e-6) / 1e9
    # layer aggregate: the four linears of one decode layer at each M
    layers = []
    for M in MS:
        b, t, _ = agg(lambda d, M=M: d["M"] == M)
        pt = sum(d["probe_us"] for d in details if d["M"] == M)
        layers.append({"M": M, "bytes": b, "fused_us": round(t, 3),
                       "GBs": round(b / t / 1e3, 1), "pct_peak": round(100 * b / t / 1e3 / HBM_PEAK_GBS, 1),
                       "pct_of_probe": round(100 * pt / t, 1)})
    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": "Llama-3-8B decode linears qkv 4096x6144, o 4096x4096, "
                        "gate_up 4096x28672, down 14336x4096 at M=1,4,8,16 (16 matmuls "
                        "per step); W_Q INT4 group 128 fp16 scales INT4 zeros; 1% uniform "
                        "bf16 outliers in Tile-COO 128x64 (library default packing: "
                        "by-bucket groups, 1 bucket per tile); bf16 Y",
            "variant": args.variant,
            "rotated_weight_copies": R,
            "pct_of_hbm_peak": round(100 * value / HBM_PEAK_GBS, 2),
            "us_per_matmul": round(ms_step * 1e3 / len(order), 3),
        },
        "roofline": {
            "bound": "hbm",
            "kernel": dom_name,
            "launches": sorted(f"{n}/M{m}" for n, m in dom_keys),
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": (traffic_rec or {}).get("hbm_bytes_per_launch"),
            "bytes_per_launch": round(dom_b / max(1, dom_n)),
            "us_per_launch": round(dom_t / max(1, dom_n), 3),
            "other_launches_GBs": round(oth_b / (oth_t * 1e-6) / 1e9, 1) if oth_t else None,
        },
        "layer_aggregate": layers,
        "tilecoo_paper_format": paper_step,
        "bf16_gemm_comparator": "hipBLASLt called directly (libfqgemm): bf16(dequant(W_Q) + "
                                "W_O) K x N weight and the same X, "
                                "fp32 accumulation, bf16 Y; fastest of up to "
                                f"{GEMM_CANDIDATES} heuristic candidates in each of the [K][N] "
                                "and [N][K] weight layouts; torch_matmul_us: torch.matmul "
                                f"on {blas}",
        "per_matmul": details,
        "pack_s": {k: round(v, 3) for k, v in pack_s.items()},
    }
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(fq)
    if args.details:
        for d in details:
            log(json.dumps(d))
    print(json.dumps(result), flush=True)

if __name__ == "__main__":
    main()
