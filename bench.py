#!/usr/bin/env python3
"""Benchmark: BITCOS ternary GEMV effective weight bandwidth on one MI355X.

A step is one batch-1 pass over a whole decode layer set (every GEMV of every
layer, inputs already resident in HBM), replayed from a HIP graph: W untimed
replays, then K timed ones, after a one-off 100 ms untimed warm-up that lifts
the GPU out of the idle clocks of the host-side packing.  Two device copies of
the set are replayed in turn, so a weight is re-read only after 2 x 411 MB of
other payload, more than twice the 256 MB Infinity Cache.  The
headline is the BitNet-2B-like set: 30 layers x {q, o 2560x2560; k, v
640x2560; gate, up 6912x2560; down 2560x6912}, z = 0.42 iid, one fp16 scale
per tensor, bf16 activations ~ N(0, 1) (the int8-quantised variant is reported
beside it).  value = sum of BITCOS payload bytes (bitmap + signs + scales) /
step time.  The same step over the five-trit and 2-bit layouts of the same
weights gives the same-GPU speedups.

--workload and --batch M select the other layer sets and M activation rows
per GEMV (BITCOS runs M > 1 in one launch per tile on its small-batch
kernel; the five-trit and 2-bit layouts have no such kernel and take M
batch-1 launches, as their entry points do).  A baseline with no kernel for
a set (bf16 activations on rows longer than 16384) is reported as null.

Prints ONE JSON line.  roofline: the dominant launch (the K = 2560 GEMVs of
the step, one persistent launch) timed alone, from a graph of ten back-to-back
launches; achieved = its
algorithmic bytes (payload + 2 K activation bytes + 4 N output bytes per GEMV)
per launch time, against the 8 TB/s HBM peak; traffic = its measured HBM
bytes (FETCH_SIZE + WRITE_SIZE scaled by a plain copy's counters, stored under
profiles/) while the kernel sources are unchanged; two_term: the launch's
time and its bytes at peak HBM bandwidth, both in CU-cycles per 32 weights
at the nominal 2.4 GHz, and which is larger.  sclk_mhz_under_load: the
shader clock rocm-smi reads while that launch replays (untimed, after the
timed runs).  cpu_baseline: the oracle's decode + dense GEMV on whole
layer-0 matrices on the host, about 12 s of work.
"""

from __future__ import annotations

import argparse
import concurrent.futures as cf
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import workloads as wl  # noqa: E402

HBM_PEAK_GBS = 8000.0
FMT_NAMES = {1: "bitcos", 2: "trit5", 3: "bit2"}
METRIC = "ternary GEMV effective weight GB/s (% of 8 TB/s HBM peak); speedup vs 5-trit"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=200)
    ap.add_argument("--workload", default="bitnet2b_layers")
    ap.add_argument("--batch", type=int, default=1,
                    help="activation rows per GEMV (1..16); BITCOS runs M > 1 on its small-batch kernel")
    ap.add_argument("--layers", type=int, default=0, help="0 = the workload's layer count")
    ap.add_argument("--copies", type=int, default=2,
                    help="device copies of the layer set, replayed in turn (2 x 411 MB > 2 x the 256 MB Infinity Cache)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-baselines", action="store_true", help="skip the five-trit / 2-bit steps")
    ap.add_argument("--threads", type=int, default=min(16, os.cpu_count() or 1))
    ap.add_argument("--profile-pass", action="store_true",
                    help="for counter runs: the dominant BITCOS launch x5, then a plain 256 MiB device copy x5")
    ap.add_argument("--sweep", action="store_true",
                    help="zero-density sweep on one 8192 x 8192 matrix: BITCOS vs five-trit vs 2-bit (own JSON line)")
    ap.add_argument("--gamma", action="store_true",
                    help="two-term roofline: cycles per 32 weights on cache-resident data vs z (own JSON line)")
    ap.add_argument("--sweep-copies", type=int, default=40,
                    help="device copies of each swept matrix streamed per launch (> 2 x the 256 MB Infinity Cache)")
    return ap.parse_args()


# Sources of the streaming BITCOS kernel: a stored HBM-traffic measurement is
# reported only while these files are unchanged.
KERNEL_SOURCES = ["bitcos_diag.h", "bitcos_fast.h", "bitcos_kernel.h", "mfma_common.h", "device_common.h", "batch.h",
                  "batch.hip", "gemv_bitcos.hip", "gemv_bitcos_d16.hip", "launch_common.h", "plan.h"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "bitcos_diag_bf16_bitnet2b_k2560_traffic.txt")
COPY_MIB = 256


def kernel_source_hash():
    import hashlib
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2609_16338_amd", "csrc", name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()[:16]


def stored_traffic():
    """HBM bytes per launch of the dominant kernel from the FETCH_SIZE / WRITE_SIZE
    passes (scaled by the copy calibration), or None if the kernel changed since."""
    try:
        with open(TRAFFIC_FILE) as f:
            kv = dict(line.split(":", 1) for line in f if ":" in line and not line.startswith("#"))
    except OSError:
        return None
    kv = {k.strip(): v.strip() for k, v in kv.items()}
    if kv.get("kernel_source_hash") != kernel_source_hash():
        return None
    try:
        return int(float(kv["traffic_bytes_per_launch"]))
    except (KeyError, ValueError):
        return None


def build_set(wk, layers, fmts, threads):
    """Pack every matrix of the layer set in every format (host), upload to HBM."""
    import torch

    from paper_2609_16338_amd import api

    jobs = [(l, mi, spec) for l in range(layers) for mi, spec in enumerate(wk.matrices)]

    def one(job):
        l, mi, spec = job
        w, sc = wl.matrix_inputs(wk.cid, l, mi, spec)
        out = {}
        for fmt in fmts:
            L, blob = api.plan_and_pack(fmt, w, sc, spec.group)
            out[fmt] = (L, blob)
        return job, out

    packed = {}
    with cf.ThreadPoolExecutor(max_workers=threads) as ex:
        for (l, mi, spec), out in ex.map(one, jobs):
            for fmt, (L, blob) in out.items():
                packed.setdefault(fmt, []).append((l, mi, spec, L, torch.from_numpy(blob).cuda()))
    return packed


def activations(wk, kinds, m=1):
    """Per distinct K: device activations [m, k] (bf16, and int8 + per-group
    scales via the library)."""
    import torch

    from paper_2609_16338_amd import api

    acts = {}
    for k in sorted({s.k for s in wk.matrices}):
        xb = wl.activation_inputs(wk.cid, "bf16", m, k)
        xbd = torch.from_numpy(xb.view(np.int16)).view(torch.bfloat16).cuda()
        acts[("bf16", k)] = (xbd, None)
        if "int8" in kinds:
            q = torch.empty((m, k), dtype=torch.int8, device="cuda")
            a = torch.empty((m, k // 128), dtype=torch.float32, device="cuda")
            api.quantize_activations(xbd, q, a)
            acts[("int8", k)] = (q, a)
    torch.cuda.synchronize()
    return acts


def supported(entries, kind, m=1):
    """Whether the library has a kernel for every GEMV of the step at m rows
    (formats without a small-batch kernel run m > 1 as m batch-1 launches)."""
    from paper_2609_16338_amd import _native as N
    from paper_2609_16338_amd import api

    xd = N.X_BF16 if kind == "bf16" else N.X_I8
    for e in entries:
        mm = m if e[3].format == N.FMT_BITCOS else 1
        try:
            api.describe(e[3], mm, xd)
        except N.BitcosError:
            return False
    return True


def make_batches(entries, acts, kind):
    """One persistent launch per tile: the step's GEMVs grouped by kernel tile.

    With m activation rows, BITCOS takes all m in one launch (small-batch
    kernel); the five-trit and 2-bit layouts, which have no small-batch
    kernel, take m batch-1 launches per tile, one per activation row, as
    their m > 1 entry points do."""
    import torch

    from paper_2609_16338_amd import _native as N
    from paper_2609_16338_amd import api

    xd = N.X_BF16 if kind == "bf16" else N.X_I8
    m = next(iter(acts.values()))[0].shape[0]
    rows_per_launch = m if entries[0][3].format == N.FMT_BITCOS else 1
    groups = {}
    for e in entries:
        info = api.describe(e[3], rows_per_launch, xd)
        groups.setdefault((info.kernel, info.per_lane, info.seg_lanes), []).append(e)
    batches = []
    for tile, ents in sorted(groups.items(), key=lambda kv: -sum(e[3].n * e[3].k for e in kv[1])):
        ys = [torch.empty((m, e[3].n), dtype=torch.float32, device="cuda") for e in ents]
        for r0 in range(0, m, rows_per_launch):
            r1 = r0 + rows_per_launch
            xs = [acts[(kind, e[2].k)][0][r0:r1] for e in ents]  # [rows, k]: the batch takes rows from its shape
            xs = [x.reshape(-1) if rows_per_launch == 1 else x for x in xs]
            xss = [acts[(kind, e[2].k)][1] for e in ents]
            xss = [None if v is None else v[r0:r1].reshape(-1) for v in xss]
            b = api.Batch([e[3] for e in ents], [e[4] for e in ents], xs, [y[r0:r1].reshape(-1) for y in ys],
                          xss if any(v is not None for v in xss) else None)
            b.tile = tile[1:]
            b.entries = ents
            b.outputs = ys
            batches.append(b)
    return batches


def make_step(entries, acts, kind):
    batches = make_batches(entries, acts, kind)

    def step():
        for b in batches:
            b.run()
    return step, batches


def capture(step):
    """A graph of one call of `step`, holding `step` (and through it the batch
    tables and outputs whose device addresses the graph's launches carry)."""
    import torch
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    g.launched = step
    return g


def time_graph(g, steps, warmup):
    import torch
    for _ in range(warmup):
        g.replay()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    start.record()
    for _ in range(steps):
        g.replay()
    end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return start.elapsed_time(end) / steps, wall


def time_graphs(graphs, steps, warmup):
    """time_graph over several graphs replayed in turn (one replay = one step)."""
    import torch
    n = len(graphs)
    for i in range(warmup):
        graphs[i % n].replay()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    start.record()
    for i in range(steps):
        graphs[i % n].replay()
    end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return start.elapsed_time(end) / steps, wall


def device_copies(entries, copies):
    """The layer set and copies - 1 clones of its device blobs (same layouts)."""
    sets = [entries]
    for _ in range(copies - 1):
        sets.append([(l, mi, spec, L, blob.clone()) for (l, mi, spec, L, blob) in entries])
    return sets


def warm_device(g, min_ms=100.0):
    """Replay a graph for at least `min_ms` of wall time, untimed.

    After the host-side packing the GPU has idled and its clocks start low:
    the first ~150 replays of the BitNet-like step run up to 20% slower than
    the steady state a decode loop sees.  This brings the device to that
    state once, before anything is timed."""
    import torch
    t0 = time.perf_counter()
    n = 0
    while (time.perf_counter() - t0) * 1e3 < min_ms:
        for _ in range(20):
            g.replay()
        n += 20
        torch.cuda.synchronize()
    return n, (time.perf_counter() - t0) * 1e3


def gpu_clock_under_load(g, seconds=1.5):
    """The GPU's current shader clock (MHz, from rocm-smi) sampled while
    `g` replays back to back for about `seconds`, untimed; None if the query
    fails.  rocm-smi takes a good part of a second to start, longer than a
    timed run, so the replays are queued first and the clock is read while
    they execute."""
    import re
    import subprocess

    import torch
    t0 = time.perf_counter()
    g.replay()
    torch.cuda.synchronize()
    one = max(time.perf_counter() - t0, 1e-5)
    for _ in range(min(int(seconds / one), 20000)):
        g.replay()
    try:
        out = subprocess.run(["rocm-smi", "-g", "--json"], capture_output=True, text=True, timeout=20).stdout
        mhz = []
        for card in json.loads(out).values():
            if isinstance(card, dict):
                mhz += [int(m) for key, v in card.items() if "sclk" in key.lower()
                        for m in re.findall(r"(\d+)\s*mhz", str(v).lower())]
        res = max(mhz) if mhz else None
    except (OSError, subprocess.SubprocessError, ValueError):
        res = None
    torch.cuda.synchronize()
    return res


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(wk, budget_s=12.0):
    """The oracle (decode + dense GEMV) on the host, on whole matrices of layer 0."""
    import oracle as O
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        cores = os.cpu_count() or 1
    done_w = 0
    done_bytes = 0
    t_total = 0.0
    mats = 0
    t_start = time.perf_counter()
    while time.perf_counter() - t_start < budget_s:
        for mi, spec in enumerate(wk.matrices):
            w, sc = wl.matrix_inputs(wk.cid, 0, mi, spec)
            xb = wl.activation_inputs(wk.cid, "bf16", 1, spec.k)
            p = O.bitcos_encode(w, sc, spec.group, 1)
            t0 = time.perf_counter()
            wd, sd = O.bitcos_decode(p)
            O.dense_gemv(wd, sd, spec.group, xb, x_is_bf16_bits=True)
            t_total += time.perf_counter() - t0
            done_w += spec.n * spec.k
            done_bytes += O.payload_bits(p) / 8
            mats += 1
            if time.perf_counter() - t_start >= budget_s:
                break
    return {
        "value": round(done_bytes / t_total / 1e9, 4),
        "unit": "GB/s",
        "cores": int(cores),
        "cpu_model": cpu_model(),
        "kind": "oracle",
        "sample": f"{mats} matrices of layer 0 of {wk.name} (decode + dense bf16 GEMV, "
                  f"{done_w / 1e6:.1f} M weights, {t_total:.1f} s)",
        "weights_per_s": round(done_w / t_total, 1),
    }


def profile_pass(args):
    """Counter runs: the dominant launch of the headline step, then a plain copy
    of known size whose FETCH_SIZE / WRITE_SIZE calibrate the counters."""
    import torch

    from paper_2609_16338_amd import _native as N

    wk = wl.WORKLOADS[args.workload]
    layers = args.layers or wk.layers
    packed = build_set(wk, layers, [N.FMT_BITCOS], args.threads)
    acts = activations(wk, ("bf16",))
    top = make_batches(packed[N.FMT_BITCOS], acts, "bf16")[0]
    for _ in range(5):
        top.run()
    torch.cuda.synchronize()
    n = COPY_MIB * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    alg = sum(e[3].payload_bits / 8 + e[3].k * 2 + e[3].n * 4 for e in top.entries)
    print(f"[profile-pass] dominant launch: {len(top.entries)} GEMVs, tile {top.tile}, "
          f"algorithmic bytes {int(alg)}; copy {COPY_MIB} MiB; kernel_source_hash {kernel_source_hash()}",
          flush=True)


def sweep(args):
    """Zero-density sweep: one 8192 x 8192 matrix with group-128 scales per z,
    batch 1, BITCOS against the five-trit and 2-bit kernels on this GPU.  Each
    format's blob is copied `--sweep-copies` times in HBM and one persistent
    launch covers all copies, so every launch streams more than twice the
    Infinity Cache; time per GEMV = launch time / copies."""
    import torch

    from paper_2609_16338_amd import _native as N
    from paper_2609_16338_amd import api

    cid, k = 4, 8192
    xi = torch.from_numpy(wl.activation_inputs(cid, "int8", 1, k)).cuda().reshape(-1)
    xb = torch.from_numpy(wl.activation_inputs(cid, "bf16", 1, k).view(np.int16)).view(torch.bfloat16).cuda().reshape(-1)
    names = {N.FMT_BITCOS: "bitcos", N.FMT_TRIT5: "trit5", N.FMT_BIT2: "bit2"}
    rows = []
    for zi, z in enumerate(wl.SWEEP_Z + (0.95,)):  # the paper's extreme point beside the config's five
        spec = wl.sweep_spec(z)
        w, sc = wl.matrix_inputs(cid, 0, zi, spec)
        row = {"z": z, "z_measured": round(float((w == 0).mean()), 5)}
        for fmt, nm in names.items():
            L, blob = api.plan_and_pack(fmt, w, sc, spec.group)
            src = torch.from_numpy(blob).cuda()
            blobs = [src.clone() for _ in range(args.sweep_copies)]
            row[f"{nm}_payload_bytes"] = L.payload_bits // 8
            row[f"{nm}_bpw"] = round(L.payload_bits / (spec.n * spec.k), 5)
            for kind, x in (("int8", xi), ("bf16", xb)):
                ys = [torch.empty(spec.n, dtype=torch.float32, device="cuda") for _ in blobs]
                b = api.Batch([L] * len(blobs), blobs, [x] * len(blobs), ys)
                g = capture(b.run)
                ms, _ = time_graph(g, args.steps, args.warmup)
                us = ms * 1e3 / len(blobs)
                row[f"{nm}_{kind}_us"] = round(us, 4)
                row[f"{nm}_{kind}_GBs"] = round(L.payload_bits / 8 / (us * 1e-6) / 1e9, 1)
                # CU-cycles per 32 weights with the weights streamed from HBM
                row[f"{nm}_{kind}_gamma_hbm"] = round(32 * CU_COUNT * CLOCK_HZ * us * 1e-6 / (spec.n * spec.k), 3)
                del g, b, ys
            del blobs, src
            torch.cuda.empty_cache()
        for kind in ("int8", "bf16"):
            t = row[f"bitcos_{kind}_us"]
            row[f"speedup_vs_trit5_{kind}"] = round(row[f"trit5_{kind}_us"] / t, 4)
            row[f"speedup_vs_bit2_{kind}"] = round(row[f"bit2_{kind}_us"] / t, 4)
        rows.append(row)
        print(f"[sweep] z={z}: " + ", ".join(f"{nm} {row[f'{nm}_int8_us']:.2f}/{row[f'{nm}_bf16_us']:.2f} us"
                                            for nm in names.values()), file=sys.stderr, flush=True)

    def crossover(kind):
        # z where the BITCOS / five-trit time ratio crosses 1 (linear between points)
        pts = [(r["z"], r[f"speedup_vs_trit5_{kind}"]) for r in rows]
        for (z0, s0), (z1, s1) in zip(pts, pts[1:]):
            if (s0 - 1) * (s1 - 1) <= 0 and s1 != s0:
                return round(z0 + (1 - s0) * (z1 - z0) / (s1 - s0), 4)
        return None

    print(json.dumps({
        "metric": "zero-density sweep, 8192x8192 g128, batch 1: per-GEMV time, effective GB/s, speedups",
        "unit": "us",
        "copies_per_launch": args.sweep_copies,
        "steps": args.steps,
        "warmup": args.warmup,
        "data": "synthetic",
        "crossover_z_vs_trit5_int8": crossover("int8"),
        "crossover_z_vs_trit5_bf16": crossover("bf16"),
        "points": rows,
    }))


GAMMA_Z = (0.30, 0.42, 0.515, 0.95)
CU_COUNT = 256
CLOCK_HZ = 2.4e9


def gamma(args):
    """The paper's two-term roofline (Sec. III-B, Eqs. (5)-(6)) on this GPU.

    gamma = CU-cycles one CU spends per 32 weights when the operands are
    L2-resident (one launch over 64 GEMVs that all read the same 2048 x 8192
    g128 blob, 3.6-4.4 MB, which each XCD's 4 MB L2 holds, so the instruction
    stream is the limit and the kernel's prologue is amortised); beta = HBM
    bytes per CU-cycle at the
    8 TB/s peak; B(z) = bytes per 32 weights of each layout.  Predicted
    effective bandwidth = min(beta, B / gamma) per CU, times all CUs."""
    import torch

    from paper_2609_16338_amd import _native as N
    from paper_2609_16338_amd import api

    cid, n, k = 6, 2048, 8192
    beta = HBM_PEAK_GBS * 1e9 / (CU_COUNT * CLOCK_HZ)
    xi = torch.from_numpy(wl.activation_inputs(cid, "int8", 1, k)).cuda().reshape(-1)
    xb = torch.from_numpy(wl.activation_inputs(cid, "bf16", 1, k).view(np.int16)).view(torch.bfloat16).cuda().reshape(-1)
    names = {N.FMT_BITCOS: "bitcos", N.FMT_TRIT5: "trit5", N.FMT_BIT2: "bit2"}
    rows = []
    for zi, z in enumerate(GAMMA_Z):
        spec = wl.MatrixSpec(f"gamma_z{z}", n, k, z, 128, 0.01, 0.1)
        w, sc = wl.matrix_inputs(cid, 0, zi, spec)
        row = {"z": z, "z_measured": round(float((w == 0).mean()), 5)}
        for fmt, nm in names.items():
            L, blob = api.plan_and_pack(fmt, w, sc, spec.group)
            dev = torch.from_numpy(blob).cuda()
            b32 = L.payload_bits / 8 / (n * k) * 32
            row[f"{nm}_bytes_per_32"] = round(b32, 4)
            reps = 64
            devs = [dev] * reps
            for kind, x in (("int8", xi), ("bf16", xb)):
                ys = [torch.empty(n, dtype=torch.float32, device="cuda") for _ in range(reps)]
                b = api.Batch([L] * reps, devs, [x] * reps, ys)
                g = capture(b.run)
                ms, _ = time_graph(g, max(args.steps, 50), args.warmup)
                rate = reps * n * k / (ms * 1e-3)
                gam = 32 * CU_COUNT * CLOCK_HZ / rate
                row[f"{nm}_{kind}_gamma"] = round(gam, 3)
                row[f"{nm}_{kind}_pred_GBs"] = round(min(beta, b32 / gam) * CU_COUNT * CLOCK_HZ / 1e9, 1)
                row[f"{nm}_{kind}_bound"] = "memory" if b32 / gam > beta else "instructions"
                del g, b, ys
            del devs
        rows.append(row)
        print(f"[gamma] z={z}: " + ", ".join(f"{nm} {row[f'{nm}_int8_gamma']:.2f}/{row[f'{nm}_bf16_gamma']:.2f}"
                                            for nm in names.values()), file=sys.stderr, flush=True)
    print(json.dumps({
        "metric": "two-term roofline: gamma = CU-cycles per 32 weights, L2-resident 2048x8192 g128 (x64 per launch), batch 1",
        "beta_bytes_per_cu_cycle": round(beta, 4),
        "clock_hz": CLOCK_HZ,
        "cus": CU_COUNT,
        "data": "synthetic",
        "points": rows,
    }))


def main():
    args = parse()
    if args.gamma:
        gamma(args)
        return
    if args.profile_pass:
        profile_pass(args)
        return
    if args.sweep:
        sweep(args)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1"}))
        sys.exit(2)
    import torch

    from paper_2609_16338_amd import _native as N
    from paper_2609_16338_amd import api

    N.lib()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    wk = wl.WORKLOADS[args.workload]
    layers = args.layers or wk.layers
    m = args.batch
    if not 1 <= m <= 16:
        print(json.dumps({"error": "--batch must be in 1..16"}))
        sys.exit(2)
    fmts = [N.FMT_BITCOS] + ([] if args.no_baselines else [N.FMT_TRIT5, N.FMT_BIT2])
    t0 = time.perf_counter()
    packed = build_set(wk, layers, fmts, args.threads)
    acts = activations(wk, ("bf16", "int8"), m)
    prep_s = time.perf_counter() - t0
    print(f"[bench] packed {layers} layers x {len(wk.matrices)} matrices in {prep_s:.1f} s", file=sys.stderr, flush=True)

    payload = {fmt: sum(e[3].payload_bits for e in ents) / 8 for fmt, ents in packed.items()}
    weights = sum(e[3].n * e[3].k for e in packed[N.FMT_BITCOS])
    res = {}
    unsupported = {}
    copies = max(1, args.copies)
    bitcos_sets = None
    warmed = False
    for fmt in fmts:
        sets = device_copies(packed[fmt], copies)
        for kind in ("bf16", "int8"):
            if not supported(packed[fmt], kind, m):
                if fmt == N.FMT_BITCOS:
                    raise SystemExit(f"no BITCOS kernel for this set with {kind} activations at batch {m}")
                res[(fmt, kind)] = None
                unsupported[f"{FMT_NAMES[fmt]}_{kind}"] = "no kernel for rows this long (K > 16384 with bf16 activations)"
                print(f"[bench] fmt={fmt} {kind}: no kernel for this set, skipped", file=sys.stderr, flush=True)
                continue
            gs = [capture(make_step(st, acts, kind)[0]) for st in sets]
            if not warmed:
                warmed = True
                n, wms = warm_device(gs[0])
                print(f"[bench] device warm-up: {n} untimed replays in {wms:.0f} ms", file=sys.stderr, flush=True)
            ms, wall = time_graphs(gs, args.steps, args.warmup)
            res[(fmt, kind)] = ms
            print(f"[bench] fmt={fmt} {kind}: {ms * 1e3:.1f} us/step, "
                  f"{payload[fmt] / (ms * 1e-3) / 1e9:.1f} GB/s", file=sys.stderr, flush=True)
            del gs
        if fmt == N.FMT_BITCOS:
            bitcos_sets = sets
        del sets

    # Dominant kernel: the batched BITCOS launch carrying most of the bytes
    # (the K = 2560 tile for this set: q, k, v, o, gate, up of every layer),
    # timed alone.
    tops = [make_batches(st, acts, "bf16")[0] for st in bitcos_sets]
    top = tops[0]
    # Ten back-to-back launches per replay, over the device copies in turn:
    # inside a graph consecutive kernels start without a gap, so replay
    # overhead stays out of the per-launch time.
    reps = 10
    gg = capture(lambda: [tops[i % len(tops)].run() for i in range(reps)])
    ms_g, _ = time_graph(gg, args.steps, args.warmup)
    per_launch_us = ms_g * 1e3 / reps
    sclk = gpu_clock_under_load(gg)
    alg_bytes = sum(e[3].payload_bits / 8 + m * (e[3].k * 2 + e[3].n * 4) for e in top.entries)
    achieved = alg_bytes / (per_launch_us * 1e-6) / 1e9
    # Two-term roofline of the launch in CU-cycles per 32 weights (nominal
    # clock): its measured time against the time its bytes take at peak HBM
    # bandwidth; the larger term binds.
    top_weights = sum(e[3].n * e[3].k for e in top.entries)
    launch_gamma = 32 * CU_COUNT * CLOCK_HZ * per_launch_us * 1e-6 / top_weights
    hbm_term = 32 * alg_bytes / top_weights / (HBM_PEAK_GBS * 1e9 / (CU_COUNT * CLOCK_HZ))
    ms = res[(N.FMT_BITCOS, "bf16")]
    value = payload[N.FMT_BITCOS] / (ms * 1e-3) / 1e9
    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": f"{wk.name}: {layers} layers x {{q,o {wk.matrices[0].n}x{wk.matrices[0].k}; "
                        f"k,v {wk.matrices[1].n}x{wk.matrices[1].k}; gate,up {wk.matrices[4].n}x{wk.matrices[4].k}; "
                        f"down {wk.matrices[6].n}x{wk.matrices[6].k}}}, z={wk.matrices[0].z} iid, "
                        f"{'per-tensor' if wk.matrices[0].group == 0 else 'group-128'} fp16 scales, "
                        f"bf16 x ~ N(0,1), batch {m}",
            "global_batch": m,
            "layers": layers,
            "gemvs_per_step": len(packed[N.FMT_BITCOS]),
            "weights_per_step": weights,
            "payload_bytes_per_step": int(payload[N.FMT_BITCOS]),
            "total_bytes_per_step": int(sum(e[3].total_bytes + m * (e[3].k * 2 + e[3].n * 4)
                                            for e in packed[N.FMT_BITCOS])),
            "device_copies": copies,
        },
        "pct_of_hbm_peak": round(100 * value / HBM_PEAK_GBS, 2),
        "weights_per_s": float(f"{weights / (ms * 1e-3):.4g}"),
        "bpw_payload": round(payload[N.FMT_BITCOS] * 8 / weights, 5),
    }
    def ratio(fmt, kind, t):
        v = res.get((fmt, kind))
        return None if v is None else round(v / t, 4)

    ms8 = res[(N.FMT_BITCOS, "int8")]
    if N.FMT_TRIT5 in fmts:
        out["speedup_vs_trit5"] = ratio(N.FMT_TRIT5, "bf16", ms)
        out["speedup_vs_bit2"] = ratio(N.FMT_BIT2, "bf16", ms)
        out["baselines_us_per_step"] = {
            f"{FMT_NAMES[f]}_{kind}": None if res[(f, kind)] is None else round(res[(f, kind)] * 1e3, 2)
            for f in (N.FMT_TRIT5, N.FMT_BIT2) for kind in ("bf16", "int8")}
        if m > 1:
            out["baselines_note"] = f"no small-batch kernel: {m} batch-1 launches per tile and step"
        if unsupported:
            out["baselines_unsupported"] = unsupported
    out["int8_variant"] = {
        "value": round(payload[N.FMT_BITCOS] / (ms8 * 1e-3) / 1e9, 2),
        "ms_per_step": round(ms8, 5),
        "speedup_vs_trit5": ratio(N.FMT_TRIT5, "int8", ms8),
        "speedup_vs_bit2": ratio(N.FMT_BIT2, "int8", ms8),
    }
    # The kernel the launcher picks (all GEMVs of the launch share layout kind and tile).
    kinds = {api.describe(e[3], m, N.X_BF16).kernel for e in top.entries}
    kname = {N.KERNEL_MATRIX: "bitcos_diag_kernel", N.KERNEL_STREAMING: "bitcos_fast_kernel",
             N.KERNEL_GENERAL: "bitcos_gemv_kernel", N.KERNEL_SMALL_BATCH: "bitcos_mfma_kernel",
             }.get(kinds.pop(), "?") if len(kinds) == 1 else "mixed"
    out["roofline"] = {
        "bound": "hbm",
        "achieved": round(achieved, 2),
        "peak": HBM_PEAK_GBS,
        "unit": "GB/s",
        "frac": round(achieved / HBM_PEAK_GBS, 4),
        "traffic": stored_traffic(),
        "kernel": f"{kname}<{top.tile[0]},{top.tile[1]},bf16,table>: {len(top.entries)} GEMVs in one launch",
        "per_launch_us": round(per_launch_us, 3),
        "bytes_per_launch": int(alg_bytes),
        "two_term": {"cu_cycles_per_32w": round(launch_gamma, 4), "hbm_cu_cycles_per_32w": round(hbm_term, 4),
                     "binds": "instructions" if launch_gamma > hbm_term else "hbm"},
    }
    out["sclk_mhz_under_load"] = sclk
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wk)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
