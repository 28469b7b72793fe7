#!/usr/bin/env python3
"""Benchmark: BITCOS ternary GEMV effective weight bandwidth on one MI355X.

A step is one batch-1 pass over a whole decode layer set (every GEMV of every
layer, inputs already resident in HBM), replayed from a HIP graph.  The
headline (N = 1) is the largest layer set that fits one GPU, the
Qwen3-32B-like set: 64 layers x {q, o 5120x5120; k, v 1024x5120; gate, up
25600x5120; down 5120x25600}, per-row zero density drawn uniform in
[0.30, 0.60], group-128 fp16 scales, bf16 activations ~ N(0, 1); the same
step with int8 activations (quantised per group of 128 by the library) is
reported beside it.  value = sum of BITCOS payload bytes (bitmap + signs +
scales) / step time.  The same step over the five-trit and 2-bit layouts of
the same weights gives the same-GPU speedups.  The BitNet-2B-like set is
timed the same way and reported as an extra block.

Timing: every (format, activation type) gets its own untimed warm-up of at
least --warm-ms milliseconds of replays (the GPU's clocks ramp for ~30 ms
after an idle stretch such as host-side packing or a graph capture), then
--warmup more untimed replays, then --steps timed ones bracketed by events
on the replay stream.  Two device copies of the set are replayed in turn, so
a weight is re-read only after more than twice the 256 MB Infinity Cache of
other payload has streamed by.

Self-check: after timing, the outputs of the last replay of every device
copy are compared, on sampled rows of every GEMV, with the dense definition
y = sum_g S a sum_k W x computed here in float64 from the same weights and
activations (bars: bf16 activations |y - ref| <= 1e-3 sum_k |S W x|; int8
activations with activation scales |y - ref| <= 1e-5 sum_g |S a A|).  A
mismatch prints an error line and exits with status 3 instead of a value.

Prints ONE JSON line.  roofline: the dominant launch (the persistent launch
carrying most of the step's bytes) timed alone from a graph of ten
back-to-back launches; achieved = its algorithmic bytes (payload + M K
activation bytes + 4 M N output bytes per GEMV) per launch time, against the
8 TB/s HBM peak; traffic = its measured HBM bytes (FETCH_SIZE + WRITE_SIZE
scaled by a plain copy's counters, stored under profiles/) while the kernel
sources are unchanged; two_term: the launch's time and its bytes at peak HBM
bandwidth in CU-cycles per 32 weights at the nominal 2.4 GHz, and which
term is larger; valu: the launch's stored VALU instruction count (rocprofv3
SQ_INSTS_VALU, same source rule) as a share of the SIMDs' issue cycles.
cpu_baseline: the oracle's decode + dense GEMV on whole layer-0 matrices on
the host (about 12 s of work).

Other modes print their own JSON line: --sweep (zero-density sweep on one
8192 x 8192 matrix), --gamma (two-term roofline on cache-resident data),
--hbm-read (plain streaming-read bandwidth of this GPU), --profile-pass (the
dominant launch and a calibration copy, for counter runs).
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
CU_COUNT = 256
CLOCK_HZ = 2.4e9
FMT_NAMES = {1: "bitcos", 2: "trit5", 3: "bit2"}
METRIC = "ternary GEMV effective weight GB/s (% of 8 TB/s HBM peak); speedup vs 5-trit"
HEADLINE = "qwen3_32b_layers"
SAMPLE_ROWS = 6  # rows of every GEMV checked after timing (first, last and random ones)


def parse(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=200)
    ap.add_argument("--warm-ms", type=float, default=200.0,
                    help="untimed replays for at least this long before each format's timed window")
    ap.add_argument("--workload", default=HEADLINE)
    ap.add_argument("--extra", default="bitnet2b_layers",
                    help="comma-separated layer sets timed after the headline and reported as extra blocks")
    ap.add_argument("--batch", type=int, default=1,
                    help="activation rows per GEMV (1..16); BITCOS runs M > 1 on its small-batch kernel")
    ap.add_argument("--layers", type=int, default=0, help="0 = the workload's layer count")
    ap.add_argument("--copies", type=int, default=2,
                    help="device copies of the layer set, replayed in turn (more than 2 x the 256 MB Infinity Cache)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-baselines", action="store_true", help="skip the five-trit / 2-bit steps")
    ap.add_argument("--no-check", action="store_true", help="skip the output self-check after timing")
    ap.add_argument("--threads", type=int, default=min(16, os.cpu_count() or 1))
    ap.add_argument("--out", default="", help="also write the JSON line to this file")
    ap.add_argument("--profile-pass", action="store_true",
                    help="for counter runs: the dominant BITCOS launch x5, then a plain 256 MiB device copy x5")
    ap.add_argument("--profile-sweep", action="store_true",
                    help="for counter runs: the z = 0.42 sweep launch of every format, int8 and bf16, x5 each")
    ap.add_argument("--sweep", action="store_true",
                    help="zero-density sweep on one 8192 x 8192 matrix: BITCOS vs five-trit vs 2-bit (own JSON line)")
    ap.add_argument("--gamma", action="store_true",
                    help="two-term roofline: cycles per 32 weights on cache-resident data vs z (own JSON line)")
    ap.add_argument("--hbm-read", action="store_true",
                    help="plain streaming-read bandwidth of this GPU (own JSON line)")
    ap.add_argument("--sweep-copies", type=int, default=40,
                    help="device copies of each swept matrix streamed per launch (> 2 x the 256 MB Infinity Cache)")
    ap.add_argument("--sweep-shape", default="8192x8192",
                    help="N x K of the swept matrix (the paper's own sweep matrix is 32768x16384)")
    ap.add_argument("--sweep-z", default="", help="comma-separated zero densities (default: the five of the sweep and 0.95)")
    return ap.parse_args(argv)


def emit(obj, args):
    line = json.dumps(obj)
    print(line, flush=True)
    if getattr(args, "out", ""):
        with open(args.out, "w") as f:
            f.write(line + "\n")


# Sources of each BITCOS kernel (its device code, the launcher that sizes its
# grid and the batch-table builder): a stored HBM-traffic measurement of a
# launch is reported only while its kernel's sources are unchanged.
_COMMON_SOURCES = ["bitcos_kernel.h", "tables.h", "device_common.h", "batch.h", "batch.hip", "launch_common.h",
                   "plan.h"]
KERNEL_SOURCES = {
    "bitcos_fast_kernel": ["bitcos_fast.h", "gemv_bitcos.hip"] + _COMMON_SOURCES,
    "bitcos_diag_kernel": ["bitcos_diag.h", "bitcos_fast.h", "mfma_common.h", "gemv_bitcos.hip"] + _COMMON_SOURCES,
    "bitcos_mfma_kernel": ["bitcos_mfma.h", "mfma_common.h", "gemv_bitcos_mfma.hip"] + _COMMON_SOURCES,
    "trit5_gemv_kernel": ["fixed_kernel.h", "fixed_trit5.hip", "gemv_fixed.hip"] + _COMMON_SOURCES,
    "bit2_gemv_kernel": ["fixed_kernel.h", "fixed_bit2.hip", "gemv_fixed.hip"] + _COMMON_SOURCES,
}
TRAFFIC_FILES = {
    "qwen3_32b_layers": [os.path.join(ROOT, "profiles", f) for f in (
        "bitcos_fast_bf16_qwen3_32b_k5120_traffic.txt", "bitcos_mfma_bf16_qwen3_32b_m16_traffic.txt")],
    "bitnet2b_layers": [os.path.join(ROOT, "profiles", "bitcos_diag_bf16_bitnet2b_k2560_traffic.txt")],
}
COUNTER_FILES = {
    "qwen3_32b_layers": [os.path.join(ROOT, "profiles", "bitcos_fast_bf16_qwen3_32b_counters.txt")],
}
COPY_MIB = 256


def kernel_source_hash(kernel="bitcos_fast_kernel"):
    """Hash of a kernel's sources without their // comments and blank space,
    so that editing a comment keeps a stored measurement valid."""
    import hashlib
    import re
    h = hashlib.sha256()
    for name in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, "paper_2609_16338_amd", "csrc", name), encoding="utf-8") as f:
            code = re.sub(r"//[^\n]*", "", f.read())
        h.update(name.encode() + b"\0" + " ".join(code.split()).encode())
    return h.hexdigest()[:16]


def _stored(files, launch):
    """key: value lines of the first stored measurement of `launch` whose
    kernel sources are unchanged, or None."""
    for path in files:
        try:
            with open(path) as f:
                kv = dict(line.split(":", 1) for line in f if ":" in line and not line.startswith("#"))
        except OSError:
            continue
        kv = {k.strip(): v.strip() for k, v in kv.items()}
        kernel = launch.split("<")[0]
        if kv.get("launch") != launch or kernel not in KERNEL_SOURCES:
            continue
        if kv.get("kernel_source_hash") != kernel_source_hash(kernel):
            continue
        return kv
    return None


def stored_valu(workload, launch):
    """VALU instructions per launch of the dominant launch (rocprofv3
    SQ_INSTS_VALU, wave instructions summed over the GPU) from the stored
    counter passes of the same launch, or None if there are none or the
    kernel sources changed since."""
    kv = _stored(COUNTER_FILES.get(workload, []), launch)
    try:
        return None if kv is None else int(float(kv["sq_insts_valu_per_launch"]))
    except (KeyError, ValueError):
        return None


def stored_traffic(workload, launch):
    """HBM bytes per launch of the dominant launch from the FETCH_SIZE / WRITE_SIZE
    passes (scaled by the copy calibration): from the stored measurement of
    the same launch (`launch`: its label, say "bitcos_fast_kernel<5,32,bf16,
    table>: 704 GEMVs in one launch"), or None if there is none or the kernel
    sources changed since it was taken."""
    kv = _stored(TRAFFIC_FILES.get(workload, []), launch)
    try:
        return None if kv is None else int(float(kv["traffic_bytes_per_launch"]))
    except (KeyError, ValueError):
        return None


def launch_label(top, m):
    """Kernel, tile and GEMV count of a batched launch (bf16 activations)."""
    from paper_2609_16338_amd import _native as N
    from paper_2609_16338_amd import api

    kinds = {api.describe(e[3], m, N.X_BF16).kernel for e in top.entries}
    kname = {N.KERNEL_MATRIX: "bitcos_diag_kernel", N.KERNEL_STREAMING: "bitcos_fast_kernel",
             N.KERNEL_GENERAL: "bitcos_gemv_kernel", N.KERNEL_SMALL_BATCH: "bitcos_mfma_kernel",
             }.get(kinds.pop(), "?") if len(kinds) == 1 else "mixed"
    return f"{kname}<{top.tile[0]},{top.tile[1]},bf16,table>: {len(top.entries)} GEMVs in one launch"


# ---------------------------------------------------------------------------
# Inputs
# ---------------------------------------------------------------------------

def sample_rows(n, l, mi, count=SAMPLE_ROWS):
    rng = np.random.default_rng([l, mi, n])
    rows = {0, n - 1} | set(rng.choice(n, size=min(max(count - 2, 0), n), replace=False).tolist())
    return np.array(sorted(rows))


KSPLIT_MAX = 16384  # longest row a batch-1 tile holds (bf16: 64 lanes x 8 words of 32 weights)


def column_blocks(k):
    """[(k0, width)] of a row of k weights: the whole row, or, for rows longer
    than KSPLIT_MAX, equal column blocks (a split of K, as row-parallel
    layers are split across GPUs) whose width is a multiple of 128 that some
    batch-1 tile covers without idle lanes (the widest such), else the widest
    multiple of 128 that divides k.  Each block is packed as a matrix of its
    own; their GEMVs add into one output (the library's _ADD output modes)."""
    if k <= KSPLIT_MAX:
        return [(0, k)]
    cands = [b for b in range(128, KSPLIT_MAX + 1, 128) if k % b == 0]
    if not cands:
        return [(0, k)]

    def full(b):
        words = b // 32
        return any(words % seg == 0 and words // seg <= 8 for seg in (64, 32, 16, 8, 4))
    b = max([c for c in cands if full(c)] or cands)
    return [(k0, b) for k0 in range(0, k, b)]


def build_set(wk, layers, fmts, threads, samples=None):
    """Pack every matrix of the layer set in every format (host), upload to HBM.

    Entries are (layer, matrix, spec, layout, device blob, (block, k0, width)):
    one per matrix, or one per column block for rows longer than a batch-1
    tile (column_blocks).  With `samples` (a dict), the weights and scales of
    a few rows of every matrix are kept there, keyed by (layer, matrix), for
    the self-check."""
    import torch

    from paper_2609_16338_amd import api

    jobs = [(l, mi, spec) for l in range(layers) for mi, spec in enumerate(wk.matrices)]

    def one(job):
        l, mi, spec = job
        w, sc = wl.matrix_inputs(wk.cid, l, mi, spec)
        out = {}
        for fmt in fmts:
            out[fmt] = []
            for c, (k0, kb) in enumerate(column_blocks(spec.k)):
                wb = np.ascontiguousarray(w[:, k0:k0 + kb])
                sb = sc.reshape(spec.n, spec.k // 128)[:, k0 // 128:(k0 + kb) // 128] if spec.group == 128 else sc
                out[fmt].append((api.plan_and_pack(fmt, wb, np.ascontiguousarray(sb).reshape(-1), spec.group),
                                 (c, k0, kb)))
        keep = None
        if samples is not None:  # (rows, their weights, their fp16 scale bits [rows][k/128] or [1][1])
            rows = sample_rows(spec.n, l, mi)
            sbits = sc.reshape(spec.n, spec.k // 128)[rows] if spec.group == 128 else sc.reshape(1, 1)
            keep = (rows, np.ascontiguousarray(w[rows]), np.ascontiguousarray(sbits))
        return job, out, keep

    packed = {}
    with cf.ThreadPoolExecutor(max_workers=threads) as ex:
        for (l, mi, spec), out, keep in ex.map(one, jobs):
            for fmt, parts in out.items():
                for (L, blob), part in parts:
                    packed.setdefault(fmt, []).append((l, mi, spec, L, torch.from_numpy(blob).cuda(), part))
            if keep is not None:
                samples[(l, mi)] = keep
    return packed


def bf16_bits_to_f64(bits):
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def activations(wk, kinds, m=1):
    """Per distinct K: device activations [m, k] (bf16, and int8 + per-group
    scales via the library), and host float64 copies of what the GEMVs read."""
    import torch

    from paper_2609_16338_amd import api

    acts, host = {}, {}
    for k in sorted({s.k for s in wk.matrices}):
        xb = wl.activation_inputs(wk.cid, "bf16", m, k)
        xbd = torch.from_numpy(xb.view(np.int16)).view(torch.bfloat16).cuda()
        acts[("bf16", k)] = (xbd, None)
        host[("bf16", k)] = (bf16_bits_to_f64(xb).reshape(m, k), None)
        if "int8" in kinds:
            q = torch.empty((m, k), dtype=torch.int8, device="cuda")
            a = torch.empty((m, k // 128), dtype=torch.float32, device="cuda")
            api.quantize_activations(xbd, q, a)
            acts[("int8", k)] = (q, a)
    torch.cuda.synchronize()
    for (kind, k), (x, a) in acts.items():
        if kind == "int8":  # the GEMV's own inputs, as the library quantised them
            host[(kind, k)] = (x.cpu().numpy().astype(np.float64), a.cpu().numpy().astype(np.float64))
    return acts, host


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


class AddPartials:
    """The step's last launch: the partial outputs of the split matrices'
    later column blocks added into their outputs (bitcos_add_partials), one
    call per stacked output buffer."""

    def __init__(self, sums):
        self.sums = sums  # [(Y [count, m, n], P [blocks - 1, count, m, n])]
        self.entries, self.outputs = [], []
        self.phase, self.tile, self.kernel = 1, ("partials",), "add_partials"

    def run(self, stream=None):
        from paper_2609_16338_amd import api
        for y, parts in self.sums:
            api.add_partials(y, parts, stream)


def make_batches(entries, acts, kind):
    """One persistent launch per tile: the step's GEMVs grouped by kernel tile.

    Column blocks of a long row (column_blocks) all run in those launches:
    a matrix's first block writes its output, block c + 1 writes slice c of
    a partial buffer, and a last step (AddPartials) adds the slices into the
    outputs in block order -- the same fp32 additions as the accumulating
    output mode with one launch per block, so each output is a deterministic
    sum.  The outputs of split matrices of one shape are stacked in one
    buffer (and their partials in another) so that one call sums them all.
    With m activation rows, BITCOS takes all m in one launch (small-batch
    kernel); the five-trit and 2-bit layouts, which have no small-batch
    kernel, take m batch-1 launches per tile, one per activation row, as
    their m > 1 entry points do.  A batch's `outputs` are the matrices' final
    outputs (what a check reads after the whole step)."""
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
    # Outputs: one [m, n] per matrix; split matrices of one (n, blocks) in a
    # stacked [count, m, n] buffer with their partials in [blocks - 1, count, m, n].
    nblocks, nrows = {}, {}
    for e in entries:
        nblocks[(e[0], e[1])] = max(nblocks.get((e[0], e[1]), 0), e[5][0] + 1)
        nrows[(e[0], e[1])] = e[2].n
    ys, part, stacks = {}, {}, {}
    for key, nb in nblocks.items():
        if nb == 1:
            ys[key] = torch.empty((m, nrows[key]), dtype=torch.float32, device="cuda")
        else:
            stacks.setdefault((nrows[key], nb), []).append(key)
    sums = []
    for (n, nb), keys in stacks.items():
        y_all = torch.empty((len(keys), m, n), dtype=torch.float32, device="cuda")
        p_all = torch.empty((nb - 1, len(keys), m, n), dtype=torch.float32, device="cuda")
        for i, key in enumerate(keys):
            ys[key] = y_all[i]
            for c in range(1, nb):
                part[key + (c,)] = p_all[c - 1, i]
        sums.append((y_all, p_all))
    # Activations of a block: a contiguous copy of its columns (made once).
    blk = {}

    def x_of(e):
        c, k0, kb = e[5]
        x, a = acts[(kind, e[2].k)]
        if kb == e[2].k:
            return x, a
        key = (e[2].k, k0, kb)
        if key not in blk:
            blk[key] = (x[:, k0:k0 + kb].contiguous(),
                        None if a is None else a[:, k0 // 128:(k0 + kb) // 128].contiguous())
        return blk[key]

    batches = []
    order = sorted(groups.items(), key=lambda kv: -sum(e[3].n * e[3].k for e in kv[1]))
    for key, ents in order:
        outs = [ys[(e[0], e[1])] for e in ents]
        dsts = [outs[i] if e[5][0] == 0 else part[(e[0], e[1], e[5][0])] for i, e in enumerate(ents)]
        for r0 in range(0, m, rows_per_launch):
            r1 = r0 + rows_per_launch
            xs = [x_of(e)[0][r0:r1] for e in ents]  # [rows, k]: the batch takes rows from its shape
            xs = [x.reshape(-1) if rows_per_launch == 1 else x for x in xs]
            xss = [x_of(e)[1] for e in ents]
            xss = [None if v is None else v[r0:r1].reshape(-1) for v in xss]
            b = api.Batch([e[3] for e in ents], [e[4] for e in ents], xs, [y[r0:r1].reshape(-1) for y in dsts],
                          xss if any(v is not None for v in xss) else None, y_mode=N.Y_F32)
            b.tile = key[1:]
            b.kernel = key[0]
            b.phase = 0
            b.entries = ents
            b.outputs = outs
            b.keep_x = blk
            batches.append(b)
    if sums:
        batches.append(AddPartials(sums))
    return batches


def make_step(entries, acts, kind):
    batches = make_batches(entries, acts, kind)

    def step():
        for b in batches:
            b.run()
    step.batches = batches
    return step, batches


# ---------------------------------------------------------------------------
# Graphs and timing
# ---------------------------------------------------------------------------

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


def warm(graphs, min_ms):
    """Replay the graphs in turn for at least `min_ms` of wall time, untimed.

    After an idle stretch (host-side packing, graph capture, another
    format's checks) the GPU's clocks start low and the first ~150 replays
    of a step run up to 20% slower than the steady state a decode loop
    sees; every timed window is preceded by this."""
    import torch
    t0 = time.perf_counter()
    n = 0
    while (time.perf_counter() - t0) * 1e3 < min_ms:
        for _ in range(10):
            graphs[n % len(graphs)].replay()
            n += 1
        torch.cuda.synchronize()
    return n, (time.perf_counter() - t0) * 1e3


def time_graphs(graphs, steps, warmup, warm_ms=0.0):
    """Per-replay time (ms) of the graphs replayed in turn, one replay = one
    step: a time-based warm-up, `warmup` more replays, then `steps` timed."""
    import torch
    if warm_ms > 0:
        warm(graphs, warm_ms)
    n = len(graphs)
    for i in range(warmup):
        graphs[i % n].replay()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record()
    for i in range(steps):
        graphs[i % n].replay()
    end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end) / steps


def time_graph(g, steps, warmup, warm_ms=0.0):
    return time_graphs([g], steps, warmup, warm_ms)


def device_copies(entries, copies):
    """The layer set and copies - 1 clones of its device blobs (same layouts)."""
    sets = [entries]
    for _ in range(copies - 1):
        sets.append([(l, mi, spec, L, blob.clone(), part) for (l, mi, spec, L, blob, part) in entries])
    return sets


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


# ---------------------------------------------------------------------------
# Self-check of the timed outputs
# ---------------------------------------------------------------------------

def dense_rows(w_rows, s_bits, group, x, xscale):
    """y[m, r] and its error scales for the sampled rows, from the definition
    y = sum_g S[r, g] a[m, g] sum_{k in g} W[r, k] x[m, k] in float64 (S from
    the fp16 bits s_bits: [r][k/128], or [1][1] for one scale per tensor).

    Returns (y, sum_k |S W x| (bf16 bar), sum_g |S a A| (int8 bar))."""
    r, k = w_rows.shape
    m = x.shape[0]
    wf = w_rows.astype(np.float64)
    s_rows = np.asarray(s_bits, dtype=np.uint16).view(np.float16).astype(np.float64)
    if group == 128 or xscale is not None:
        g = k // 128
        A = np.einsum("rgk,mgk->mrg", wf.reshape(r, g, 128), x.reshape(m, g, 128))
        S = s_rows if s_rows.shape[1] == g else np.full((r, g), s_rows[0, 0])
        a = np.ones((m, 1, g)) if xscale is None else xscale.reshape(m, 1, g)
        terms = S[None] * a * A
        y = terms.sum(axis=2)
        gbar = np.abs(terms).sum(axis=2)
        Sk = np.repeat(S, 128, axis=1)
        ak = np.ones((m, k)) if xscale is None else np.repeat(xscale.reshape(m, g), 128, axis=1)
        kbar = (np.abs(ak * x)) @ np.abs(Sk * wf).T
    else:
        s = s_rows[0, 0]
        y = s * (x @ wf.T)
        kbar = s * (np.abs(x) @ np.abs(wf).T)
        gbar = np.abs(y)
    return y, kbar, gbar


def check_outputs(batches, samples, xhost, kind):
    """Compare the outputs of the last replay with dense_rows on the sampled
    rows of every GEMV.  Returns (ok, rows checked, worst error / allowed)."""
    import torch
    torch.cuda.synchronize()
    ok, rows_checked, worst = True, 0, 0.0
    seen = set()
    for b in batches:
        for e, y in zip(b.entries, b.outputs):
            l, mi, spec = e[0], e[1], e[2]
            if (l, mi) in seen:  # the column blocks of a matrix share its output
                continue
            seen.add((l, mi))
            rows, w_rows, s_rows = samples[(l, mi)]
            x, xs = xhost[(kind, spec.k)]
            ref, kbar, gbar = dense_rows(w_rows, s_rows, spec.group, x, xs)
            got = y.cpu().numpy().astype(np.float64)[:, rows]
            err = np.abs(got - ref)
            allowed = 1e-3 * kbar if kind == "bf16" else 1e-5 * gbar
            ratio = float(np.max(err / (allowed + 1e-30)))
            worst = max(worst, ratio)
            rows_checked += got.size
            if not np.all(err <= allowed + 1e-30) or not np.all(np.isfinite(got)):
                ok = False
    return ok, rows_checked, worst


# ---------------------------------------------------------------------------
# One layer set
# ---------------------------------------------------------------------------

def describe_workload(wk, layers, m):
    mats = wk.matrices
    z = (f"per-row z ~ U[{mats[0].row_z[0]}, {mats[0].row_z[1]}]" if mats[0].row_z else f"z={mats[0].z} iid")
    return (f"{wk.name}: {layers} layers x {{q,o {mats[0].n}x{mats[0].k}; k,v {mats[1].n}x{mats[1].k}; "
            f"gate,up {mats[4].n}x{mats[4].k}; down {mats[6].n}x{mats[6].k}}}, {z}, "
            f"{'per-tensor' if mats[0].group == 0 else 'group-128'} fp16 scales, batch {m}")


def run_workload(name, args, m, fmts, check=True, say=None):
    """Time the step of one layer set in every format and activation type.

    Returns a dict with the per-format step times, bytes, the self-check
    result, and what the dominant-launch roofline needs."""
    from paper_2609_16338_amd import _native as N

    say = say or (lambda *a: print("[bench]", *a, file=sys.stderr, flush=True))
    wk = wl.WORKLOADS[name]
    layers = args.layers or wk.layers
    t0 = time.perf_counter()
    samples = {} if check else None
    packed = build_set(wk, layers, fmts, args.threads, samples)
    acts, xhost = activations(wk, ("bf16", "int8"), m)
    say(f"{name}: packed {layers} layers x {len(wk.matrices)} matrices in {time.perf_counter() - t0:.1f} s")

    payload = {fmt: sum(e[3].payload_bits for e in ents) / 8 for fmt, ents in packed.items()}
    total = {fmt: sum(e[3].total_bytes for e in ents) for fmt, ents in packed.items()}
    res, checks, unsupported = {}, {}, {}
    copies = max(1, args.copies)
    keep_sets = None
    for fmt in fmts:
        sets = device_copies(packed[fmt], copies)
        for kind in ("bf16", "int8"):
            if not supported(packed[fmt], kind, m):
                if fmt == N.FMT_BITCOS:
                    raise SystemExit(f"no BITCOS kernel for {name} with {kind} activations at batch {m}")
                res[(fmt, kind)] = None
                unsupported[f"{FMT_NAMES[fmt]}_{kind}"] = "no kernel for rows this long (K > 16384 with bf16 activations)"
                say(f"{name} {FMT_NAMES[fmt]} {kind}: no kernel for this set, skipped")
                continue
            steps = [make_step(st, acts, kind) for st in sets]
            gs = [capture(s) for s, _ in steps]
            ms = time_graphs(gs, args.steps, args.warmup, args.warm_ms)
            res[(fmt, kind)] = ms
            if check:
                rows_checked, worst, good = 0, 0.0, True
                for _, batches in steps:
                    g_ok, nrows, w_ = check_outputs(batches, samples, xhost, kind)
                    good &= g_ok
                    rows_checked += nrows
                    worst = max(worst, w_)
                checks[f"{FMT_NAMES[fmt]}_{kind}"] = {"ok": good, "outputs_checked": rows_checked,
                                                      "worst_error_over_allowed": round(worst, 6)}
                if not good:
                    say(f"{name} {FMT_NAMES[fmt]} {kind}: OUTPUTS DIFFER from the dense definition "
                        f"(worst error / allowed = {worst:.3g})")
            say(f"{name} {FMT_NAMES[fmt]} {kind}: {ms * 1e3:.1f} us/step, {payload[fmt] / (ms * 1e-3) / 1e9:.1f} GB/s"
                + (f", self-check {'ok' if checks[f'{FMT_NAMES[fmt]}_{kind}']['ok'] else 'FAILED'}" if check else ""))
            del gs, steps
        if fmt == N.FMT_BITCOS:
            keep_sets = sets
        del sets
    return {"wk": wk, "layers": layers, "m": m, "packed": packed, "acts": acts, "payload": payload,
            "total": total, "res": res, "checks": checks, "unsupported": unsupported, "bitcos_sets": keep_sets}


def summary(r, fmts):
    """The reported numbers of one layer set (value = BITCOS bf16)."""
    from paper_2609_16338_amd import _native as N

    res, payload, total, m = r["res"], r["payload"], r["total"], r["m"]
    packed = r["packed"]
    weights = sum(e[3].n * e[3].k for e in packed[N.FMT_BITCOS])
    ms = res[(N.FMT_BITCOS, "bf16")]
    ms8 = res[(N.FMT_BITCOS, "int8")]
    value = payload[N.FMT_BITCOS] / (ms * 1e-3) / 1e9

    def ratio(fmt, kind, t):
        v = res.get((fmt, kind))
        return None if v is None else round(v / t, 4)

    out = {
        "value": round(value, 2),
        "ms_per_step": round(ms, 5),
        "pct_of_hbm_peak": round(100 * value / HBM_PEAK_GBS, 2),
        "weights_per_s": float(f"{weights / (ms * 1e-3):.4g}"),
        "bpw_payload": round(payload[N.FMT_BITCOS] * 8 / weights, 5),
        "bpw_total": round(total[N.FMT_BITCOS] * 8 / weights, 5),
        "total_bytes_GBs": round(total[N.FMT_BITCOS] / (ms * 1e-3) / 1e9, 2),
    }
    if N.FMT_TRIT5 in fmts:
        out["speedup_vs_trit5"] = ratio(N.FMT_TRIT5, "bf16", ms)
        out["speedup_vs_bit2"] = ratio(N.FMT_BIT2, "bf16", ms)
        out["baselines_us_per_step"] = {
            f"{FMT_NAMES[f]}_{kind}": None if res[(f, kind)] is None else round(res[(f, kind)] * 1e3, 2)
            for f in (N.FMT_TRIT5, N.FMT_BIT2) for kind in ("bf16", "int8")}
        # Time ratios above; the byte ratios they compare against, on the
        # formats' payload (symbols + scales) and on whole blobs (payload +
        # sign offsets, padding and alignment).
        out["byte_ratio_payload"] = {f"{FMT_NAMES[f]}_over_bitcos": round(payload[f] / payload[N.FMT_BITCOS], 4)
                                     for f in (N.FMT_TRIT5, N.FMT_BIT2)}
        out["byte_ratio_total"] = {f"{FMT_NAMES[f]}_over_bitcos": round(total[f] / total[N.FMT_BITCOS], 4)
                                   for f in (N.FMT_TRIT5, N.FMT_BIT2)}
        if m > 1:
            out["baselines_note"] = f"no small-batch kernel: {m} batch-1 launches per tile and step"
        if r["unsupported"]:
            out["baselines_unsupported"] = r["unsupported"]
    out["int8_variant"] = {
        "value": round(payload[N.FMT_BITCOS] / (ms8 * 1e-3) / 1e9, 2),
        "ms_per_step": round(ms8, 5),
        "speedup_vs_trit5": ratio(N.FMT_TRIT5, "int8", ms8),
        "speedup_vs_bit2": ratio(N.FMT_BIT2, "int8", ms8),
    }
    if r["checks"]:
        out["self_check"] = r["checks"]
    return out


def dominant_roofline(r, args, name):
    """The persistent launch carrying most of the step's bytes (bf16), timed
    alone: ten back-to-back launches per graph replay, over the device copies
    in turn (inside a graph consecutive kernels start without a gap)."""
    from paper_2609_16338_amd import _native as N
    from paper_2609_16338_amd import api

    m = r["m"]
    tops = [make_batches(st, r["acts"], "bf16")[0] for st in r["bitcos_sets"]]
    top = tops[0]
    reps = 10
    gg = capture(lambda: [tops[i % len(tops)].run() for i in range(reps)])
    ms_g = time_graph(gg, args.steps, args.warmup, args.warm_ms)
    per_launch_us = ms_g * 1e3 / reps
    sclk = gpu_clock_under_load(gg)
    alg_bytes = sum(e[3].payload_bits / 8 + m * (e[3].k * 2 + e[3].n * 4) for e in top.entries)
    achieved = alg_bytes / (per_launch_us * 1e-6) / 1e9
    # Two-term roofline in CU-cycles per 32 weights (nominal clock): the
    # launch's measured time against the time its bytes take at peak HBM
    # bandwidth.  The operation sits under the HBM roofline (about 3
    # operations per byte); the larger term says what limits this kernel.
    top_weights = sum(e[3].n * e[3].k for e in top.entries)
    launch_gamma = 32 * CU_COUNT * CLOCK_HZ * per_launch_us * 1e-6 / top_weights
    hbm_term = 32 * alg_bytes / top_weights / (HBM_PEAK_GBS * 1e9 / (CU_COUNT * CLOCK_HZ))
    label = launch_label(top, m)
    # VALU issue: every SIMD (4 per CU) issues one wave instruction per 4
    # cycles (wave64 over 16 lanes; half-rate instructions count once, so
    # this is a lower bound); the share of the launch's SIMD-cycles at the
    # clock measured under load that the counted instructions occupy.
    valu_n = stored_valu(name, label)
    clk = (sclk or CLOCK_HZ / 1e6) * 1e6
    valu = None if valu_n is None else {
        "insts_per_launch": valu_n,
        "busy_frac": round(4 * valu_n / (4 * CU_COUNT * clk * per_launch_us * 1e-6), 4),
        "clock_mhz": round(clk / 1e6),
    }
    return {
        # The roofline the metric is read against (weight bytes per second vs
        # HBM peak); what limits the kernel today is the larger two_term term,
        # restated as "limiter".
        "bound": "hbm",
        "limiter": "instructions" if launch_gamma > hbm_term else "hbm",
        "achieved": round(achieved, 2),
        "peak": HBM_PEAK_GBS,
        "unit": "GB/s",
        "frac": round(achieved / HBM_PEAK_GBS, 4),
        "traffic": stored_traffic(name, label),
        "kernel": label,
        "per_launch_us": round(per_launch_us, 3),
        "bytes_per_launch": int(alg_bytes),
        "weights_per_launch": int(top_weights),
        "two_term": {"cu_cycles_per_32w": round(launch_gamma, 4), "hbm_cu_cycles_per_32w": round(hbm_term, 4),
                     "larger_term": "instructions" if launch_gamma > hbm_term else "hbm"},
        "valu": valu,
    }, sclk


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
    """The oracle (decode + dense GEMV) on the host, on whole matrices of layer 0
    taken in turn until about `budget_s` seconds of oracle work are timed
    (input generation and the oracle's packing are not timed)."""
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
    while t_total < budget_s:
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
            if t_total >= budget_s:
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


# ---------------------------------------------------------------------------
# Other modes
# ---------------------------------------------------------------------------

def profile_pass(args):
    """Counter runs: the dominant launch of the headline step, then a plain copy
    of known size whose FETCH_SIZE / WRITE_SIZE calibrate the counters."""
    import torch

    from paper_2609_16338_amd import _native as N

    wk = wl.WORKLOADS[args.workload]
    layers = args.layers or wk.layers
    packed = build_set(wk, layers, [N.FMT_BITCOS], args.threads)
    acts, _ = activations(wk, ("bf16",), args.batch)
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
    alg = sum(e[3].payload_bits / 8 + args.batch * (e[3].k * 2 + e[3].n * 4) for e in top.entries)
    print(f"[profile-pass] {args.workload} dominant launch: {launch_label(top, args.batch)}, "
          f"algorithmic bytes {int(alg)}; copy {COPY_MIB} MiB; "
          f"kernel_source_hash {kernel_source_hash(launch_label(top, args.batch).split('<')[0])}",
          flush=True)


def profile_sweep(args):
    """Counter runs on the zero-density sweep's launch at z = 0.42 (one 8192 x
    8192 g128 matrix, --sweep-copies device copies in one launch): BITCOS,
    five-trit and 2-bit, int8 then bf16 activations, each launch 5 times."""
    import torch

    from paper_2609_16338_amd import _native as N
    from paper_2609_16338_amd import api

    cid, k, z = 4, 8192, 0.42
    zi = wl.SWEEP_Z.index(z)
    spec = wl.sweep_spec(z)
    w, sc = wl.matrix_inputs(cid, 0, zi, spec)
    xi = torch.from_numpy(wl.activation_inputs(cid, "int8", 1, k)).cuda().reshape(-1)
    xb = torch.from_numpy(wl.activation_inputs(cid, "bf16", 1, k).view(np.int16)).view(torch.bfloat16).cuda().reshape(-1)
    for fmt in (N.FMT_BITCOS, N.FMT_TRIT5, N.FMT_BIT2):
        L, blob = api.plan_and_pack(fmt, w, sc, spec.group)
        src = torch.from_numpy(blob).cuda()
        blobs = [src.clone() for _ in range(args.sweep_copies)]
        for kind, x in (("int8", xi), ("bf16", xb)):
            ys = [torch.empty(spec.n, dtype=torch.float32, device="cuda") for _ in blobs]
            b = api.Batch([L] * len(blobs), blobs, [x] * len(blobs), ys)
            for _ in range(5):
                b.run()
            torch.cuda.synchronize()
            try:
                d = api.describe(L, 1, N.X_I8 if kind == "int8" else N.X_BF16)
                tile = f"kernel {d.kernel}, tile ({d.per_lane}, {d.seg_lanes})"
            except N.BitcosError:
                tile = "tile n/a"
            print(f"[profile-sweep] {FMT_NAMES[fmt]} {kind}: {len(blobs)} GEMVs of {spec.n}x{spec.k}, {tile}, "
                  f"payload bytes per GEMV {L.payload_bits // 8}", flush=True)
            del b, ys
        del blobs, src
        torch.cuda.empty_cache()


def hbm_read(args):
    """Plain streaming-read bandwidth of this GPU, for scale: torch reductions
    that read every byte of a 4 GiB tensor once and write one value (max of
    int32, sum of float32, sum of int64 viewed from the same bytes), and a
    4 GiB device copy (reads + writes counted).  Each is timed from a graph
    of ten back-to-back calls; value = the fastest read rate."""
    import torch
    nbytes = 4 << 30
    x = torch.randint(-1000, 1000, (nbytes // 4,), dtype=torch.int32, device="cuda")
    reps = 10
    res = {}
    outs = {"amax_int32": torch.empty((), dtype=torch.int32, device="cuda"),
            "sum_float32": torch.empty((), dtype=torch.float32, device="cuda"),
            "sum_int64": torch.empty((), dtype=torch.int64, device="cuda")}
    ops = {"amax_int32": lambda: torch.amax(x, dim=0, out=outs["amax_int32"]),
           "sum_float32": lambda: torch.sum(x.view(torch.float32), dim=0, out=outs["sum_float32"]),
           "sum_int64": lambda: torch.sum(x.view(torch.int64), dim=0, out=outs["sum_int64"])}
    for name, op in ops.items():
        g = capture(lambda op=op: [op() for _ in range(reps)])
        ms = time_graph(g, 20, 5, args.warm_ms)
        res[name] = round(reps * nbytes / (ms * 1e-3) / 1e9, 1)
        del g
    y = torch.empty_like(x)
    g = capture(lambda: [y.copy_(x) for _ in range(reps)])
    ms = time_graph(g, 20, 5, args.warm_ms)
    res["copy_read_plus_write"] = round(reps * 2 * nbytes / (ms * 1e-3) / 1e9, 1)
    best = max(v for k, v in res.items() if k != "copy_read_plus_write")
    emit({"metric": "plain streaming read bandwidth (torch reductions over 4 GiB; copy for comparison)",
          "value": best, "unit": "GB/s", "frac_of_peak": round(best / HBM_PEAK_GBS, 4), "bytes_per_read": nbytes,
          "rates_GBs": res}, args)


def sweep_points(args):
    """(n, k, [(z index, z)]) of the sweep: `--sweep-shape` N x K (multiples of
    128) and the `--sweep-z` densities, by default the five of the sweep and
    the paper's extreme 0.95; a z of the sweep keeps its seed index."""
    n, k = (int(v) for v in args.sweep_shape.lower().split("x"))
    if n < 1 or k < 128 or k % 128:
        raise SystemExit(f"--sweep-shape {args.sweep_shape}: N >= 1 and K a multiple of 128")
    allz = wl.SWEEP_Z + (0.95,)
    zs = [float(v) for v in args.sweep_z.split(",") if v] if args.sweep_z else list(allz)
    return n, k, [(allz.index(z) if z in allz else len(allz) + i, z) for i, z in enumerate(zs)]


def sweep(args):
    """Zero-density sweep: one N x K matrix (8192 x 8192 by default) with
    group-128 scales per z, batch 1, BITCOS against the five-trit and 2-bit
    kernels on this GPU.  Each format's blob is copied `--sweep-copies` times
    in HBM and one persistent launch covers all copies, so every launch
    streams more than twice the Infinity Cache; time per GEMV = launch time /
    copies."""
    import torch

    from paper_2609_16338_amd import _native as N
    from paper_2609_16338_amd import api

    cid = 4
    n, k, zpts = sweep_points(args)
    xi = torch.from_numpy(wl.activation_inputs(cid, "int8", 1, k)).cuda().reshape(-1)
    xb = torch.from_numpy(wl.activation_inputs(cid, "bf16", 1, k).view(np.int16)).view(torch.bfloat16).cuda().reshape(-1)
    names = {N.FMT_BITCOS: "bitcos", N.FMT_TRIT5: "trit5", N.FMT_BIT2: "bit2"}
    rows = []
    for zi, z in zpts:
        spec = wl.sweep_spec(z, n, k)
        w, sc = wl.matrix_inputs(cid, 0, zi, spec)
        row = {"z": z, "z_measured": round(float((w == 0).mean()), 5)}
        for fmt, nm in names.items():
            L, blob = api.plan_and_pack(fmt, w, sc, spec.group)
            src = torch.from_numpy(blob).cuda()
            blobs = [src.clone() for _ in range(args.sweep_copies)]
            row[f"{nm}_payload_bytes"] = L.payload_bits // 8
            row[f"{nm}_total_bytes"] = L.total_bytes
            row[f"{nm}_bpw"] = round(L.payload_bits / (spec.n * spec.k), 5)
            for kind, x in (("int8", xi), ("bf16", xb)):
                ys = [torch.empty(spec.n, dtype=torch.float32, device="cuda") for _ in blobs]
                b = api.Batch([L] * len(blobs), blobs, [x] * len(blobs), ys)
                g = capture(b.run)
                ms = time_graph(g, args.steps, args.warmup, args.warm_ms)
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

    emit({
        "metric": f"zero-density sweep, {n}x{k} g128, batch 1: per-GEMV time, effective GB/s, speedups",
        "unit": "us",
        "copies_per_launch": args.sweep_copies,
        "steps": args.steps,
        "warmup": args.warmup,
        "data": "synthetic",
        "crossover_z_vs_trit5_int8": crossover("int8"),
        "crossover_z_vs_trit5_bf16": crossover("bf16"),
        "points": rows,
    }, args)


GAMMA_Z = (0.30, 0.42, 0.515, 0.95)


def gamma(args):
    """The paper's two-term roofline (Sec. III-B, Eqs. (5)-(6)) on this GPU.

    gamma = CU-cycles one CU spends per 32 weights when the operands are
    L2-resident (one launch over 64 GEMVs that all read the same 2048 x 8192
    g128 blob, 3.6-4.4 MB, which each XCD's 4 MB L2 holds, so the instruction
    stream is the limit and the kernel's prologue is amortised); beta = HBM
    bytes per CU-cycle at the 8 TB/s peak; B(z) = bytes per 32 weights of each
    layout.  Predicted effective bandwidth = min(beta, B / gamma) per CU,
    times all CUs."""
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
                ms = time_graph(g, max(args.steps, 50), args.warmup, args.warm_ms)
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
    emit({
        "metric": "two-term roofline: gamma = CU-cycles per 32 weights, L2-resident 2048x8192 g128 (x64 per launch), batch 1",
        "beta_bytes_per_cu_cycle": round(beta, 4),
        "clock_hz": CLOCK_HZ,
        "cus": CU_COUNT,
        "data": "synthetic",
        "points": rows,
    }, args)


# ---------------------------------------------------------------------------
# Headline
# ---------------------------------------------------------------------------

def main(argv=None):
    args = parse(argv)
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1"}))
        sys.exit(2)
    if args.gamma:
        gamma(args)
        return
    if args.profile_pass:
        profile_pass(args)
        return
    if args.profile_sweep:
        profile_sweep(args)
        return
    if args.sweep:
        sweep(args)
        return
    if args.hbm_read:
        hbm_read(args)
        return
    import torch

    from paper_2609_16338_amd import _native as N

    N.lib()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    m = args.batch
    if not 1 <= m <= 16:
        print(json.dumps({"error": "--batch must be in 1..16"}))
        sys.exit(2)
    fmts = [N.FMT_BITCOS] + ([] if args.no_baselines else [N.FMT_TRIT5, N.FMT_BIT2])
    check = not args.no_check

    r = run_workload(args.workload, args, m, fmts, check)
    head = summary(r, fmts)
    roof, sclk = dominant_roofline(r, args, args.workload)
    wk, layers = r["wk"], r["layers"]
    packed = r["packed"]
    weights = sum(e[3].n * e[3].k for e in packed[N.FMT_BITCOS])
    out = {
        "metric": METRIC,
        "value": head.pop("value"),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head.pop("ms_per_step"),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": describe_workload(wk, layers, m) + ", bf16 x ~ N(0,1)",
            "global_batch": m,
            "layers": layers,
            "gemvs_per_step": len(packed[N.FMT_BITCOS]),
            "matrices_per_step": len({(e[0], e[1]) for e in packed[N.FMT_BITCOS]}),
            "column_blocks": {f"{s.name} {s.n}x{s.k}": len(column_blocks(s.k)) for s in wk.matrices
                              if len(column_blocks(s.k)) > 1},
            "weights_per_step": weights,
            "payload_bytes_per_step": int(r["payload"][N.FMT_BITCOS]),
            "total_bytes_per_step": int(r["total"][N.FMT_BITCOS]
                                        + sum(m * (e[3].k * 2 + e[3].n * 4) for e in packed[N.FMT_BITCOS])),
            "device_copies": max(1, args.copies),
            "warm_ms_per_format": args.warm_ms,
        },
    }
    out.update(head)
    out["roofline"] = roof
    out["sclk_mhz_under_load"] = sclk
    failed = [k for k, v in r["checks"].items() if not v["ok"]]
    del r
    torch.cuda.empty_cache()

    extras = {}
    for name in [s for s in args.extra.split(",") if s and s != args.workload]:
        re_ = run_workload(name, args, m, fmts, check)
        extras[name] = dict(workload=describe_workload(re_["wk"], re_["layers"], m), **summary(re_, fmts))
        failed += [f"{name}:{k}" for k, v in re_["checks"].items() if not v["ok"]]
        del re_
        torch.cuda.empty_cache()
    if extras:
        out["extra_workloads"] = extras
    if failed:
        print(json.dumps({"error": "self-check failed: GPU outputs differ from the dense definition",
                          "failed": failed}), flush=True)
        sys.exit(3)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wk)
    emit(out, args)


if __name__ == "__main__":
    main()
