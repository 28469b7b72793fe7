"""Shared pieces of the GPU parity tests: seeded inputs, one GEMV through the
C ABI, and the tolerance checks against the oracle's dense definition.

Bars:
  * int32 raw row sums (int8 x): bit-exact.
  * one scale per tensor, int8 x, no activation scales: bit-exact (one fp32
    multiply of the exact row sum, which is what the oracle rounds).
  * group scales or activation scales, int8 x: |y - ref| <= 1e-5 * sum_g |S a A|
    (fp32 products and sums of at most K/128 group terms).
  * bf16 x: |y - ref| <= 1e-3 * sum_k |S W x| per element and
    ||y - ref|| <= 1e-3 ||ref|| (fp32 accumulation of at most K products).
"""

import sys

import numpy as np

import oracle as O
import workloads as wl
from paper_2609_16338_amd import _native as N
from paper_2609_16338_amd import api

FMT_NAME = {1: "bitcos", 2: "trit5", 3: "bit2"}


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def to_dev_x(x, kind):
    import torch
    if kind == "int8":
        return torch.from_numpy(np.ascontiguousarray(x, dtype=np.int8)).cuda()
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.uint16).view(np.int16)).view(torch.bfloat16).cuda()


def run(fmt, w, sc, group, x, kind, xscale=None, y_mode=N.Y_F32, unit=0):
    import torch
    L, blob = api.plan_and_pack(fmt, w, sc, group, unit)
    say(FMT_NAME[fmt], w.shape, f"group={group}", kind, "xscale" if xscale is not None else "",
        "raw" if y_mode == N.Y_I32_RAW else "f32", f"unit={L.unit_rows}")
    blob_d = torch.from_numpy(blob).cuda()
    xd = to_dev_x(x, kind)
    m = x.shape[0]
    y = torch.full((m, w.shape[0]), -7, dtype=torch.int32 if y_mode == N.Y_I32_RAW else torch.float32,
                   device="cuda")
    xs = None if xscale is None else torch.from_numpy(np.ascontiguousarray(xscale, np.float32)).cuda()
    api.gemv(L, blob_d, xd, y, xs, y_mode)
    torch.cuda.synchronize()
    return y.cpu().numpy(), L


def group_bound(w, sc, group, x, xscale=None):
    """sum_g |S a A| per output (int8 x)."""
    n, k = w.shape
    g = k // 128
    A = np.einsum("ngk,mgk->mng", w.astype(np.float64).reshape(n, g, 128),
                  np.atleast_2d(x).astype(np.float64).reshape(-1, g, 128))
    S = O.fp16_bits_to_f64(sc).reshape(n, g) if group == 128 else np.full((n, g), O.fp16_bits_to_f64(sc)[0])
    a = np.ones((A.shape[0], g)) if xscale is None else np.asarray(xscale, np.float64).reshape(-1, g)
    return np.abs(S[None] * a[:, None, :] * A).sum(axis=2)


def bf16_bound(w, sc, group, xbits):
    n, k = w.shape
    xf = O.bf16_bits_to_f64(xbits).reshape(-1, k)
    if group == 128:
        S = np.repeat(O.fp16_bits_to_f64(sc).reshape(n, k // 128), 128, axis=1)
    else:
        S = np.full((n, k), O.fp16_bits_to_f64(sc)[0])
    return np.abs(xf) @ np.abs(S * w).T


def check_bf16(y, ref, bound):
    err = np.abs(y.astype(np.float64) - ref.astype(np.float64))
    assert np.all(err <= 1e-3 * bound + 1e-30), float((err / (bound + 1e-30)).max())
    assert np.linalg.norm(err) <= 1e-3 * np.linalg.norm(ref.astype(np.float64)) + 1e-30


def check_grouped(y, ref, bound):
    err = np.abs(y.astype(np.float64) - ref.astype(np.float64))
    assert np.all(err <= 1e-5 * bound + 1e-30), float((err / (bound + 1e-30)).max())


def inputs(n, k, z, group, seed, lo=0.01, hi=0.1):
    w = wl.ternary(n, k, z, wl.rng_for(90, seed, n, k))
    ns = n * (k // 128) if group == 128 else 1
    sc = wl.fp16_uniform((ns,), lo, hi, wl.rng_for(91, seed, n, k))
    return w, sc


def sampled_rows(n, count, seed):
    rng = np.random.default_rng(seed)
    rows = set(rng.choice(n, size=min(count, n), replace=False).tolist()) | {0, n - 1}
    return np.array(sorted(rows))
