"""GPU parity of the batch-1 BITCOS kernel that multiplies on the matrix cores.

The launcher runs it for layouts with one scale per tensor (or raw int32 sums)
and no activation scales; every row-segment width it is instantiated for
(4, 8, 16, 32, 64 lanes per row) is exercised below, with ragged row counts
and words, degenerate densities, extreme activations, batches (descriptor
tables) and the layouts that must fall back to the streaming kernel.  Bars as
in test_gpu_parity.py: int32 raw sums and per-tensor int8 bit-exact; bf16
within 1e-3 of sum |S W x| per element and in norm.
"""

import numpy as np
import pytest

import oracle as O
import workloads as wl
from parity_checks import bf16_bound, check_bf16, inputs, run, say, to_dev_x

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
api = pytest.importorskip("paper_2609_16338_amd.api")
from paper_2609_16338_amd import _native as N  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    N.lib()


# K -> (words per lane, lanes per row): 96 -> (1, 4) ragged, 128 -> (1, 4),
# 256 -> (2, 4), 512 -> (4, 4), 1024 -> (8, 4), 2048 -> (8, 8),
# 2400 -> (5, 16) ragged, 2560 -> (5, 16), 4096 -> (8, 16), 5120 -> (5, 32),
# 6912 -> (7, 32) ragged, 8192 -> (8, 32), 12288 -> (6, 64), 16384 -> (8, 64)
# (int8; bf16 takes at most 5 words where an equally full tile allows it:
# 1024 -> (4, 8), 2048 -> (4, 16), 4096 -> (4, 32), 8192 -> (4, 64)).
KS = [96, 128, 256, 512, 1024, 2048, 2400, 2560, 4096, 5120, 6912, 8192, 12288, 16384]


def _matrix_kernel(L, kind):
    return api.describe(L, 1, N.X_I8 if kind == "int8" else N.X_BF16).kernel == N.KERNEL_MATRIX


@pytest.mark.parametrize("k", KS)
def test_matrix_kernel_int8_raw_and_per_tensor(k):
    n = 77  # not a multiple of any step's rows
    w, sc = inputs(n, k, 0.42, 0, 11)
    x = wl.act_int8(1, k, wl.rng_for(110, k))
    y, L = run(N.FMT_BITCOS, w, sc, 0, x, "int8", y_mode=N.Y_I32_RAW)
    assert _matrix_kernel(L, "int8")
    assert np.array_equal(y, O.dense_gemv_raw(w, x).astype(np.int32))
    y, _ = run(N.FMT_BITCOS, w, sc, 0, x, "int8")
    assert np.array_equal(y, O.dense_gemv(w, sc, 0, x))


@pytest.mark.parametrize("k", KS)
def test_matrix_kernel_bf16_per_tensor(k):
    n = 53
    w, sc = inputs(n, k, 0.467, 0, 12)
    xb = wl.act_bf16(1, k, wl.rng_for(111, k))
    y, L = run(N.FMT_BITCOS, w, sc, 0, xb, "bf16")
    assert _matrix_kernel(L, "bf16")
    check_bf16(y, O.dense_gemv(w, sc, 0, xb, x_is_bf16_bits=True), bf16_bound(w, sc, 0, xb))


@pytest.mark.parametrize("k", [128, 256, 2560, 6912, 8192])
@pytest.mark.parametrize("z", [0.0, 1.0, 0.95])
def test_matrix_kernel_degenerate_densities(k, z):
    n = 19
    w, sc = inputs(n, k, z, 0, 13)
    x = wl.act_int8(1, k, wl.rng_for(112, k))
    y, _ = run(N.FMT_BITCOS, w, sc, 0, x, "int8", y_mode=N.Y_I32_RAW)
    assert np.array_equal(y, O.dense_gemv_raw(w, x).astype(np.int32))
    xb = wl.act_bf16(1, k, wl.rng_for(113, k))
    y, _ = run(N.FMT_BITCOS, w, sc, 0, xb, "bf16")
    check_bf16(y, O.dense_gemv(w, sc, 0, xb, x_is_bf16_bits=True), bf16_bound(w, sc, 0, xb))


def test_matrix_kernel_extreme_activations_and_rows():
    """All-(-1) and all-(+1) rows against +-127 / large bf16 activations."""
    for k in (256, 2560, 6912):
        w, sc = inputs(29, k, 0.42, 0, 14)
        w[0, :] = -1
        w[1, :] = 1
        w[2, :] = 0
        w[3, ::2] = 1
        x = np.full((1, k), -127, np.int8)
        x[0, ::3] = 127
        y, _ = run(N.FMT_BITCOS, w, sc, 0, x, "int8", y_mode=N.Y_I32_RAW)
        assert np.array_equal(y, O.dense_gemv_raw(w, x).astype(np.int32))
        xf = np.where(np.arange(k) % 2 == 0, 3.0e4, -2.5e4).astype(np.float32)[None]
        xb = (xf.view(np.uint32) >> 16).astype(np.uint16)
        y, _ = run(N.FMT_BITCOS, w, sc, 0, xb, "bf16")
        check_bf16(y, O.dense_gemv(w, sc, 0, xb, x_is_bf16_bits=True), bf16_bound(w, sc, 0, xb))


@pytest.mark.parametrize("k,unit,expect", [(2560, 2, N.KERNEL_STREAMING), (6912, 2, N.KERNEL_MATRIX),
                                           (5120, 2, N.KERNEL_MATRIX), (8192, 4, N.KERNEL_GENERAL),
                                           (2560, 3, N.KERNEL_GENERAL)])
def test_matrix_kernel_unit_rows_fallbacks(k, unit, expect):
    """Several rows per sign offset: at 16 or fewer lanes per row the streaming
    kernel runs, at 32 the matrix cores still do; a unit that does not divide
    the wave step (8192: two rows per step) takes the general kernel."""
    w, sc = inputs(37, k, 0.42, 0, 15)
    x = wl.act_int8(1, k, wl.rng_for(114, k))
    y, L = run(N.FMT_BITCOS, w, sc, 0, x, "int8", y_mode=N.Y_I32_RAW, unit=unit)
    assert L.unit_rows == unit and api.describe(L, 1, N.X_I8).kernel == expect
    assert np.array_equal(y, O.dense_gemv_raw(w, x).astype(np.int32))
    xb = wl.act_bf16(1, k, wl.rng_for(115, k))
    y, _ = run(N.FMT_BITCOS, w, sc, 0, xb, "bf16", unit=unit)
    check_bf16(y, O.dense_gemv(w, sc, 0, xb, x_is_bf16_bits=True), bf16_bound(w, sc, 0, xb))


@pytest.mark.parametrize("k", [256, 2560, 6912, 8192])
@pytest.mark.parametrize("kind", ["int8", "bf16"])
def test_matrix_kernel_batch_tables(k, kind):
    """Several GEMVs of one tile in one launch (descriptor table), twice: same bits."""
    specs = [(64, 0.42), (5, 0.0), (300, 0.5), (33, 1.0), (129, 0.467)]
    layouts, blobs, xs, ys, refs, bounds = [], [], [], [], [], []
    for i, (n, z) in enumerate(specs):
        w, sc = inputs(n, k, z, 0, 400 + i)
        if kind == "int8":
            x = wl.act_int8(1, k, wl.rng_for(401, i, k))
            refs.append(O.dense_gemv(w, sc, 0, x))
            bounds.append(None)
        else:
            x = wl.act_bf16(1, k, wl.rng_for(402, i, k))
            refs.append(O.dense_gemv(w, sc, 0, x, x_is_bf16_bits=True))
            bounds.append(bf16_bound(w, sc, 0, x))
        L, blob = api.plan_and_pack(N.FMT_BITCOS, w, sc, 0)
        layouts.append(L)
        blobs.append(torch.from_numpy(blob).cuda())
        xs.append(to_dev_x(x, kind).reshape(-1))
        ys.append(torch.full((n,), -7.0, dtype=torch.float32, device="cuda"))
    say("matrix-kernel batch", k, kind)
    b = api.Batch(layouts, blobs, xs, ys)
    for rep in range(2):
        b.run()
        torch.cuda.synchronize()
        got = [y.cpu().numpy()[None] for y in ys]
        for g, ref, bound in zip(got, refs, bounds):
            if kind == "int8":
                assert np.array_equal(g, ref)
            else:
                check_bf16(g, ref, bound)
        if rep == 0:
            first = [g.copy() for g in got]
        else:
            for g, f in zip(got, first):
                assert np.array_equal(g.view(np.uint32), f.view(np.uint32))


def test_matrix_kernel_batch_mixed_units_falls_back():
    """A batch with one layout of two rows per offset at 16 lanes per row runs
    the streaming kernel for all of its GEMVs, with the same results."""
    k = 2560
    layouts, blobs, xs, ys, refs = [], [], [], [], []
    for i, unit in enumerate((1, 2, 4)):
        w, sc = inputs(41, k, 0.42, 0, 500 + i)
        x = wl.act_int8(1, k, wl.rng_for(501, i))
        L, blob = api.plan_and_pack(N.FMT_BITCOS, w, sc, 0, unit)
        layouts.append(L)
        blobs.append(torch.from_numpy(blob).cuda())
        xs.append(to_dev_x(x, "int8").reshape(-1))
        ys.append(torch.zeros(41, dtype=torch.float32, device="cuda"))
        refs.append(O.dense_gemv(w, sc, 0, x))
    b = api.Batch(layouts, blobs, xs, ys)
    b.run()
    torch.cuda.synchronize()
    for y, ref in zip(ys, refs):
        assert np.array_equal(y.cpu().numpy()[None], ref)
